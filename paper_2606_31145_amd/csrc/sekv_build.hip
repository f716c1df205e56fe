// Prefill-side cache builder for gfx950: the step before the decode path (Sec. 3.1 and
// Sec. 3.2).  Three kernels:
//
//   segment_kernel   surprisal segmentation of one sequence per workgroup: mu and sigma
//                    of the sequence's surprisal in one fixed summation order (1024
//                    strided float64 partials, then halving), boundaries where
//                    H_t > mu + alpha sigma, the local window, runs between neighbouring
//                    anchors shorter than min_span back to full resolution; anchors and
//                    spans listed in token order.  Integer results, exact.
//   gather_kernel    anchor rows of the token keys/values into the anchor arrays, and the
//                    surprisal-weighted mean key and value of every span (eq.
//                    surprisal_weight; float32 accumulation), |S| and ln|S|.
//   svd_kernel       one (sequence, KV head, span, side) per workgroup: a randomized
//                    truncated SVD of the span's |S| x d matrix X (eq. key_svd, rank
//                    r = min(|S|, d, R_max)).  Sketch Y = X Omega with the caller's d x l
//                    test matrix; G = Y^T Y (float64) = R^T R by Cholesky with diagonal
//                    pivoting, stopped where the remaining pivots fall below 1e-8 of the
//                    largest diagonal (a rank-deficient sketch keeps k < l columns), so
//                    Q = Y_piv R^-1 is an orthonormal basis of the sketch's range;
//                    B = Q^T X = R^-T (Y_piv^T X).  Each subspace iteration replaces Omega
//                    by an orthonormal basis of B's row space (pivoted Cholesky of B B^T
//                    again) and sketches anew.  Last, B B^T = E diag(sigma^2) E^T by
//                    cyclic Jacobi rotations (stopped once a sweep rotates nothing),
//                    V^T = diag(1/sigma) E^T B and U = Q E = Y_piv (R^-1 E).  The factors go
//                    into the span's block of the factor arena, stored with the rank
//                    rounded up to the 16-byte granule (the extra components zero).

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "sekv_internal.h"
#include "sekv_build_internal.h"

namespace sekv {
namespace {

constexpr int kSegThreads = 1024;
constexpr int BT = 256;                 // builder threads per workgroup
constexpr int kMaxL = 40;               // largest sketch width
constexpr int kTile = 16;               // tokens per streamed tile in the SVD
template <int N> struct Cint { static constexpr int value = N; };

__device__ inline float ld_elem(const void *base, size_t i, int elem) {
    if (elem == 2) {
        const uint16_t u = reinterpret_cast<const uint16_t *>(base)[i];
        return __uint_as_float(uint32_t(u) << 16);
    }
    return reinterpret_cast<const float *>(base)[i];
}

__device__ inline void st_elem(void *base, size_t i, float v, int elem) {
    if (elem == 2) {
        uint32_t u = __float_as_uint(v);
        u += 0x7FFFu + ((u >> 16) & 1u);                 // round to nearest even
        reinterpret_cast<uint16_t *>(base)[i] = uint16_t(u >> 16);
    } else {
        reinterpret_cast<float *>(base)[i] = v;
    }
}

// ---------------------------------------------------------------------------
// segmentation
// ---------------------------------------------------------------------------

// Exclusive scan of cnt[0, kSegThreads) in place (Hillis-Steele); returns the total.
__device__ int block_scan(int *cnt, int *tmp, int tid) {
    int v = cnt[tid];
    for (int off = 1; off < kSegThreads; off <<= 1) {
        tmp[tid] = v;
        __syncthreads();
        if (tid >= off) v += tmp[tid - off];
        __syncthreads();
    }
    tmp[tid] = v;                                       // inclusive
    __syncthreads();
    const int total = tmp[kSegThreads - 1];
    cnt[tid] = tid > 0 ? tmp[tid - 1] : 0;
    __syncthreads();
    return total;
}

// Sum of the values in the fixed order of the segmentation rule.
__device__ double fixed_order_sum(double mine, double *part, int tid) {
    part[tid] = mine;
    __syncthreads();
    for (int h = kSegThreads / 2; h >= 1; h >>= 1) {
        if (tid < h) part[tid] = part[tid] + part[tid + h];
        __syncthreads();
    }
    const double s = part[0];
    __syncthreads();
    return s;
}

__global__ void __launch_bounds__(kSegThreads) segment_kernel(SegArgs a) {
    __shared__ double part[kSegThreads];
    __shared__ int cnt[kSegThreads], tmp[kSegThreads];
    const int tid = threadIdx.x, b = blockIdx.x;
    int n = a.n_tokens[b];
    n = n < 0 ? 0 : (n > a.N ? a.N : n);
    const float *H = a.surprisal + size_t(b) * a.N;
    unsigned char *flag = a.ws_flag + size_t(b) * a.N;
    unsigned char *inspan = a.ws_inspan + size_t(b) * a.N;
    int32_t *pos = a.ws_pos + size_t(b) * (a.N + 2);
    int32_t *anchor_idx = a.anchor_idx + size_t(b) * a.N;
    int32_t *span_start = a.span_start + size_t(b) * a.N;
    int32_t *span_len = a.span_len + size_t(b) * a.N;
    if (n == 0) {
        if (tid == 0) { a.n_anchors[b] = 0; a.n_spans[b] = 0; }
        return;
    }
    // 1. mu and sigma, each sum in the fixed order; no fused multiply-add anywhere
    double thr;
    {
#pragma clang fp contract(off)
        double acc = 0.0;
        for (int t = tid; t < n; t += kSegThreads) acc = acc + double(H[t]);
        const double mu = fixed_order_sum(acc, part, tid) / double(n);
        double acc2 = 0.0;
        for (int t = tid; t < n; t += kSegThreads) {
            const double dv = double(H[t]) - mu;
            const double sq = dv * dv;
            acc2 = acc2 + sq;
        }
        const double sigma = sqrt(fixed_order_sum(acc2, part, tid) / double(n));
        const double as = a.alpha * sigma;
        thr = mu + as;
    }
    // 2. boundary and window flags; inspan cleared
    for (int t = tid; t < n; t += kSegThreads) {
        flag[t] = (double(H[t]) > thr || t >= n - a.window) ? 1 : 0;
        inspan[t] = 0;
    }
    __syncthreads();
    // 3. positions of the flagged tokens, in order, between sentinels -1 and n
    const int chunk = (n + kSegThreads - 1) / kSegThreads;
    const int t0 = tid * chunk, t1 = min(n, t0 + chunk);
    int c = 0;
    for (int t = t0; t < t1; ++t) c += flag[t];
    cnt[tid] = c;
    __syncthreads();
    const int m = block_scan(cnt, tmp, tid);
    {
        int w = cnt[tid];
        for (int t = t0; t < t1; ++t)
            if (flag[t]) pos[1 + w++] = t;
    }
    if (tid == 0) { pos[0] = -1; pos[m + 1] = n; }
    __syncthreads();
    // 4. the m + 1 gaps between consecutive positions: long ones are spans
    const int ng = m + 1;
    const int gchunk = (ng + kSegThreads - 1) / kSegThreads;
    const int g0 = tid * gchunk, g1 = min(ng, g0 + gchunk);
    c = 0;
    for (int i = g0; i < g1; ++i) c += (pos[i + 1] - pos[i] - 1 >= a.min_span) ? 1 : 0;
    cnt[tid] = c;
    __syncthreads();
    const int ns = block_scan(cnt, tmp, tid);
    {
        int w = cnt[tid];
        for (int i = g0; i < g1; ++i) {
            const int s = pos[i] + 1, L = pos[i + 1] - pos[i] - 1;
            if (L >= a.min_span) {
                span_start[w] = s;
                span_len[w] = L;
                ++w;
                for (int t = s; t < s + L; ++t) inspan[t] = 1;
            }
        }
    }
    __syncthreads();
    // 5. anchors: every token outside the spans, in order
    c = 0;
    for (int t = t0; t < t1; ++t) c += inspan[t] ? 0 : 1;
    cnt[tid] = c;
    __syncthreads();
    const int na = block_scan(cnt, tmp, tid);
    {
        int w = cnt[tid];
        for (int t = t0; t < t1; ++t)
            if (!inspan[t]) anchor_idx[w++] = t;
    }
    if (tid == 0) { a.n_anchors[b] = na; a.n_spans[b] = ns; }
}

// ---------------------------------------------------------------------------
// anchors and summaries
// ---------------------------------------------------------------------------

// Tokens of sequence b, clamped to [0, N] as the segmentation clamps them.
__device__ inline int seq_tokens(const BuildArgs &a, int b) {
    const int n = a.n_tokens[b];
    return n < 0 ? 0 : min(n, a.N);
}

// An anchor index or span outside the sequence's tokens: the row or span is skipped.
__device__ inline void flag_table(const BuildArgs &a) {
    __hip_atomic_fetch_or(a.error, kErrSelRange, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// grid = B * Hkv * rows workgroups; workgroup (pair, y) copies anchor rows
// [64 y, 64 y + 64) and summarises span y.
__global__ void __launch_bounds__(BT) gather_kernel(BuildArgs a, int rows) {
    const int pair = blockIdx.x / rows, b = pair / a.Hkv, g = pair % a.Hkv;
    const int y = blockIdx.x % rows, tid = threadIdx.x;
    const int d = a.d, e = a.elem;
    const size_t tok0 = size_t(pair) * a.N;                 // row of token 0 of (b, g)
    const int nt = seq_tokens(a, b);
    int na = a.n_anchors[b];
    na = na < 0 ? 0 : min(na, min(a.A_max, a.N));
    int ns = a.n_spans[b];
    ns = ns < 0 ? 0 : min(ns, min(a.M_max, a.N));
    // anchor rows
    for (int i = tid; i < 64 * d; i += BT) {
        const int r = y * 64 + i / d, col = i % d;
        if (r < na) {
            const int t = a.anchor_idx[size_t(b) * a.N + r];
            if (t >= 0 && t < nt) {
                const size_t dst = (size_t(pair) * a.A_max + r) * d + col;
                st_elem(a.anchor_k, dst, ld_elem(a.keys, (tok0 + t) * d + col, e), e);
                st_elem(a.anchor_v, dst, ld_elem(a.values, (tok0 + t) * d + col, e), e);
            } else if (col == 0) {
                flag_table(a);
            }
        }
    }
    // span y: surprisal-weighted means; |S| and ln|S| once per sequence (g == 0)
    if (y >= ns) return;
    const int s0 = a.span_start[size_t(b) * a.N + y];
    int L = a.span_len_seg[size_t(b) * a.N + y];
    if (s0 < 0 || L < 1 || s0 + L > nt) {
        if (tid == 0 && g == 0) flag_table(a);
        return;
    }
    __shared__ float red[2][BT];
    __shared__ float hs;
    // weight normaliser sum_t H_t over the span (float64 then float32)
    {
        double acc = 0.0;
        for (int t = tid; t < L; t += BT) acc += double(a.surprisal[size_t(b) * a.N + s0 + t]);
        red[0][tid] = float(acc);
        __syncthreads();
        if (tid == 0) {
            double s = 0.0;
            for (int i = 0; i < BT; ++i) s += double(red[0][i]);
            hs = float(s);
        }
        __syncthreads();
    }
    const float tot = hs;
    const bool uniform = !(tot > 0.0f);
    // thread: column col, token parity par (two tokens streams), then one pass through LDS
    const int col = tid % d, par = tid / d, npar = BT / d;
    float ak = 0.0f, av = 0.0f;
    for (int t = par; t < L; t += npar) {
        const float w = uniform ? 1.0f / float(L) : a.surprisal[size_t(b) * a.N + s0 + t] / tot;
        ak += w * ld_elem(a.keys, (tok0 + s0 + t) * d + col, e);
        av += w * ld_elem(a.values, (tok0 + s0 + t) * d + col, e);
    }
    red[0][tid] = ak;
    red[1][tid] = av;
    __syncthreads();
    if (par == 0) {
        float sk = 0.0f, sv = 0.0f;
        for (int p = 0; p < npar; ++p) { sk += red[0][p * d + col]; sv += red[1][p * d + col]; }
        const size_t dst = (size_t(pair) * a.M_max + y) * d + col;
        st_elem(a.sum_k, dst, sk, e);
        st_elem(a.sum_v, dst, sv, e);
    }
    if (g == 0 && tid == 0) {
        a.span_len_out[size_t(b) * a.M_max + y] = L;
        a.span_logsize[size_t(b) * a.M_max + y] = log(double(L));
    }
}

// ---------------------------------------------------------------------------
// randomized truncated SVD of one span side
// ---------------------------------------------------------------------------

// LDS of the SVD.  Region a holds the passes' tiles or, between passes, the two Cholesky
// factors / Jacobi vectors; bm accumulates Y^T X during a pass and then holds B; am
// accumulates G during a pass, then B B^T (and the Jacobi matrix, or Rinv), and last T.
constexpr int KL = kMaxL;
struct SvdSmem {
    union {
        struct {                              // passes over X
            uint16_t om[KL][128 + 4];         // the test matrix, transposed (l x d), as
                                              //   bfloat16 (any fixed test matrix serves;
                                              //   both passes of an iteration use this one);
                                              //   rows padded to 8-byte vectors off the
                                              //   same banks
            float x[kTile][128 + 4];          // token tile (rows: 16-byte vectors)
            float yt[kTile][KL + 4];          // sketch tile Y = X Omega (rows: 16-byte vectors)
        } p;
        struct {                              // between passes (float64: a Gram matrix
            double rg[KL][KL + 1];            //   squares the condition number)
            double em[KL][KL + 1];            // rg: R of G (rows: pivot steps, columns:
        } s;                                  //   sketch columns); em: R of B B^T
    } u;                                      //   (subspace iteration) or E (last pass)
    float bm[KL][128 + 4];                    // Y^T X, then B (rows in pivot order; 16-byte vectors)
    double am[KL][KL + 1];                    // G; B B^T; Rinv; T = R^-1 E
    double a2[KL][KL + 1];                    // Jacobi: the second copy of the rotated matrix
    double2 jcs[BT / 64][KL / 2];             // Jacobi: each wave's (c, s) of the round
    uint16_t jpq[KL - 1][KL / 2];             // Jacobi: pair i of round k is (p, q) = (lo, hi byte)
    double sig[KL];
    double dg[2][KL];                         // remaining Cholesky diagonal (two copies)
    int piv[KL], piv2[KL], order[KL];
    int pos[KL];                              // U pass: column of sketch column m (pivot order)
    int nconv[2];
};

// Two workgroups share a CU's 160 KiB of LDS (the occupancy the launch bounds ask for).
static_assert(sizeof(SvdSmem) <= 80 * 1024, "SVD LDS over half a CU's LDS");

// Round-robin pairing of round k among n (even) indices: index n-1 stays, the others
// rotate; pair i of the round is (p, q) with p < q.  Every pair meets once per sweep.
// (0 <= k < n - 1, 0 <= i < n / 2: every reduction below is one conditional step.)
__device__ inline void rr_pair(int n, int k, int i, int *p, int *q) {
    const int m = n - 1;
    int a0, b0;
    if (i == 0) { a0 = m; b0 = k; }
    else {
        a0 = k + i;
        if (a0 >= m) a0 -= m;
        b0 = k - i;
        if (b0 < 0) b0 += m;
    }
    *p = min(a0, b0);
    *q = max(a0, b0);
}

// Cyclic Jacobi on the symmetric n x n matrix A (n even): A is rotated towards diagonal,
// V (set to I here) accumulates the rotations, so that A_in = V diag(A_out) V^T; on
// return the diagonal of A holds A_out's (the rest of A is left undefined).  A pair is
// rotated when its off-diagonal entry exceeds 1e-10 of the geometric mean of its
// diagonal entries; the sweeps stop after one that rotates no pair.
//
// One barrier per round.  A is kept in two copies (A and sm.a2): a round reads one and
// writes the other in full, so lanes 0 .. n/2 - 1 of every wave can take the round's
// rotations from the copy being read while other waves already write theirs.  Each wave
// keeps its rotations in its own row of sm.jcs (written and read by that wave only: its
// LDS accesses complete in order).  A is updated as 2 x 2 blocks of pairs (I <= J), each
// block and its transpose by one thread; V as column pairs, one pair J and several rows
// per thread.
__device__ void jacobi(double (*A)[KL + 1], double (*V)[KL + 1], SvdSmem &sm, int n, int sweeps, int tid) {
    const int lane = tid & 63, wave = tid >> 6, np = n / 2;
    for (int idx = tid; idx < n * n; idx += BT) V[idx / n][idx % n] = (idx / n == idx % n) ? 1.0 : 0.0;
    for (int idx = tid; idx < (n - 1) * np; idx += BT) {
        int p, q;
        rr_pair(n, idx / np, idx % np, &p, &q);
        sm.jpq[idx / np][idx % np] = uint16_t(p | (q << 8));
    }
    if (tid < 2) sm.nconv[tid] = 0;
    // this thread's block (bI, bJ), bI <= bJ, of the np (np + 1) / 2 blocks
    const int nblk = np * (np + 1) / 2;
    int bI = 0, bJ = 0;
    if (tid < nblk) {
        int t = tid;
        while (t >= np - bI) { t -= np - bI; ++bI; }
        bJ = bI + t;
    }
    // this thread's V column pair vJ and rows vr0, vr0 + vstep, ... (threads past
    // vstep * np have none)
    const int vstep = BT / np, vJ = tid % np, vr0 = tid / np;
    constexpr int NVR = (KL + (BT / (KL / 2)) - 1) / (BT / (KL / 2)) + 1;   // rows per thread, bound
    __syncthreads();
    double(*cur)[KL + 1] = A;
    double(*nxt)[KL + 1] = sm.a2;
    for (int sweep = 0; sweep < sweeps; ++sweep) {
        const int par = sweep & 1;
        for (int k = 0; k < n - 1; ++k) {
            double c = 1.0, s = 0.0;
            if (lane < np) {
                const uint32_t pq = sm.jpq[k][lane];
                const int p = pq & 255, q = pq >> 8;
                const double app = cur[p][p], aqq = cur[q][q], apq = cur[p][q];
                // the test and the rotation side by side (no branch between them): when
                // the test fails, the rotation (possibly of a zero apq) is dropped
                const bool rot = fabs(apq) > 1e-10 * sqrt(fabs(app) * fabs(aqq)) && apq != 0.0;
                const double th = (aqq - app) / (2.0 * apq);
                const double t = (th >= 0.0 ? 1.0 : -1.0) / (fabs(th) + sqrt(1.0 + th * th));
                const double cr = 1.0 / sqrt(1.0 + t * t);
                if (rot) { c = cr; s = t * cr; }
            }
            // a round that rotates no pair leaves A and V as they are (its update would
            // copy them exactly): every wave sees the same rotations, so all skip it
            // together, with no barrier and no change of copy
            if (__ballot(s != 0.0) == 0) continue;
            if (lane == 0) sm.nconv[par] = 1;
            if (lane < np) sm.jcs[wave][lane] = make_double2(c, s);
            __builtin_amdgcn_wave_barrier();
            if (tid < nblk) {
                const uint32_t pqI = sm.jpq[k][bI], pqJ = sm.jpq[k][bJ];
                const int pI = pqI & 255, qI = pqI >> 8, pJ = pqJ & 255, qJ = pqJ >> 8;
                const double2 csI = sm.jcs[wave][bI], csJ = sm.jcs[wave][bJ];
                const double cI = csI.x, sI = csI.y, cJ = csJ.x, sJ = csJ.y;
                const double a = cur[pI][pJ], b = cur[pI][qJ], cc = cur[qI][pJ], dd = cur[qI][qJ];
                const double t00 = cI * a - sI * cc, t01 = cI * b - sI * dd;
                const double t10 = sI * a + cI * cc, t11 = sI * b + cI * dd;
                const double n00 = t00 * cJ - t01 * sJ, n01 = t00 * sJ + t01 * cJ;
                const double n10 = t10 * cJ - t11 * sJ, n11 = t10 * sJ + t11 * cJ;
                nxt[pI][pJ] = n00; nxt[pI][qJ] = n01; nxt[qI][pJ] = n10; nxt[qI][qJ] = n11;
                if (bI != bJ) { nxt[pJ][pI] = n00; nxt[qJ][pI] = n01; nxt[pJ][qI] = n10; nxt[qJ][qI] = n11; }
            }
            if (vr0 < vstep) {
                const uint32_t pqJ = sm.jpq[k][vJ];
                const int pJ = pqJ & 255, qJ = pqJ >> 8;
                const double2 csJ = sm.jcs[wave][vJ];
                if (csJ.y != 0.0) {
#pragma unroll
                    for (int u = 0; u < NVR; ++u) {
                        const int r = vr0 + vstep * u;
                        if (r < n) {
                            const double vp = V[r][pJ], vq = V[r][qJ];
                            V[r][pJ] = csJ.x * vp - csJ.y * vq;
                            V[r][qJ] = csJ.y * vp + csJ.x * vq;
                        }
                    }
                }
            }
            __syncthreads();
            double(*sw)[KL + 1] = cur;
            cur = nxt;
            nxt = sw;
        }
        const int rotated = sm.nconv[par];
        if (tid == 0) sm.nconv[par ^ 1] = 0;     // the next sweep's flag; this one is read
        __syncthreads();                         // by every thread before it is reset again
        if (!rotated) break;
    }
    if (cur != A && tid < n) A[tid][tid] = cur[tid][tid];
    __syncthreads();
}

// Largest 64-bit key over the wave, in every lane: quad and row steps by DPP, then the
// row and half swaps (permlane16 / permlane32), all without LDS round trips.
template <int CTRL>
__device__ inline uint64_t dpp64(uint64_t x) {
    const uint32_t lo = uint32_t(__builtin_amdgcn_update_dpp(0, int(uint32_t(x)), CTRL, 0xF, 0xF, false));
    const uint32_t hi = uint32_t(__builtin_amdgcn_update_dpp(0, int(uint32_t(x >> 32)), CTRL, 0xF, 0xF, false));
    return (uint64_t(hi) << 32) | lo;
}
__device__ inline uint64_t max64(uint64_t a, uint64_t b) { return a > b ? a : b; }
__device__ inline uint64_t wave_max_key(uint64_t x) {
    x = max64(x, dpp64<0xB1>(x));                               // quad_perm [1,0,3,2]
    x = max64(x, dpp64<0x4E>(x));                               // quad_perm [2,3,0,1]
    x = max64(x, dpp64<0x124>(x));                              // row_ror:4
    x = max64(x, dpp64<0x128>(x));                              // row_ror:8
    {
        const auto lo = __builtin_amdgcn_permlane16_swap(uint32_t(x), uint32_t(x), false, false);
        const auto hi = __builtin_amdgcn_permlane16_swap(uint32_t(x >> 32), uint32_t(x >> 32), false, false);
        x = max64((uint64_t(hi[0]) << 32) | lo[0], (uint64_t(hi[1]) << 32) | lo[1]);
    }
    {
        const auto lo = __builtin_amdgcn_permlane32_swap(uint32_t(x), uint32_t(x), false, false);
        const auto hi = __builtin_amdgcn_permlane32_swap(uint32_t(x >> 32), uint32_t(x >> 32), false, false);
        x = max64((uint64_t(hi[0]) << 32) | lo[0], (uint64_t(hi[1]) << 32) | lo[1]);
    }
    return x;
}

// Cholesky with diagonal pivoting of the symmetric positive semi-definite n x n matrix A
// (destroyed): step j takes the largest remaining diagonal entry p = piv[j] and stores
// row j of the factor over the original indices in Rm (Rm[j][piv[i]] = 0 for i < j), so
// that A ~ Rm^T Rm.  Stops when the largest remaining entry is not above tau times the
// largest initial diagonal entry; returns the number of steps k.  Ties go to the lower
// index.  One barrier per step: every wave finds the pivot itself from the remaining
// diagonal, kept in two alternating copies (-1 marks a row already taken): the largest
// positive entry by a wave maximum of the entries' bits (a positive double's bits order as
// its value), its lowest row by a ballot; every thread keeps the set of taken rows as a
// bit mask.
__device__ int piv_chol(double (*A)[KL + 1], double (*Rm)[KL + 1], int *piv, SvdSmem &sm, int n, double tau,
                        int tid) {
    constexpr int NE = (KL * KL + BT - 1) / BT;
    const int lane = tid & 63;
    if (tid < KL) {
        piv[tid] = 0;
        sm.dg[0][tid] = tid < n ? A[tid][tid] : -1.0;
    }
    __syncthreads();
    double floor_ = 0.0;
    uint64_t taken = 0;
    int k = 0;
    for (int j = 0; j < n; ++j) {
        const int cur = j & 1;
        const double dl = lane < n ? sm.dg[cur][lane] : -1.0;
        const uint64_t key = dl > 0.0 ? uint64_t(__double_as_longlong(dl)) : 0ull;
        const uint64_t kmax = wave_max_key(key);
        if (kmax == 0ull) break;                              // nothing positive remains
        const double v = __longlong_as_double(static_cast<long long>(kmax));
        if (j == 0) floor_ = tau * v;
        if (!(v > floor_)) break;                             // the same decision in every wave
        const int p = __ffsll(static_cast<long long>(__ballot(key == kmax))) - 1;
        const double rinv = 1.0 / sqrt(A[p][p]);
        taken |= uint64_t(1) << p;
        if (tid < n) {
            double r = 0.0;
            if (tid == p) r = 1.0 / rinv;
            else if (!((taken >> tid) & 1)) r = A[p][tid] * rinv;
            Rm[j][tid] = r;
        }
        if (tid == 0) piv[j] = p;
#pragma unroll
        for (int u = 0; u < NE; ++u) {
            const int idx = tid + BT * u;
            const int i = idx / KL, m = idx % KL;
            if (i < n && m < n) {
                const bool live = !((taken >> i) & 1) && !((taken >> m) & 1);
                double nv = -1.0;
                if (live) {
                    nv = A[i][m] - (A[p][i] * rinv) * (A[p][m] * rinv);
                    A[i][m] = nv;
                }
                if (i == m) sm.dg[cur ^ 1][i] = nv;
            }
        }
        __syncthreads();
        k = j + 1;
    }
    return k;
}

// Ri = Rt^-1 for Rt[j][m] = Rm[j][piv[m]] (k x k upper triangular; entries past k zero).
// Rt goes into Rp first; then thread i < k forms column i of Ri by back substitution,
// rows from the last up: a column needs only its own earlier entries, so no thread waits
// for another (Ri may be the storage of Rm).
__device__ inline void tri_inverse(const double (*Rm)[KL + 1], const int *piv, double (*Rp)[KL + 1],
                                   double (*Ri)[KL + 1], int k, int tid) {
    for (int idx = tid; idx < KL * KL; idx += BT) {
        const int j = idx / KL, m = idx % KL;
        Rp[j][m] = (j < k && m < k && m >= j) ? Rm[j][piv[m]] : 0.0;
    }
    __syncthreads();
    for (int idx = tid; idx < KL * KL; idx += BT) {
        const int j = idx / KL, i = idx % KL;
        if (j >= k || i >= k) Ri[j][i] = 0.0;
    }
    if (tid < k) {
        const int i = tid;
        for (int j = k - 1; j >= 0; --j) {
            // the same trip count in every lane (terms past the lane's diagonal are not
            // added), so the loop's LDS reads can be issued ahead of the sums
            double acc = j == i ? 1.0 : 0.0;
#pragma unroll 4
            for (int m = j + 1; m < k; ++m) {
                const double t = acc - Rp[j][m] * Ri[m][i];
                acc = m <= i ? t : acc;
            }
            Ri[j][i] = j <= i ? acc / Rp[j][j] : 0.0;
        }
    }
    __syncthreads();
}

// Z = Ri^T W[piv] with W and Z in the same LDS rows (rows >= k of Z zero).  Thread tid
// forms the 5 x CW block of Z at rows 5 (tid / 32), columns CW (tid % 32) (CW = d / 32),
// each entry summed over i in order, reads every row of W before a barrier, then writes.
template <int CW>
__device__ inline void apply_rinv_t_cw(float (*W)[128 + 4], const double (*Ri)[KL + 1], const int *piv, int k,
                                       int tid) {
    const int j0 = 5 * (tid >> 5), c0 = CW * (tid & 31);
    double acc[5][CW];
#pragma unroll
    for (int jj = 0; jj < 5; ++jj)
#pragma unroll
        for (int cc = 0; cc < CW; ++cc) acc[jj][cc] = 0.0;
    for (int i = 0; i < k; ++i) {
        double w[CW];
        if constexpr (CW == 4) {
            const float4 v = *reinterpret_cast<const float4 *>(&W[piv[i]][c0]);
            w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
        } else {
            const float2 v = *reinterpret_cast<const float2 *>(&W[piv[i]][c0]);
            w[0] = v.x; w[1] = v.y;
        }
#pragma unroll
        for (int jj = 0; jj < 5; ++jj) {
            const int j = j0 + jj;
            if (j >= i) {
                const double r = Ri[i][j];
#pragma unroll
                for (int cc = 0; cc < CW; ++cc) acc[jj][cc] += r * w[cc];
            }
        }
    }
    __syncthreads();
#pragma unroll
    for (int jj = 0; jj < 5; ++jj) {
        const int j = j0 + jj;
#pragma unroll
        for (int cc = 0; cc < CW; ++cc) W[j][c0 + cc] = j < k ? float(acc[jj][cc]) : 0.0f;
    }
}
__device__ inline void apply_rinv_t(float (*W)[128 + 4], const double (*Ri)[KL + 1], const int *piv, int k, int d,
                                    int tid) {
    if (d == 128) apply_rinv_t_cw<4>(W, Ri, piv, k, tid);
    else apply_rinv_t_cw<2>(W, Ri, piv, k, tid);
}

// Phase marks of the diagnostic trace (builds with SEKV_PHASE_TRACE): slot 0 holds the
// span length, then one s_memrealtime stamp per mark, for the first trace_items items.
enum : int {
    kSvStart = 1, kSvPass = 2, kSvChol = 3, kSvForward = 4, kSvGram = 5, kSvIter = 6,
    kSvPass2 = 7, kSvChol2 = 8, kSvForward2 = 9, kSvGram2 = 10, kSvJacobi = 11, kSvVrows = 12,
    kSvT = 13, kSvEnd = 14,
};
#ifdef SEKV_PHASE_TRACE
#define SV_STAMP(SLOT)                                                                         \
    do {                                                                                       \
        if (tid == 0 && a.trace && item_ < a.trace_items)                                      \
            a.trace[item_ * kTraceSlots + (SLOT)] = int64_t(__builtin_amdgcn_s_memrealtime()); \
    } while (0)
#else
#define SV_STAMP(SLOT) do {} while (0)
#endif

__global__ void __launch_bounds__(BT, 2) svd_kernel(BuildArgs a) {
    __shared__ SvdSmem sm;
    const int tid = threadIdx.x;
#ifdef SEKV_PHASE_TRACE
    const int64_t item_ = int64_t(blockIdx.y) * gridDim.x + blockIdx.x;
#endif
    const int side = blockIdx.y;                              // 0 keys, 1 values
    const int pair = blockIdx.x / a.M_max, S = blockIdx.x % a.M_max;
    const int b = pair / a.Hkv;
    const int d = a.d, e = a.elem, R = a.R;
    int ns = a.n_spans[b];
    ns = ns < 0 ? 0 : min(ns, min(a.M_max, a.N));
    if (S >= ns) return;
    const int s0 = a.span_start[size_t(b) * a.N + S];
    const int L = a.span_len_seg[size_t(b) * a.N + S];
    if (s0 < 0 || L < 1 || s0 + L > seq_tokens(a, b)) return;   // flagged by the gather kernel
    const int gran = 16 / e;
    const int r = min(min(L, d), R);                        // rank kept (eq. key_svd)
    const int rs = (r + gran - 1) / gran * gran;            // stored rank
    const int l = max(2, min(a.l, d) & ~1);                 // sketch width (even, for pairing)
    const void *src = side == 0 ? a.keys : a.values;
    const size_t row0 = size_t(pair) * a.N + s0;
    // block layout: U_K | sigma_K | Vt_K | U_V | sigma_V | Vt_V, both sides of rank rs
    const int64_t boff = a.block_off[size_t(pair) * a.M_max + S];
    const int64_t side_elems = int64_t(L + 1 + d) * rs;
    const int64_t need = 2 * side_elems * e;
    if (boff < 0 || (boff & 15) || boff + need > a.factors_bytes) {
        if (tid == 0) __hip_atomic_fetch_or(a.error, kErrBlockRange, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
    }
    unsigned char *blk = static_cast<unsigned char *>(a.factors) + boff + (side ? side_elems * e : 0);
    const int64_t s_off = int64_t(L) * rs, v_off = s_off + rs;    // in elements; U at 0
#ifdef SEKV_PHASE_TRACE
    if (tid == 0 && a.trace && item_ < a.trace_items) a.trace[item_ * kTraceSlots] = L;
#endif
    SV_STAMP(kSvStart);

    auto bf16_bits = [](float f) -> uint32_t {
        uint32_t q = __float_as_uint(f);
        q += 0x7FFFu + ((q >> 16) & 1u);                      // round to nearest even
        return q >> 16;
    };
    // the caller's test matrix into om (bfloat16, transposed)
    for (int idx = tid; idx < l * d; idx += BT) {
        const int j = idx / d, c = idx % d;
        sm.u.p.om[j][c] = uint16_t(bf16_bits(a.omega[size_t(c) * a.l + j]));
    }
    // the X rows of tile [t0, t0 + nt) as this thread's 16-byte pieces (rows past nt zero);
    // fetched one tile ahead, so that a tile's loads are in flight while the one before is used
    constexpr int NQ = 2;                                    // pieces per thread (f32, d = 128)
    auto tile_fetch = [&](int t0, int nt, uint4 (&q)[NQ]) __attribute__((always_inline)) {
        const int per = 16 / e;                              // elements per 16-byte load
#pragma unroll
        for (int u = 0; u < NQ; ++u) {
            const int i = tid + BT * u;
            const int t = i / (d / per), c = (i % (d / per)) * per;
            q[u] = make_uint4(0u, 0u, 0u, 0u);
            if (i < kTile * d / per && t < nt)
                q[u] = *reinterpret_cast<const uint4 *>(
                    static_cast<const unsigned char *>(src) + ((row0 + t0 + t) * d + c) * e);
        }
    };
    // one fetched tile of X rows into LDS (float32), and its sketch rows
    auto tile = [&](const uint4 (&q)[NQ], const int *cmap) __attribute__((always_inline)) {
        const int per = 16 / e;
#pragma unroll
        for (int u = 0; u < NQ; ++u) {
            const int i = tid + BT * u;
            if (i < kTile * d / per) {
                const int t = i / (d / per), c = (i % (d / per)) * per;
                const uint32_t w[4] = {q[u].x, q[u].y, q[u].z, q[u].w};
                float *xr = &sm.u.p.x[t][c];
                if (e == 2) {
#pragma unroll
                    for (int h = 0; h < 4; ++h) {
                        xr[2 * h] = __uint_as_float(w[h] << 16);
                        xr[2 * h + 1] = __uint_as_float(w[h] & 0xFFFF0000u);
                    }
                } else {
#pragma unroll
                    for (int h = 0; h < 4; ++h) xr[h] = __uint_as_float(w[h]);
                }
            }
        }
        __syncthreads();
        {   // Y rows: thread (t, jb) forms Y[t][jb], Y[t][jb + 16], Y[t][jb + 32], summing
            // over c in order, four columns per LDS read; rows of om past l are read but
            // their sums dropped
            const int t = tid >> 4, jb = tid & 15;
            const float4 *xr = reinterpret_cast<const float4 *>(sm.u.p.x[t]);
            const uint2 *o0 = reinterpret_cast<const uint2 *>(sm.u.p.om[jb]);
            const uint2 *o1 = reinterpret_cast<const uint2 *>(sm.u.p.om[jb + 16]);
            const uint2 *o2 = reinterpret_cast<const uint2 *>(sm.u.p.om[min(jb + 32, KL - 1)]);
            auto lo = [](uint32_t w) { return __uint_as_float(w << 16); };
            auto hi = [](uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); };
            float a0 = 0.0f, a1 = 0.0f, a2 = 0.0f;
#pragma unroll 4
            for (int c4 = 0; c4 < d / 4; ++c4) {
                const float4 xv = xr[c4];
                const uint2 w0 = o0[c4], w1 = o1[c4], w2 = o2[c4];
                a0 += xv.x * lo(w0.x); a1 += xv.x * lo(w1.x); a2 += xv.x * lo(w2.x);
                a0 += xv.y * hi(w0.x); a1 += xv.y * hi(w1.x); a2 += xv.y * hi(w2.x);
                a0 += xv.z * lo(w0.y); a1 += xv.z * lo(w1.y); a2 += xv.z * lo(w2.y);
                a0 += xv.w * hi(w0.y); a1 += xv.w * hi(w1.y); a2 += xv.w * hi(w2.y);
            }
            // column j of Y goes to column cmap[j] of yt (the identity without a map)
            if (jb < l) sm.u.p.yt[t][cmap ? cmap[jb] : jb] = a0;
            if (jb + 16 < l) sm.u.p.yt[t][cmap ? cmap[jb + 16] : jb + 16] = a1;
            if (jb + 32 < l) sm.u.p.yt[t][cmap ? cmap[jb + 32] : jb + 32] = a2;
        }
        __syncthreads();
    };
    // a pass over X with the test matrix in om: G = Y^T Y (float64 sums) into am and
    // P = Y^T X (float32 sums) into bm, accumulated in registers token by token.  Thread
    // tid owns the 5 x CW block of P at rows 5 (tid / 32), columns CW (tid % 32) (CW = d / 32)
    // and, for tid < 200, the 2 x 4 block of G at rows 2 (tid / 10), columns 4 (tid % 10);
    // sums over blocks past l are dropped.
    auto sketch_pass = [&](auto cw_c) __attribute__((always_inline)) {
        constexpr int CW = decltype(cw_c)::value;
        constexpr int GI = KL / 2, GJ = KL / 4;               // G blocks: GI x GJ of 2 x 4
        const int j0 = 5 * (tid >> 5), c0 = CW * (tid & 31);
        const bool gown = tid < GI * GJ;
        const int i0 = 2 * (tid / GJ), jj0 = 4 * (tid % GJ);
        float pacc[5][CW];
        double gacc[2][4];
#pragma unroll
        for (int jj = 0; jj < 5; ++jj)
#pragma unroll
            for (int cc = 0; cc < CW; ++cc) pacc[jj][cc] = 0.0f;
#pragma unroll
        for (int a2 = 0; a2 < 2; ++a2)
#pragma unroll
            for (int b4 = 0; b4 < 4; ++b4) gacc[a2][b4] = 0.0;
        __syncthreads();
        uint4 qn[NQ];
        tile_fetch(0, min(kTile, L), qn);
        for (int t0 = 0; t0 < L; t0 += kTile) {
            const int nt = min(kTile, L - t0);
            uint4 q[NQ];
#pragma unroll
            for (int u = 0; u < NQ; ++u) q[u] = qn[u];
            if (t0 + kTile < L) tile_fetch(t0 + kTile, min(kTile, L - t0 - kTile), qn);
            tile(q, nullptr);
            for (int t = 0; t < nt; ++t) {
                float xv[CW];
                if constexpr (CW == 4) {
                    const float4 v = *reinterpret_cast<const float4 *>(&sm.u.p.x[t][c0]);
                    xv[0] = v.x; xv[1] = v.y; xv[2] = v.z; xv[3] = v.w;
                } else {
                    const float2 v = *reinterpret_cast<const float2 *>(&sm.u.p.x[t][c0]);
                    xv[0] = v.x; xv[1] = v.y;
                }
                float yv[5];
#pragma unroll
                for (int jj = 0; jj < 5; ++jj) yv[jj] = sm.u.p.yt[t][j0 + jj];
#pragma unroll
                for (int jj = 0; jj < 5; ++jj)
#pragma unroll
                    for (int cc = 0; cc < CW; ++cc) pacc[jj][cc] += yv[jj] * xv[cc];
                if (gown) {
                    const float2 yi = *reinterpret_cast<const float2 *>(&sm.u.p.yt[t][i0]);
                    const float4 yj = *reinterpret_cast<const float4 *>(&sm.u.p.yt[t][jj0]);
                    const double di[2] = {double(yi.x), double(yi.y)};
                    const double dj[4] = {double(yj.x), double(yj.y), double(yj.z), double(yj.w)};
#pragma unroll
                    for (int a2 = 0; a2 < 2; ++a2)
#pragma unroll
                        for (int b4 = 0; b4 < 4; ++b4) gacc[a2][b4] += di[a2] * dj[b4];
                }
            }
            __syncthreads();
        }
#pragma unroll
        for (int jj = 0; jj < 5; ++jj)
#pragma unroll
            for (int cc = 0; cc < CW; ++cc)
                if (j0 + jj < l) sm.bm[j0 + jj][c0 + cc] = pacc[jj][cc];
        if (gown)
#pragma unroll
            for (int a2 = 0; a2 < 2; ++a2)
#pragma unroll
                for (int b4 = 0; b4 < 4; ++b4)
                    if (i0 + a2 < l && jj0 + b4 < l) sm.am[i0 + a2][jj0 + b4] = gacc[a2][b4];
        __syncthreads();
    };
    auto sketch = [&]() __attribute__((always_inline)) {
        if (d == 128) sketch_pass(Cint<4>{});
        else sketch_pass(Cint<2>{});
    };
    // after a pass: G = R^T R (pivoted) into rg, B = R^-T P[piv] over P, B B^T into am;
    // rg then holds R^-1 (pivot order)
    auto factor_b = [&](int it) __attribute__((always_inline)) -> int {
        const int kk = piv_chol(sm.am, sm.u.s.rg, sm.piv, sm, l, 1e-8, tid);
        SV_STAMP(it == 0 ? kSvChol : kSvChol2);
        tri_inverse(sm.u.s.rg, sm.piv, sm.am, sm.u.s.rg, kk, tid);
        apply_rinv_t(sm.bm, sm.u.s.rg, sm.piv, kk, d, tid);
        __syncthreads();
        SV_STAMP(it == 0 ? kSvForward : kSvForward2);
        {   // B B^T (rows >= kk of B are zero): thread tid < 200 forms the 2 x 4 block at
            // rows 2 (tid / 10), columns 4 (tid % 10), each entry summed over c in order
            constexpr int GJ = KL / 4;
            if (tid < (KL / 2) * GJ) {
                const int i0 = 2 * (tid / GJ), jj0 = 4 * (tid % GJ);
                double acc[2][4];
#pragma unroll
                for (int a2 = 0; a2 < 2; ++a2)
#pragma unroll
                    for (int b4 = 0; b4 < 4; ++b4) acc[a2][b4] = 0.0;
                const int ilim = min(2, max(0, kk - i0)), jlim = min(4, max(0, kk - jj0));
                if (ilim > 0 && jlim > 0) {
                    for (int c = 0; c < d; c += 4) {
                        float4 vi[2], vj[4];
#pragma unroll
                        for (int a2 = 0; a2 < 2; ++a2)
                            vi[a2] = *reinterpret_cast<const float4 *>(&sm.bm[i0 + a2][c]);
#pragma unroll
                        for (int b4 = 0; b4 < 4; ++b4)
                            vj[b4] = *reinterpret_cast<const float4 *>(&sm.bm[jj0 + b4][c]);
#pragma unroll
                        for (int a2 = 0; a2 < 2; ++a2)
#pragma unroll
                            for (int b4 = 0; b4 < 4; ++b4) {
                                acc[a2][b4] += double(vi[a2].x) * double(vj[b4].x);
                                acc[a2][b4] += double(vi[a2].y) * double(vj[b4].y);
                                acc[a2][b4] += double(vi[a2].z) * double(vj[b4].z);
                                acc[a2][b4] += double(vi[a2].w) * double(vj[b4].w);
                            }
                    }
                }
#pragma unroll
                for (int a2 = 0; a2 < 2; ++a2)
#pragma unroll
                    for (int b4 = 0; b4 < 4; ++b4) {
                        const int i = i0 + a2, j = jj0 + b4;
                        if (i < l && j < l) sm.am[i][j] = (a2 < ilim && b4 < jlim) ? acc[a2][b4] : 0.0;
                    }
            }
        }
        __syncthreads();
        SV_STAMP(it == 0 ? kSvGram : kSvGram2);
        return kk;
    };

    // subspace iterations: the next test matrix is an orthonormal basis of B's row space,
    // R2^-T B[piv2] from the pivoted Cholesky B B^T = R2^T R2, written into om
    // a span of at most l tokens is spanned by its sketch already (X Omega has the rank of X
    // for a generic Omega): an iteration would change nothing but the rounding
    const int power = L <= l ? 0 : a.power;
    for (int it = 0; it < power; ++it) {
        sketch();
        SV_STAMP(kSvPass);
        factor_b(0);
        const int k2 = piv_chol(sm.am, sm.u.s.em, sm.piv2, sm, l, 1e-8, tid);
        tri_inverse(sm.u.s.em, sm.piv2, sm.am, sm.u.s.em, k2, tid);
        apply_rinv_t(sm.bm, sm.u.s.em, sm.piv2, k2, d, tid);
        __syncthreads();
        for (int idx = tid; idx < l * d; idx += BT) {
            const int j = idx / d, c = idx % d;
            sm.u.p.om[j][c] = uint16_t(bf16_bits(sm.bm[j][c]));
        }
        SV_STAMP(kSvIter);
    }
    // the last pass; its test matrix is kept in registers (bfloat16 pairs) for the U pass
    constexpr int NO = (KL * 128 / BT + 1) / 2;
    uint32_t omk[NO];
    __syncthreads();
#pragma unroll
    for (int u = 0; u < NO; ++u) {
        uint32_t w = 0;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int idx = tid + BT * (2 * u + h);
            const int j = idx / d, c = idx % d;
            if (j < l) w |= uint32_t(sm.u.p.om[j][c]) << (16 * h);
        }
        omk[u] = w;
    }
    sketch();
    SV_STAMP(kSvPass2);
    const int k = factor_b(1);
    // B B^T = E diag(sigma^2) E^T; order (descending, ties to the lower index); components
    // below 1e-10 of the largest eigenvalue are numerically undetermined: zero
    jacobi(sm.am, sm.u.s.em, sm, l, a.sweeps, tid);
    SV_STAMP(kSvJacobi);
    if (tid < l) {
        const double me = sm.am[tid][tid];
        int rank = 0;
        for (int j = 0; j < l; ++j) {
            const double o = sm.am[j][j];
            rank += (o > me || (o == me && j < tid)) ? 1 : 0;
        }
        sm.order[rank] = tid;
    }
    __syncthreads();
    if (tid < KL) {
        double sg = 0.0;
        if (tid < l && tid < k) {
            const double lam = sm.am[sm.order[tid]][sm.order[tid]];
            const double top = sm.am[sm.order[0]][sm.order[0]];
            sg = (lam > 0.0 && lam > 1e-10 * top) ? sqrt(lam) : 0.0;
        }
        sm.sig[tid] = sg;
    }
    __syncthreads();
    if (tid < rs) st_elem(blk, size_t(s_off) + tid, tid < r ? float(sm.sig[tid]) : 0.0f, e);
    // V^T rows (E_i^T B) / sigma_i for the kept components, zero rows after
    for (int idx = tid; idx < rs * d; idx += BT) {
        const int i = idx / d, c = idx % d;
        double v = 0.0;
        if (i < r && sm.sig[i] > 0.0) {
            const int ci = sm.order[i];
            for (int j = 0; j < k; ++j) v += sm.u.s.em[j][ci] * double(sm.bm[j][c]);
            v /= sm.sig[i];
        }
        st_elem(blk, size_t(v_off) + size_t(i) * d + c, float(v), e);
    }
    __syncthreads();
    SV_STAMP(kSvVrows);
    // T = R^-1 E_r = Ri E_r (Ri upper triangular, in rg), over the Jacobi matrix
    for (int idx = tid; idx < KL * KL; idx += BT) {
        const int j = idx / KL, i = idx % KL;
        double v = 0.0;
        if (j < k && i < r && sm.sig[i] > 0.0) {
            const int ci = sm.order[i];
            for (int m = j; m < k; ++m) v += sm.u.s.rg[j][m] * sm.u.s.em[m][ci];
        }
        sm.am[j][i] = v;
    }
    __syncthreads();
    SV_STAMP(kSvT);
    // the U pass writes Y's columns in pivot order: column piv[j] to j (j < k), the other
    // columns after them
    if (tid == 0) {
        int nxt = k;
        for (int m = 0; m < l; ++m) sm.pos[m] = -1;
        for (int j = 0; j < k; ++j) sm.pos[sm.piv[j]] = j;
        for (int m = 0; m < l; ++m)
            if (sm.pos[m] < 0) sm.pos[m] = nxt++;
    }
    // last pass over X: U rows = Y[:, piv] T with the kept test matrix
#pragma unroll
    for (int u = 0; u < NO; ++u) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int idx = tid + BT * (2 * u + h);
            const int j = idx / d, c = idx % d;
            if (j < l) sm.u.p.om[j][c] = uint16_t(omk[u] >> (16 * h));
        }
    }
    __syncthreads();
    uint4 qn[NQ];
    tile_fetch(0, min(kTile, L), qn);
    for (int t0 = 0; t0 < L; t0 += kTile) {
        const int nt = min(kTile, L - t0);
        uint4 q[NQ];
#pragma unroll
        for (int u = 0; u < NQ; ++u) q[u] = qn[u];
        if (t0 + kTile < L) tile_fetch(t0 + kTile, min(kTile, L - t0 - kTile), qn);
        tile(q, sm.pos);
        {   // thread (t, ig) forms U[t][ig + 16 o], o < 3, summing over j in order; yt holds
            // Y's columns in pivot order, four per LDS read
            const int t = tid >> 4, ig = tid & 15;
            if (t < nt) {
                double v[3] = {0.0, 0.0, 0.0};
                const float *yr = sm.u.p.yt[t];
                int j = 0;
                for (; j + 4 <= k; j += 4) {
                    const float4 y4 = *reinterpret_cast<const float4 *>(yr + j);
                    const float yy[4] = {y4.x, y4.y, y4.z, y4.w};
#pragma unroll
                    for (int jj = 0; jj < 4; ++jj)
#pragma unroll
                        for (int o = 0; o < 3; ++o)
                            if (ig + 16 * o < r) v[o] += double(yy[jj]) * sm.am[j + jj][ig + 16 * o];
                }
                for (; j < k; ++j) {
                    const float y = yr[j];
#pragma unroll
                    for (int o = 0; o < 3; ++o)
                        if (ig + 16 * o < r) v[o] += double(y) * sm.am[j][ig + 16 * o];
                }
#pragma unroll
                for (int o = 0; o < 3; ++o) {
                    const int i = ig + 16 * o;
                    if (i < rs) st_elem(blk, size_t(t0 + t) * rs + i, i < r ? float(v[o]) : 0.0f, e);
                }
            }
        }
        __syncthreads();
    }
    SV_STAMP(kSvEnd);
}

}  // namespace

hipError_t launch_segment(const SegArgs &a, int batch, hipStream_t stream) {
    if (batch <= 0) return hipSuccess;
    hipLaunchKernelGGL(segment_kernel, dim3(unsigned(batch)), dim3(kSegThreads), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_build(const BuildArgs &a, int batch, hipStream_t stream) {
    if (batch <= 0) return hipSuccess;
    if (a.d > 128 || a.l > kMaxL || a.l < 2 || a.R > kMaxL) return hipErrorInvalidValue;
    const unsigned pairs = unsigned(batch * a.Hkv);
    const int rows = max(max((a.A_max + 63) / 64, a.M_max), 1);
    hipLaunchKernelGGL(gather_kernel, dim3(pairs * unsigned(rows)), dim3(BT), 0, stream, a, rows);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess || a.M_max == 0) return err;
    hipLaunchKernelGGL(svd_kernel, dim3(pairs * unsigned(a.M_max), 2), dim3(BT), 0, stream, a);
    return hipGetLastError();
}

}  // namespace sekv
