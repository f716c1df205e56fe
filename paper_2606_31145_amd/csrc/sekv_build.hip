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
//                    r = min(|S|, d, R_max)): sketch Y = X Omega with the caller's random
//                    d x l test matrix; G = Y^T Y = W diag(lambda) W^T and the orthonormal
//                    basis Q = Y W diag(lambda^-1/2) of the sketch's range (directions with
//                    lambda below 1e-6 of the largest dropped, so a rank-deficient sketch
//                    is handled); B = Q^T X = diag(lambda^-1/2) W^T (Y^T X); B B^T =
//                    E diag(sigma^2) E^T; V^T = diag(1/sigma) E^T B and U = Q E = Y T with
//                    T = W diag(lambda^-1/2) E.  Both small eigen-decompositions are cyclic
//                    Jacobi rotations in LDS.  The factors go into the span's block of the
//                    factor arena, stored with the rank rounded up to the 16-byte granule
//                    (the extra components zero).
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "sekv_internal.h"

namespace sekv {
namespace {

constexpr int kSegThreads = 1024;
constexpr int BT = 256;                 // builder threads per workgroup
constexpr int kMaxL = 48;               // largest sketch width
constexpr int kTile = 16;               // tokens per streamed tile in the SVD

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

// grid = B * Hkv * rows workgroups; workgroup (pair, y) copies anchor rows
// [64 y, 64 y + 64) and summarises span y.
__global__ void __launch_bounds__(BT) gather_kernel(BuildArgs a, int rows) {
    const int pair = blockIdx.x / rows, b = pair / a.Hkv, g = pair % a.Hkv;
    const int y = blockIdx.x % rows, tid = threadIdx.x;
    const int d = a.d, e = a.elem;
    const size_t tok0 = size_t(pair) * a.N;                 // row of token 0 of (b, g)
    int na = a.n_anchors[b];
    na = na < 0 ? 0 : min(na, min(a.A_max, a.N));
    int ns = a.n_spans[b];
    ns = ns < 0 ? 0 : min(ns, min(a.M_max, a.N));
    // anchor rows
    for (int i = tid; i < 64 * d; i += BT) {
        const int r = y * 64 + i / d, col = i % d;
        if (r < na) {
            const int t = a.anchor_idx[size_t(b) * a.N + r];
            if (t >= 0 && t < a.N) {
                const size_t dst = (size_t(pair) * a.A_max + r) * d + col;
                st_elem(a.anchor_k, dst, ld_elem(a.keys, (tok0 + t) * d + col, e), e);
                st_elem(a.anchor_v, dst, ld_elem(a.values, (tok0 + t) * d + col, e), e);
            }
        }
    }
    // span y: surprisal-weighted means; |S| and ln|S| once per sequence (g == 0)
    if (y >= ns) return;
    const int s0 = a.span_start[size_t(b) * a.N + y];
    int L = a.span_len_seg[size_t(b) * a.N + y];
    if (s0 < 0 || L < 1 || s0 + L > a.N) return;
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

struct SvdSmem {
    union {
        struct {                              // passes over X
            float om[kMaxL][128];             // Omega^T (l x d)
            float x[kTile][128 + 1];          // token tile
            float yt[kTile][kMaxL + 1];       // sketch tile
        } p;
        struct {                              // small dense algebra (float64: the Gram
            float bm[kMaxL][128 + 1];         // matrices square the condition number)
            double am[kMaxL][kMaxL + 1];      // G, then B B^T (rotated to diagonal)
        } s;                                  // bm: Y^T X, then B
    } u;
    double wm[kMaxL][kMaxL + 1];              // eigenvectors of G, then T = W diag E
    double em[kMaxL][kMaxL + 1];              // eigenvectors of B B^T
    double cs[kMaxL / 2][2];                  // a round's rotations (c, s)
    double scale[kMaxL];                      // lambda^-1/2 of the kept directions, else 0
    double sig[kMaxL];
    int order[kMaxL];
    double lmax;
};

// Round-robin pairing of round k among n (even) indices: index n-1 stays, the others
// rotate; pair i of the round is (p, q) with p < q.  Every pair meets once per sweep.
__device__ inline void rr_pair(int n, int k, int i, int *p, int *q) {
    int a0, b0;
    if (i == 0) { a0 = n - 1; b0 = k % (n - 1); }
    else { a0 = (k + i) % (n - 1); b0 = (k - i + (n - 1)) % (n - 1); }
    *p = min(a0, b0);
    *q = max(a0, b0);
}

// Cyclic Jacobi on the symmetric n x n matrix A (n even): A is rotated towards diagonal,
// V (set to I here) accumulates the rotations, so that A_in = V diag(A_out) V^T.
__device__ void jacobi(double (*A)[kMaxL + 1], double (*V)[kMaxL + 1], double (*cs)[2], int n, int sweeps,
                       int tid) {
    for (int idx = tid; idx < n * n; idx += BT) V[idx / n][idx % n] = (idx / n == idx % n) ? 1.0 : 0.0;
    __syncthreads();
    for (int sweep = 0; sweep < sweeps; ++sweep) {
        for (int k = 0; k < n - 1; ++k) {
            if (tid < n / 2) {
                int p, q;
                rr_pair(n, k, tid, &p, &q);
                const double app = A[p][p], aqq = A[q][q], apq = A[p][q];
                double c = 1.0, s = 0.0;
                if (apq != 0.0 && fabs(apq) > 1e-300 * (fabs(app) + fabs(aqq))) {
                    const double th = (aqq - app) / (2.0 * apq);
                    const double t = (th >= 0.0 ? 1.0 : -1.0) / (fabs(th) + sqrt(1.0 + th * th));
                    c = 1.0 / sqrt(1.0 + t * t);
                    s = t * c;
                }
                cs[tid][0] = c;
                cs[tid][1] = s;
            }
            __syncthreads();
            for (int idx = tid; idx < (n / 2) * n; idx += BT) {        // rows p, q
                const int i = idx / n, col = idx % n;
                int p, q;
                rr_pair(n, k, i, &p, &q);
                const double c = cs[i][0], s = cs[i][1];
                const double xp = A[p][col], xq = A[q][col];
                A[p][col] = c * xp - s * xq;
                A[q][col] = s * xp + c * xq;
            }
            __syncthreads();
            for (int idx = tid; idx < (n / 2) * n; idx += BT) {        // columns p, q
                const int i = idx / n, row = idx % n;
                int p, q;
                rr_pair(n, k, i, &p, &q);
                const double c = cs[i][0], s = cs[i][1];
                const double xp = A[row][p], xq = A[row][q];
                A[row][p] = c * xp - s * xq;
                A[row][q] = s * xp + c * xq;
                const double vp = V[row][p], vq = V[row][q];
                V[row][p] = c * vp - s * vq;
                V[row][q] = s * vp + c * vq;
            }
            __syncthreads();
        }
    }
}

__global__ void __launch_bounds__(BT) svd_kernel(BuildArgs a) {
    __shared__ SvdSmem sm;
    const int tid = threadIdx.x;
    const int side = blockIdx.y;                              // 0 keys, 1 values
    const int pair = blockIdx.x / a.M_max, S = blockIdx.x % a.M_max;
    const int b = pair / a.Hkv;
    const int d = a.d, e = a.elem, R = a.R;
    int ns = a.n_spans[b];
    ns = ns < 0 ? 0 : min(ns, min(a.M_max, a.N));
    if (S >= ns) return;
    const int s0 = a.span_start[size_t(b) * a.N + S];
    const int L = a.span_len_seg[size_t(b) * a.N + S];
    if (s0 < 0 || L < 1 || s0 + L > a.N) return;
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

    constexpr int NP = kMaxL * 128 / BT;                     // entries of an l x d matrix per thread
    constexpr int NG = (kMaxL * kMaxL + BT - 1) / BT;
    // the test matrix, transposed (l x d), entries tid + BT u of thread tid: the caller's
    // Omega, then after each subspace iteration the right singular vectors of that pass
    float omr[NP];
#pragma unroll
    for (int u = 0; u < NP; ++u) {
        const int idx = tid + BT * u;
        const int j = idx / d, c = idx % d;
        omr[u] = j < l ? a.omega[size_t(c) * a.l + j] : 0.0f;
    }
    auto load_omega = [&]() {
#pragma unroll
        for (int u = 0; u < NP; ++u) {
            const int idx = tid + BT * u;
            const int j = idx / d, c = idx % d;
            if (j < l) sm.u.p.om[j][c] = omr[u];
        }
    };
    // one tile of X rows [t0, t0 + nt) and its sketch rows Y = X Omega
    auto tile = [&](int t0, int nt) {
        for (int i = tid; i < kTile * d; i += BT) {
            const int t = i / d, c = i % d;
            sm.u.p.x[t][c] = t < nt ? ld_elem(src, (row0 + t0 + t) * d + c, e) : 0.0f;
        }
        __syncthreads();
        for (int i = tid; i < kTile * l; i += BT) {
            const int t = i / l, j = i % l;
            float acc = 0.0f;
            for (int c = 0; c < d; ++c) acc += sm.u.p.x[t][c] * sm.u.p.om[j][c];
            sm.u.p.yt[t][j] = acc;
        }
        __syncthreads();
    };

    for (int it = 0;; ++it) {
        const bool last = it >= a.power;
        // 1. pass over X: G = Y^T Y (float64 sums) and P = Y^T X (float32), in registers
        float pacc[NP];
        double gacc[NG];
#pragma unroll
        for (int u = 0; u < NP; ++u) pacc[u] = 0.0f;
#pragma unroll
        for (int u = 0; u < NG; ++u) gacc[u] = 0.0;
        load_omega();
        __syncthreads();
        for (int t0 = 0; t0 < L; t0 += kTile) {
            const int nt = min(kTile, L - t0);
            tile(t0, nt);
#pragma unroll
            for (int u = 0; u < NP; ++u) {
                const int idx = tid + BT * u;
                const int j = idx / d, c = idx % d;
                if (j < l) {
                    float acc = pacc[u];
                    for (int t = 0; t < nt; ++t) acc += sm.u.p.yt[t][j] * sm.u.p.x[t][c];
                    pacc[u] = acc;
                }
            }
#pragma unroll
            for (int u = 0; u < NG; ++u) {
                const int idx = tid + BT * u;
                const int i = idx / kMaxL, j = idx % kMaxL;
                if (i < l && j < l) {
                    double acc = gacc[u];
                    for (int t = 0; t < nt; ++t) acc += double(sm.u.p.yt[t][i]) * double(sm.u.p.yt[t][j]);
                    gacc[u] = acc;
                }
            }
            __syncthreads();
        }
#pragma unroll
        for (int u = 0; u < NP; ++u) {
            const int idx = tid + BT * u;
            const int j = idx / d, c = idx % d;
            if (j < l) sm.u.s.bm[j][c] = pacc[u];
        }
#pragma unroll
        for (int u = 0; u < NG; ++u) {
            const int idx = tid + BT * u;
            const int i = idx / kMaxL, j = idx % kMaxL;
            if (i < l && j < l) sm.u.s.am[i][j] = gacc[u];
        }
        __syncthreads();
        // 2. G = W diag(lambda) W^T; keep directions above 1e-6 of the largest eigenvalue
        jacobi(sm.u.s.am, sm.wm, sm.cs, l, a.sweeps, tid);
        if (tid == 0) {
            double mx = 0.0;
            for (int i = 0; i < l; ++i) mx = fmax(mx, sm.u.s.am[i][i]);
            sm.lmax = mx;
        }
        __syncthreads();
        if (tid < l) {
            const double lam = sm.u.s.am[tid][tid];
            sm.scale[tid] = (lam > 1e-6 * sm.lmax && lam > 0.0) ? 1.0 / sqrt(lam) : 0.0;
        }
        __syncthreads();
        // 3. B = diag(scale) W^T P, in place of P: each column c from its own column
        for (int c = tid; c < d; c += BT) {
            float col[kMaxL];
#pragma unroll
            for (int k = 0; k < kMaxL; ++k) col[k] = k < l ? sm.u.s.bm[k][c] : 0.0f;
            for (int i = 0; i < l; ++i) {
                double v = 0.0;
#pragma unroll
                for (int k = 0; k < kMaxL; ++k)
                    if (k < l) v += sm.wm[k][i] * double(col[k]);     // rows >= l of W unset
                sm.u.s.bm[i][c] = float(sm.scale[i] * v);
            }
        }
        __syncthreads();
        // 4. B B^T = E diag(sigma^2) E^T
        for (int idx = tid; idx < l * l; idx += BT) {
            const int i = idx / l, j = idx % l;
            double acc = 0.0;
            for (int c = 0; c < d; ++c) acc += double(sm.u.s.bm[i][c]) * double(sm.u.s.bm[j][c]);
            sm.u.s.am[i][j] = acc;
        }
        __syncthreads();
        jacobi(sm.u.s.am, sm.em, sm.cs, l, a.sweeps, tid);
        // 5. order (descending, ties to the lower index), sigma; components below 1e-10 of
        //    the largest eigenvalue are numerically undetermined: zero
        if (tid < l) {
            const double me = sm.u.s.am[tid][tid];
            int rank = 0;
            for (int j = 0; j < l; ++j) {
                const double o = sm.u.s.am[j][j];
                rank += (o > me || (o == me && j < tid)) ? 1 : 0;
            }
            sm.order[rank] = tid;
        }
        __syncthreads();
        if (tid < kMaxL) {
            double sg = 0.0;
            if (tid < l) {
                const double lam = sm.u.s.am[sm.order[tid]][sm.order[tid]];
                const double top = sm.u.s.am[sm.order[0]][sm.order[0]];
                sg = (lam > 0.0 && lam > 1e-10 * top) ? sqrt(lam) : 0.0;
            }
            sm.sig[tid] = sg;
        }
        __syncthreads();
        if (last) break;
        // subspace iteration: the next test matrix is V (all l right singular vectors of
        // B = Q^T X), which spans the row space of X^T Q with orthonormal columns
#pragma unroll
        for (int u = 0; u < NP; ++u) {
            const int idx = tid + BT * u;
            const int i = idx / d, c = idx % d;
            double v = 0.0;
            if (i < l && sm.sig[i] > 0.0) {
                const int ci = sm.order[i];
                for (int k = 0; k < l; ++k) v += sm.em[k][ci] * double(sm.u.s.bm[k][c]);
                v /= sm.sig[i];
            }
            omr[u] = float(v);
        }
        __syncthreads();
    }
    if (tid < rs) st_elem(blk, size_t(s_off) + tid, tid < r ? float(sm.sig[tid]) : 0.0f, e);
    // 6. V^T rows (E_i^T B) / sigma_i for the kept components, zero rows after
    for (int idx = tid; idx < rs * d; idx += BT) {
        const int i = idx / d, c = idx % d;
        double v = 0.0;
        if (i < r && i < l && sm.sig[i] > 0.0) {
            const int ci = sm.order[i];
            for (int k = 0; k < l; ++k) v += sm.em[k][ci] * double(sm.u.s.bm[k][c]);
            v /= sm.sig[i];
        }
        st_elem(blk, size_t(v_off) + size_t(i) * d + c, float(v), e);
    }
    // 7. T = W diag(scale) E_r, row j by thread j, written over row j of W
    if (tid < l) {
        double trow[kMaxL];
#pragma unroll
        for (int i = 0; i < kMaxL; ++i) {
            double v = 0.0;
            if (i < r && i < l && sm.sig[i] > 0.0) {
                const int ci = sm.order[i];
                for (int k = 0; k < l; ++k) v += sm.wm[tid][k] * sm.scale[k] * sm.em[k][ci];
            }
            trow[i] = v;
        }
#pragma unroll
        for (int i = 0; i < kMaxL; ++i) sm.wm[tid][i] = trow[i];
    }
    __syncthreads();
    // 8. second pass over X: U rows = (X Omega) T
    load_omega();
    __syncthreads();
    for (int t0 = 0; t0 < L; t0 += kTile) {
        const int nt = min(kTile, L - t0);
        tile(t0, nt);
        for (int idx = tid; idx < nt * rs; idx += BT) {
            const int t = idx / rs, i = idx % rs;
            double v = 0.0;
            if (i < r && i < l)
                for (int j = 0; j < l; ++j) v += double(sm.u.p.yt[t][j]) * sm.wm[j][i];
            st_elem(blk, size_t(t0 + t) * rs + i, float(v), e);
        }
        __syncthreads();
    }
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
