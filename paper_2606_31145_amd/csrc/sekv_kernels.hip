// SeKV decode step for gfx950: one persistent kernel over typed work items.
//
// Work items (per (sequence b, KV head g) "pair"):
//   route   chunk of 64 spans: routing scores in float64 (eq. routing_gate with the
//           coarse mean key as summary), the chunk's local top-k as sorted candidates,
//           and -- fused mode -- the coarse softmax partial of its non-candidate spans,
//           so each summary row (k_bar, v_bar) is read from HBM once.
//   anchor  chunk of full-resolution tokens: softmax partial.
//   zoom    selection slot j of a pair: once every route chunk of the pair is done, the
//           item ranks the pair's candidates (Sec. 3.3 budget rule: decreasing routing
//           score, here top-k), takes the j-th span, and attends to its tokens through
//           the factors, K_hat = U diag(sigma) V^T (eq. key_reconstruction), never
//           forming K_hat in memory.  The same partial also covers every k-th losing
//           candidate's coarse entry, so no span is dropped from the softmax.
// Every partial (max, sum, weighted value sum) lands in a fixed slot; the item that
// completes a pair's last slot merges them in slot order into the output (one softmax
// over the mixed-resolution memory, Sec. 3.3).  No floating-point atomics: results are
// bitwise deterministic.
//
// Data movement: an item issues its global loads up front, as 16-byte vectors mapped
// (row, column) onto the workgroup -- a wave reads 1 KB of contiguous rows per
// instruction -- and keeps them in registers; row sums are lane shuffles inside a row
// plus one cross-wave pass through LDS.
//
// Cross-workgroup protocol: data another workgroup reads (candidates, partials,
// selection records) is stored with agent-scope relaxed atomic stores -- write-through
// to the device coherence point on this chip -- every wave then waits for its stores to
// complete (s_waitcnt vmcnt(0)), the workgroup synchronises, and one thread bumps the
// pair's counter with a relaxed agent-scope atomic.  Readers use agent-scope relaxed
// atomic loads, issued only after they have observed the counter.  This orders exactly
// the data that is shared without writing back or invalidating whole L2 caches.
//
// Scheduling: workgroup w takes items w, w + grid, w + 2 grid, ... with grid no larger
// than the number of workgroups the device holds at once.  Route items have the lowest
// indices and never wait, so every route item a zoom item waits for is reached by its
// workgroup after finitely many non-waiting items: the waits always end (they are
// bounded anyway and flag the workspace on timeout).  The last workgroup to leave zeroes
// the counters, so the workspace is ready for the next launch.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sekv_internal.h"

namespace sekv {
namespace {

constexpr int NT = kThreads;
constexpr int CR = kRouteChunk;
constexpr float kLog2e = 1.4426950408889634f;
constexpr double kLog2eD = 1.4426950408889634074;
constexpr uint32_t kSpinLimit = 1u << 22;
constexpr uint32_t kInvalidIdx = 0xFFFFFFFFu;

// ---------------------------------------------------------------------------
// storage types: 16-byte vectors of bf16 (8 values) or f32 (4 values)
// ---------------------------------------------------------------------------
struct BF16 {
    static constexpr int kBytes = 2;
    static constexpr int kVec = 8;
    __device__ static inline void unpack(const uint4 &v, float *f) {
        f[0] = __uint_as_float(v.x << 16); f[1] = __uint_as_float(v.x & 0xFFFF0000u);
        f[2] = __uint_as_float(v.y << 16); f[3] = __uint_as_float(v.y & 0xFFFF0000u);
        f[4] = __uint_as_float(v.z << 16); f[5] = __uint_as_float(v.z & 0xFFFF0000u);
        f[6] = __uint_as_float(v.w << 16); f[7] = __uint_as_float(v.w & 0xFFFF0000u);
    }
    __device__ static inline float load1(const void *base, size_t i) {
        const uint16_t u = reinterpret_cast<const uint16_t *>(base)[i];
        return __uint_as_float(uint32_t(u) << 16);
    }
};

struct F32 {
    static constexpr int kBytes = 4;
    static constexpr int kVec = 4;
    __device__ static inline void unpack(const uint4 &v, float *f) {
        f[0] = __uint_as_float(v.x); f[1] = __uint_as_float(v.y);
        f[2] = __uint_as_float(v.z); f[3] = __uint_as_float(v.w);
    }
    __device__ static inline float load1(const void *base, size_t i) {
        return reinterpret_cast<const float *>(base)[i];
    }
};

// Row geometry of a d-row (one key/value/summary row) for a storage type.
template <class T, int D>
struct Geo {
    static constexpr int VEC = T::kVec;             // values per 16-byte vector
    static constexpr int RV = D * T::kBytes / 16;   // vectors per row: 8, 16 or 32
    static constexpr int RPP = NT / RV;             // rows per workgroup pass
    static constexpr int RB = D * T::kBytes;        // bytes per row
    static constexpr int RS = RB + 16;              // padded LDS row stride
};

__device__ inline uint4 ld16(const void *p) { return *reinterpret_cast<const uint4 *>(p); }

__device__ inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

// Order-preserving map of a finite double to uint64 (-0.0 folded onto +0.0).
__device__ inline uint64_t order_key(double x) {
    uint64_t u = uint64_t(__double_as_longlong(x));
    if (u == 0x8000000000000000ull) u = 0;
    return (u & 0x8000000000000000ull) ? ~u : (u | 0x8000000000000000ull);
}

// (key, idx) a precedes b: larger key first, then lower index.
__device__ inline bool better(uint64_t ka, uint32_t ia, uint64_t kb, uint32_t ib) {
    return ka > kb || (ka == kb && ia < ib);
}

__device__ inline float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}
__device__ inline float safe_exp2(float x) { return x == -INFINITY ? 0.0f : exp2f(x); }

// ---------------------------------------------------------------------------
// cross-workgroup protocol (see the file comment)
// ---------------------------------------------------------------------------
template <class V>
__device__ inline void st_shared(V *p, V v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <class V>
__device__ inline V ld_shared(const V *p) {
    return __hip_atomic_load(const_cast<V *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline uint32_t counter_add(uint32_t *p, uint32_t v) {
    return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Every wave waits for its own stores to complete; then the workgroup synchronises.
__device__ inline void stores_done_barrier() {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
}
__device__ inline void flag_error(const Params &p, int32_t bit) {
    __hip_atomic_fetch_or(&p.hdr->error, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// shared memory
// ---------------------------------------------------------------------------
template <class T, int D, int G>
struct Smem {
    using GE = Geo<T, D>;
    static constexpr int CA = 8 * NT / GE::RV;           // anchor tokens per item
    struct Route {                                       // route / summary item
        double qd[G][D];                                 // query, float64
        unsigned char kb[CR * GE::RS];                   // summary key rows (fp64 dots)
        double lns[CR];                                  // ln|S| of the chunk's spans
        double lg[G][CR];                                // routing scores, natural units
        float pw[G][CR];                                 // coarse weights
        int32_t excl[CR];                                // 1 = candidate / selected
    };
    struct Anchor {
        float qf[G][D];
        float sc[G][CA];                                 // scores, then weights
    };
    struct Zoom {
        float qf[G][D];
        uint4 cand[kMergeBuf];                           // {key lo, key hi, span, rank}
        float cand_lg[kMergeBuf][G];                     // candidates' natural-unit scores
        int32_t sel[kMaxTopK];                           // the pair's selection
        int32_t loser[kLoserWin];                        // this item's losing candidates
        float lw[G][kLoserWin];                          // their base-2 logits, then weights
        float w[G][kMaxTopK];                            // scale*log2e*sigma_K*(Vt_K q)
        float zs[G][kZoomBlock];                         // token scores, then weights
        float yr[4][G][kMaxTopK];                        // per-wave partial sums of p^T U_V
        float y[G][kMaxTopK];                            // (p^T U_V) * sigma_V
        float sig[2][kMaxTopK];                          // sigma_K, sigma_V
    };
    struct Merge {                                       // single-merger selection
        uint64_t key[kMergeBuf];
        uint32_t idx[kMergeBuf];
        int32_t sel[kMaxTopK];
        int32_t loser[kLoserWin];
        float pw[G][kLoserWin];
    };
    struct Final {                                       // softmax merge
        float ml[kMergeBuf][G][2];
        float wgt[kMergeBuf][G];
        float L[G];
    };
    union {
        Route route;
        Anchor anchor;
        Zoom zoom;
        Merge merge;
        Final fin;
    } u;
    float red[4][G][D];                                  // per-wave row sums
    float m_run[G], l_run[G], scale_old[G];              // online softmax state
    int32_t bcast[8];
};

// ---------------------------------------------------------------------------
// row-sum helpers: thread (rgrp = tid / RV, col = tid % RV) holds acc[G][VEC]
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__device__ inline void acc_zero(float (&acc)[G][T::kVec]) {
#pragma unroll
    for (int hl = 0; hl < G; ++hl)
#pragma unroll
        for (int e = 0; e < T::kVec; ++e) acc[hl][e] = 0.0f;
}

template <class T, int D, int G>
__device__ inline void acc_scale(float (&acc)[G][T::kVec], const float *so) {
#pragma unroll
    for (int hl = 0; hl < G; ++hl) {
        const float s = so[hl];
#pragma unroll
        for (int e = 0; e < T::kVec; ++e) acc[hl][e] *= s;
    }
}

// acc += w[row] * row vector (rows of this thread: rgrp + RPP*j, j < NJ, row < nrows)
template <class T, int D, int G, int NJ>
__device__ inline void acc_rows(float (&acc)[G][T::kVec], const uint4 (&v)[NJ],
                                const float *w, int wstride, int nrows, int rgrp) {
    using GE = Geo<T, D>;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int row = rgrp + GE::RPP * j;
        if (row < nrows) {
            float f[GE::VEC];
            T::unpack(v[j], f);
#pragma unroll
            for (int hl = 0; hl < G; ++hl) {
                const float wt = w[hl * wstride + row];
#pragma unroll
                for (int e = 0; e < GE::VEC; ++e) acc[hl][e] += wt * f[e];
            }
        }
    }
}

// Sum acc over the rows held by all threads into sm.red (caller syncs before reading).
template <class T, int D, int G>
__device__ inline void rows_to_red(Smem<T, D, G> &sm, float (&acc)[G][T::kVec], int tid) {
    using GE = Geo<T, D>;
    const int lane = tid & 63, wave = tid >> 6;
#pragma unroll
    for (int o = GE::RV; o < 64; o <<= 1)
#pragma unroll
        for (int hl = 0; hl < G; ++hl)
#pragma unroll
            for (int e = 0; e < GE::VEC; ++e) acc[hl][e] += __shfl_xor(acc[hl][e], o, 64);
    if (lane < (GE::RV < 64 ? GE::RV : 64)) {
        const int col = tid % GE::RV;
#pragma unroll
        for (int hl = 0; hl < G; ++hl)
#pragma unroll
            for (int e = 0; e < GE::VEC; ++e) sm.red[wave][hl][col * GE::VEC + e] = acc[hl][e];
    }
}

// Write the partial of `slot`: m, l from the online state; o = the 4 wave rows of red.
template <class T, int D, int G>
__device__ inline void write_partial(const Params &p, Smem<T, D, G> &sm, int pair, int slot,
                                     int tid) {
    const size_t base = (size_t(pair) * p.n_slots + slot) * G;
    if (tid < G) {
        st_shared(&p.part_ml[(base + tid) * 2 + 0], sm.m_run[tid]);
        st_shared(&p.part_ml[(base + tid) * 2 + 1], sm.l_run[tid]);
    }
    for (int o = tid; o < G * D; o += NT) {
        const int hl = o / D, d = o % D;
        st_shared(&p.part_o[base * D + o],
                  sm.red[0][hl][d] + sm.red[1][hl][d] + sm.red[2][hl][d] + sm.red[3][hl][d]);
    }
}

// Fold a batch of base-2 scores (LDS, -inf = excluded) into the online state: weights
// are written in place relative to the new running max; scale_old gets the factor the
// already accumulated sums must be multiplied by.
__device__ inline void online_fold(float *sc, int stride, int n, int G, float *m_run,
                                   float *l_run, float *scale_old, int tid) {
    const int wave = tid >> 6, lane = tid & 63;
    for (int hl = wave; hl < G; hl += 4) {
        float *row = sc + hl * stride;
        float mx = -INFINITY;
        for (int i = lane; i < n; i += 64) mx = fmaxf(mx, row[i]);
        mx = wave_max(mx);
        const float mo = m_run[hl];
        const float mn = fmaxf(mo, mx);
        float ls = 0.0f;
        for (int i = lane; i < n; i += 64) {
            const float w = (mn == -INFINITY) ? 0.0f : safe_exp2(row[i] - mn);
            row[i] = w;
            ls += w;
        }
        ls = wave_sum(ls);
        if (lane == 0) {
            const float so = (mn == -INFINITY) ? 1.0f : safe_exp2(mo - mn);
            scale_old[hl] = so;
            l_run[hl] = l_run[hl] * so + ls;
            m_run[hl] = mn;
        }
    }
}

__device__ inline void online_reset(int G, float *m_run, float *l_run, float *scale_old, int tid) {
    if (tid < G) { m_run[tid] = -INFINITY; l_run[tid] = 0.0f; scale_old[tid] = 1.0f; }
}

// ---------------------------------------------------------------------------
// final softmax merge of one pair (slot order fixed => deterministic)
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__device__ void final_merge(const Params &p, Smem<T, D, G> &sm, int pair, int tid) {
    auto &F = sm.u.fin;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    const int ns = p.n_slots;
    const bool use_losers = (p.mode == kModeFused) && p.merger;
    const float *ml = p.part_ml + size_t(pair) * ns * G * 2;
    for (int i = tid; i < ns * G * 2; i += NT) (&F.ml[0][0][0])[i] = ld_shared(ml + i);
    __syncthreads();
    const int wave = tid >> 6, lane = tid & 63;
    for (int hl = wave; hl < G; hl += 4) {
        float mx = -INFINITY;
        for (int s = lane; s < ns; s += 64) {
            const bool on = use_losers || s != p.slot_losers;
            if (on && F.ml[s][hl][1] > 0.0f) mx = fmaxf(mx, F.ml[s][hl][0]);
        }
        mx = wave_max(mx);
        float lsum = 0.0f;
        for (int s = lane; s < ns; s += 64) {
            const bool on = use_losers || s != p.slot_losers;
            float wgt = 0.0f;
            if (on && F.ml[s][hl][1] > 0.0f) {
                wgt = exp2f(F.ml[s][hl][0] - mx);
                lsum += wgt * F.ml[s][hl][1];
            }
            F.wgt[s][hl] = wgt;
        }
        lsum = wave_sum(lsum);
        if (lane == 0) F.L[hl] = lsum;
    }
    __syncthreads();
    const float *po = p.part_o + size_t(pair) * ns * G * D;
    for (int o = tid; o < G * D; o += NT) {
        const int hl = o / D, d = o % D;
        float a = 0.0f;
        int s = 0;
        for (; s + 8 <= ns; s += 8) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = ld_shared(po + (size_t(s + u) * G + hl) * D + d);
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const float wgt = F.wgt[s + u][hl];
                a += (wgt != 0.0f) ? wgt * v[u] : 0.0f;
            }
        }
        for (; s < ns; ++s) {
            const float wgt = F.wgt[s][hl];
            const float v = ld_shared(po + (size_t(s) * G + hl) * D + d);
            a += (wgt != 0.0f) ? wgt * v : 0.0f;
        }
        const float L = F.L[hl];
        const float r = (L > 0.0f) ? a / L : 0.0f;
        const size_t oi = (size_t(b) * p.Hq + size_t(g) * G + hl) * D + d;
        if (p.out_f32) reinterpret_cast<float *>(p.out)[oi] = r;
        else reinterpret_cast<uint16_t *>(p.out)[oi] = f32_to_bf16_rne(r);
    }
}

__device__ inline int parts_per_pair(const Params &p) {
    int n = p.n_ac + p.n_rc + p.k;
    if (p.mode == kModeFused && p.merger) n += 1;
    return n;
}

// Count `n` finished partials of `pair` (written, stores completed by every wave); the
// item completing the pair merges.
template <class T, int D, int G>
__device__ inline void count_partials(const Params &p, Smem<T, D, G> &sm, int pair, uint32_t n,
                                      int tid) {
    if (tid == 0) {
        const uint32_t prev = counter_add(&p.part_cnt[pair], n);
        sm.bcast[0] = (prev + n == uint32_t(parts_per_pair(p)));
    }
    __syncthreads();
    if (sm.bcast[0]) final_merge<T, D, G>(p, sm, pair, tid);
    __syncthreads();
}

// ---------------------------------------------------------------------------
// selection by a single merger (route mode, or more candidates than kMergeBuf)
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__device__ void merge_selection(const Params &p, Smem<T, D, G> &sm, int pair, int tid) {
    auto &M = sm.u.merge;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    const int k = p.k, kc = p.kc;
    int m_b = p.n_spans[b];
    m_b = m_b < 0 ? 0 : (m_b > p.M_max ? p.M_max : m_b);
    const int n_cand = p.n_rc * kc;
    constexpr int kHead = kMaxTopK;
    constexpr int kFill = kMergeBuf - kMaxTopK;
    for (int j = tid; j < kMaxTopK; j += NT) M.sel[j] = -1;
    for (int i = tid; i < kMergeBuf; i += NT) { M.key[i] = 0; M.idx[i] = kInvalidIdx - i; }
    __syncthreads();
    for (int base = 0; base < n_cand; base += kFill) {
        for (int i = tid; i < kFill; i += NT) {
            const int c = base + i;
            uint64_t key = 0;
            uint32_t idx = kInvalidIdx - (kHead + i);
            if (c < n_cand) {
                const int chunk = c / kc, j = c % kc;
                if (j < ld_shared(&p.cand_cnt[pair * p.n_rc + chunk])) {
                    const size_t ci = (size_t(pair) * p.n_rc + chunk) * kc + j;
                    key = ld_shared(&p.cand_key[ci]);
                    idx = uint32_t(ld_shared(&p.cand_idx[ci]));
                }
            }
            M.key[kHead + i] = key;
            M.idx[kHead + i] = idx;
        }
        __syncthreads();
        for (int size = 2; size <= kMergeBuf; size <<= 1) {
            for (int stride = size >> 1; stride > 0; stride >>= 1) {
                for (int t = tid; t < kMergeBuf / 2; t += NT) {
                    const int i = (t / stride) * 2 * stride + (t % stride);
                    const int j = i + stride;
                    const bool up = (i & size) == 0;
                    const uint64_t ki = M.key[i], kj = M.key[j];
                    const uint32_t ii = M.idx[i], ij = M.idx[j];
                    const bool swap = up ? better(kj, ij, ki, ii) : better(ki, ii, kj, ij);
                    if (swap) { M.key[i] = kj; M.idx[i] = ij; M.key[j] = ki; M.idx[j] = ii; }
                }
                __syncthreads();
            }
        }
        for (int i = tid; i < kHead; i += NT)
            if (i >= k) { M.key[i] = 0; M.idx[i] = kInvalidIdx - i; }
        __syncthreads();
    }
    const int take = k < m_b ? k : m_b;
    for (int j = tid; j < take; j += NT)
        if (M.idx[j] < 0x80000000u) M.sel[j] = int32_t(M.idx[j]);
    __syncthreads();
    for (int j = tid; j < k; j += NT) {
        const int s = M.sel[j];
        if (p.sel_out) p.sel_out[size_t(pair) * k + j] = s;
        if (p.mode == kModeFused) {
            int L = 0;
            int64_t off = 0;
            if (s >= 0) {
                L = p.span_len[size_t(b) * p.M_max + s];
                off = p.block_off[(size_t(b) * p.Hkv + g) * p.M_max + s];
            }
            int32_t *rec = reinterpret_cast<int32_t *>(&p.zrec[size_t(pair) * k + j]);
            st_shared(rec + 0, s);
            st_shared(rec + 1, L);
            st_shared(rec + 2, int32_t(off & 0xFFFFFFFF));
            st_shared(rec + 3, int32_t(off >> 32));
        }
    }
    stores_done_barrier();
    if (p.mode == kModeFused && tid == 0) st_shared(&p.sel_ready[pair], 1u);
}

// Coarse partial over the candidates that lost (single-merger fused mode).
template <class T, int D, int G>
__device__ void losers_partial(const Params &p, Smem<T, D, G> &sm, int pair, int tid) {
    using GE = Geo<T, D>;
    auto &M = sm.u.merge;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    const int k = p.k, kc = p.kc;
    const int rgrp = tid / GE::RV, col = tid % GE::RV;
    constexpr int NJ = (kLoserWin + GE::RPP - 1) / GE::RPP;
    const unsigned char *sv = reinterpret_cast<const unsigned char *>(p.sum_v) +
                              (size_t(b) * p.Hkv + g) * size_t(p.M_max) * GE::RB;
    const int n_cand = p.n_rc * kc;
    float acc[G][GE::VEC];
    acc_zero<T, D, G>(acc);
    online_reset(G, sm.m_run, sm.l_run, sm.scale_old, tid);
    for (int base = 0; base < n_cand; base += kLoserWin) {
        for (int t = tid; t < kLoserWin; t += NT) {
            const int c = base + t;
            int idx = -1;
            size_t ci = 0;
            if (c < n_cand) {
                const int chunk = c / kc, j = c % kc;
                if (j < ld_shared(&p.cand_cnt[pair * p.n_rc + chunk])) {
                    ci = (size_t(pair) * p.n_rc + chunk) * kc + j;
                    idx = ld_shared(&p.cand_idx[ci]);
                    for (int q = 0; q < k; ++q) idx = (M.sel[q] == idx) ? -1 : idx;
                }
            }
            M.loser[t] = idx;
            for (int hl = 0; hl < G; ++hl)
                M.pw[hl][t] = (idx >= 0) ? ld_shared(&p.cand_lg[ci * G + hl]) * kLog2e : -INFINITY;
        }
        __syncthreads();
        uint4 v[NJ];
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int row = rgrp + GE::RPP * j;
            v[j] = make_uint4(0, 0, 0, 0);
            if (row < kLoserWin && M.loser[row] >= 0)
                v[j] = ld16(sv + size_t(M.loser[row]) * GE::RB + col * 16);
        }
        online_fold(&M.pw[0][0], kLoserWin, kLoserWin, G, sm.m_run, sm.l_run, sm.scale_old, tid);
        __syncthreads();
        acc_scale<T, D, G>(acc, sm.scale_old);
        acc_rows<T, D, G, NJ>(acc, v, &M.pw[0][0], kLoserWin, kLoserWin, rgrp);
        __syncthreads();
    }
    rows_to_red<T, D, G>(sm, acc, tid);
    __syncthreads();
    write_partial<T, D, G>(p, sm, pair, p.slot_losers, tid);
}

// ---------------------------------------------------------------------------
// route / summary item: one chunk of CR spans of a pair
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__device__ void route_item(const Params &p, Smem<T, D, G> &sm, int pair, int chunk, int tid) {
    using GE = Geo<T, D>;
    auto &R = sm.u.route;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    int m_b = p.n_spans[b];
    m_b = m_b < 0 ? 0 : (m_b > p.M_max ? p.M_max : m_b);
    const int s0 = chunk * CR;
    const int nv = max(0, min(CR, m_b - s0));
    const bool attend = (p.mode == kModeAttend);
    const bool need_coarse = (p.mode != kModeRoute);
    const bool have_logits = attend && p.logits_in != nullptr;
    const bool need_dots = !have_logits;
    const size_t row0 = (size_t(b) * p.Hkv + g) * size_t(p.M_max) + s0;
    const int rgrp = tid / GE::RV, col = tid % GE::RV;
    constexpr int NJ = (CR + GE::RPP - 1) / GE::RPP;

    // 1. issue every load: summary values (registers), summary keys (-> LDS), query, ln|S|
    uint4 v[NJ];
    if (need_coarse) {
        const unsigned char *src = reinterpret_cast<const unsigned char *>(p.sum_v) + row0 * GE::RB;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int row = rgrp + GE::RPP * j;
            if (row < nv) v[j] = ld16(src + size_t(row) * GE::RB + col * 16);
        }
    }
    if (need_dots) {
        const unsigned char *src = reinterpret_cast<const unsigned char *>(p.sum_k) + row0 * GE::RB;
        uint4 kv[NJ];
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int row = rgrp + GE::RPP * j;
            if (row < nv) kv[j] = ld16(src + size_t(row) * GE::RB + col * 16);
        }
        for (int i = tid; i < G * D; i += NT) {
            const int hl = i / D, d = i % D;
            R.qd[hl][d] = double(T::load1(p.q, (size_t(b) * p.Hq + size_t(g) * G + hl) * D + d));
        }
        if (tid < nv) R.lns[tid] = p.span_logsize[size_t(b) * p.M_max + s0 + tid];
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int row = rgrp + GE::RPP * j;
            if (row < nv) *reinterpret_cast<uint4 *>(R.kb + size_t(row) * GE::RS + col * 16) = kv[j];
        }
    }
    __syncthreads();

    // 2. routing scores: float64, products exact, summed left to right over d,
    //    then (s * scale) + ln|S| as two separately rounded operations.
    for (int t = tid; t < G * CR; t += NT) {
        const int hl = t / CR, i = t % CR;
        double sc = -INFINITY;
        if (i < nv) {
            if (need_dots) {
                const unsigned char *row = R.kb + size_t(i) * GE::RS;
                double acc = 0.0;
#pragma unroll 4
                for (int c = 0; c < GE::RV; ++c) {
                    float f[GE::VEC];
                    T::unpack(*reinterpret_cast<const uint4 *>(row + c * 16), f);
#pragma unroll
                    for (int e = 0; e < GE::VEC; ++e)
                        acc = __builtin_fma(R.qd[hl][c * GE::VEC + e], double(f[e]), acc);
                }
                {
#pragma clang fp contract(off)
                    const double scaled = acc * p.scale;
                    sc = scaled + R.lns[i];
                }
            } else {
                sc = double(p.logits_in[(size_t(b) * p.Hq + size_t(g) * G + hl) * p.M_max + s0 + i]);
            }
        }
        R.lg[hl][i] = sc;
        if (p.logits_out && s0 + i < p.M_max)
            p.logits_out[(size_t(b) * p.Hq + size_t(g) * G + hl) * p.M_max + s0 + i] = float(sc);
    }
    __syncthreads();

    // 3. exclusions: local top-k candidates, sorted (route/fused), or the given selection
    if (!attend) {
        if (tid < 64) {
            // one wave sorts the chunk's 64 (key, idx) pairs with a bitonic network
            const int i = tid;
            uint64_t key = 0;
            uint32_t idx = kInvalidIdx - uint32_t(i);
            if (i < nv) {
                double x = R.lg[0][i];
                for (int hl = 1; hl < G; ++hl) x = fmax(x, R.lg[hl][i]);
                key = order_key(x);
                idx = uint32_t(s0 + i);
            }
            for (int size = 2; size <= 64; size <<= 1) {
                for (int stride = size >> 1; stride > 0; stride >>= 1) {
                    const uint32_t klo = __shfl_xor(uint32_t(key), stride, 64);
                    const uint32_t khi = __shfl_xor(uint32_t(key >> 32), stride, 64);
                    const uint32_t oi = __shfl_xor(idx, stride, 64);
                    const uint64_t ok = (uint64_t(khi) << 32) | klo;
                    const bool lower = (i & stride) == 0;
                    const bool up = (i & size) == 0;
                    const bool take = (lower == up) ? better(ok, oi, key, idx) : better(key, idx, ok, oi);
                    if (take) { key = ok; idx = oi; }
                }
            }
            // lane j now holds the j-th best
            const int kc = min(p.kc, nv);
            R.excl[i] = 0;
            __builtin_amdgcn_wave_barrier();
            if (i < kc) {
                const size_t ci = (size_t(pair) * p.n_rc + chunk) * p.kc + i;
                st_shared(&p.cand_key[ci], key);
                st_shared(&p.cand_idx[ci], int32_t(idx));
                const int li = int(idx) - s0;
                for (int hl = 0; hl < G; ++hl) st_shared(&p.cand_lg[ci * G + hl], float(R.lg[hl][li]));
                R.excl[li] = 1;
            }
            if (i == 0) st_shared(&p.cand_cnt[pair * p.n_rc + chunk], kc);
        }
    } else if (tid < CR) {
        int ex = 0;
        for (int j = 0; j < p.k; ++j) ex |= (p.sel_in[size_t(pair) * p.k + j] == s0 + tid);
        R.excl[tid] = ex;
    }
    __syncthreads();

    // 4. coarse partial over the chunk's remaining spans (values already in registers)
    if (need_coarse) {
        for (int t = tid; t < G * CR; t += NT) {
            const int hl = t / CR, i = t % CR;
            R.pw[hl][i] = (i < nv && !R.excl[i]) ? float(R.lg[hl][i] * kLog2eD) : -INFINITY;
        }
        online_reset(G, sm.m_run, sm.l_run, sm.scale_old, tid);
        __syncthreads();
        online_fold(&R.pw[0][0], CR, CR, G, sm.m_run, sm.l_run, sm.scale_old, tid);
        __syncthreads();
        float acc[G][GE::VEC];
        acc_zero<T, D, G>(acc);
        acc_rows<T, D, G, NJ>(acc, v, &R.pw[0][0], CR, nv, rgrp);
        rows_to_red<T, D, G>(sm, acc, tid);
        __syncthreads();
        write_partial<T, D, G>(p, sm, pair, p.slot_route0 + chunk, tid);
    }

    // 5. publish (candidates and partial complete), then count
    stores_done_barrier();
    if (tid == 0) {
        sm.bcast[1] = 0;
        if (!attend) {
            const uint32_t prev = counter_add(&p.route_cnt[pair], 1u);
            sm.bcast[1] = p.merger && (prev == uint32_t(p.n_rc - 1));
        }
    }
    __syncthreads();
    uint32_t n_done = need_coarse ? 1u : 0u;
    if (sm.bcast[1]) {
        merge_selection<T, D, G>(p, sm, pair, tid);
        __syncthreads();
        if (p.mode == kModeFused) {
            losers_partial<T, D, G>(p, sm, pair, tid);
            stores_done_barrier();
            n_done += 1;
        }
    }
    if (n_done) count_partials<T, D, G>(p, sm, pair, n_done, tid);
}

// ---------------------------------------------------------------------------
// anchor item: CA full-resolution tokens of a pair
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__device__ void anchor_item(const Params &p, Smem<T, D, G> &sm, int pair, int chunk, int tid) {
    using GE = Geo<T, D>;
    constexpr int CA = Smem<T, D, G>::CA;
    constexpr int NJ = CA / GE::RPP;                     // 8
    auto &A = sm.u.anchor;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    int An = p.n_anchors[b];
    An = An < 0 ? 0 : (An > p.A_max ? p.A_max : An);
    const int a0 = chunk * CA;
    const int na = max(0, min(CA, An - a0));
    const int rgrp = tid / GE::RV, col = tid % GE::RV;
    const size_t base = ((size_t(b) * p.Hkv + g) * size_t(p.A_max) + a0) * GE::RB;
    const unsigned char *ak = reinterpret_cast<const unsigned char *>(p.anchor_k) + base;
    const unsigned char *av = reinterpret_cast<const unsigned char *>(p.anchor_v) + base;
    uint4 kv[NJ], vv[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int row = rgrp + GE::RPP * j;
        if (row < na) {
            kv[j] = ld16(ak + size_t(row) * GE::RB + col * 16);
            vv[j] = ld16(av + size_t(row) * GE::RB + col * 16);
        }
    }
    for (int i = tid; i < G * D; i += NT) {
        const int hl = i / D, d = i % D;
        A.qf[hl][d] = T::load1(p.q, (size_t(b) * p.Hq + size_t(g) * G + hl) * D + d);
    }
    online_reset(G, sm.m_run, sm.l_run, sm.scale_old, tid);
    __syncthreads();
    // scores: partial dots over this thread's VEC columns, summed across the row's lanes
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int row = rgrp + GE::RPP * j;
        float part[G];
#pragma unroll
        for (int hl = 0; hl < G; ++hl) part[hl] = 0.0f;
        if (row < na) {
            float f[GE::VEC];
            T::unpack(kv[j], f);
#pragma unroll
            for (int hl = 0; hl < G; ++hl)
#pragma unroll
                for (int e = 0; e < GE::VEC; ++e) part[hl] += A.qf[hl][col * GE::VEC + e] * f[e];
        }
#pragma unroll
        for (int o = 1; o < GE::RV; o <<= 1)
#pragma unroll
            for (int hl = 0; hl < G; ++hl) part[hl] += __shfl_xor(part[hl], o, 64);
        if (col == 0)
#pragma unroll
            for (int hl = 0; hl < G; ++hl)
                A.sc[hl][row] = (row < na) ? part[hl] * p.scale_log2 : -INFINITY;
    }
    __syncthreads();
    online_fold(&A.sc[0][0], CA, CA, G, sm.m_run, sm.l_run, sm.scale_old, tid);
    __syncthreads();
    float acc[G][GE::VEC];
    acc_zero<T, D, G>(acc);
    acc_rows<T, D, G, NJ>(acc, vv, &A.sc[0][0], CA, na, rgrp);
    rows_to_red<T, D, G>(sm, acc, tid);
    __syncthreads();
    write_partial<T, D, G>(p, sm, pair, chunk, tid);
    stores_done_barrier();
    count_partials<T, D, G>(p, sm, pair, 1u, tid);
}

// ---------------------------------------------------------------------------
// zoom item, fused per-item selection: rank the pair's candidates (LDS)
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__device__ void rank_candidates(const Params &p, Smem<T, D, G> &sm, int pair, int j, int m_b,
                                int tid, int &n_loser) {
    auto &Z = sm.u.zoom;
    const int k = p.k, kc = p.kc;
    const int n_cand = p.n_rc * kc;
    for (int c = tid; c < kMergeBuf; c += NT) {
        uint4 e = make_uint4(0, 0, kInvalidIdx - uint32_t(c), 0);
        if (c < n_cand) {
            const int chunk = c / kc, jj = c % kc;
            if (jj < ld_shared(&p.cand_cnt[pair * p.n_rc + chunk])) {
                const size_t ci = (size_t(pair) * p.n_rc + chunk) * kc + jj;
                const uint64_t key = ld_shared(&p.cand_key[ci]);
                e = make_uint4(uint32_t(key), uint32_t(key >> 32), uint32_t(ld_shared(&p.cand_idx[ci])), 0);
#pragma unroll
                for (int hl = 0; hl < G; ++hl) Z.cand_lg[c][hl] = ld_shared(&p.cand_lg[ci * G + hl]);
            }
        }
        Z.cand[c] = e;
    }
    if (tid < kMaxTopK) Z.sel[tid] = -1;
    if (tid == 0) sm.bcast[3] = 0;
    __syncthreads();
    // rank = number of candidates ahead in (key desc, span asc); reads stay independent
    int n_valid_local = 0;
    for (int c = tid; c < n_cand; c += NT) {
        const uint4 me = Z.cand[c];
        if (me.z >= 0x80000000u) continue;
        ++n_valid_local;
        const uint64_t mk = (uint64_t(me.y) << 32) | me.x;
        int rank = 0;
        int o = 0;
        for (; o + 8 <= n_cand; o += 8) {
            uint4 e[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) e[u] = Z.cand[o + u];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                rank += better((uint64_t(e[u].y) << 32) | e[u].x, e[u].z, mk, me.z) ? 1 : 0;
        }
        for (; o < n_cand; ++o) {
            const uint4 e = Z.cand[o];
            rank += better((uint64_t(e.y) << 32) | e.x, e.z, mk, me.z) ? 1 : 0;
        }
        Z.cand[c].w = uint32_t(rank);
        if (rank < k && rank < m_b) Z.sel[rank] = int32_t(me.z);
    }
    // number of valid candidates (wave sums, then LDS)
    int nvl = n_valid_local;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) nvl += __shfl_xor(nvl, o, 64);
    if ((tid & 63) == 0) atomicAdd(&sm.bcast[3], nvl);
    __syncthreads();
    // losing candidates of this item: ranks k + j, 2k + j, ...  (deterministic slots)
    const int n_valid = sm.bcast[3];
    const int n_lose_all = max(0, n_valid - k);
    n_loser = (n_lose_all > j) ? (n_lose_all - j + k - 1) / k : 0;
    for (int c = tid; c < n_cand; c += NT) {
        const uint4 me = Z.cand[c];
        if (me.z >= 0x80000000u) continue;
        const int rank = int(me.w);
        if (rank >= k && ((rank - k) % k) == j) {
            const int slot = (rank - k) / k;
            if (slot < kLoserWin) {
                Z.loser[slot] = int32_t(me.z);
#pragma unroll
                for (int hl = 0; hl < G; ++hl) Z.lw[hl][slot] = Z.cand_lg[c][hl] * kLog2e;
            }
        }
    }
    __syncthreads();
}

// ---------------------------------------------------------------------------
// zoom item: one selection slot of a pair, attended through the span's factors
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__device__ void zoom_item(const Params &p, Smem<T, D, G> &sm, int pair, int j, int tid) {
    using GE = Geo<T, D>;
    auto &Z = sm.u.zoom;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    const int r = p.r;
    int m_b = p.n_spans[b];
    m_b = m_b < 0 ? 0 : (m_b > p.M_max ? p.M_max : m_b);
    const bool per_item_select = (p.mode == kModeFused) && !p.merger;
    const int rgrp = tid / GE::RV, col = tid % GE::RV;
    // the query does not depend on the selection: stage it first
    for (int i = tid; i < G * D; i += NT) {
        const int hl = i / D, d = i % D;
        Z.qf[hl][d] = T::load1(p.q, (size_t(b) * p.Hq + size_t(g) * G + hl) * D + d);
    }
    online_reset(G, sm.m_run, sm.l_run, sm.scale_old, tid);
    // wait for the pair's routing (fused mode)
    if (tid == 0) {
        bool ok = true;
        if (p.mode == kModeFused) {
            uint32_t n = 0;
            const uint32_t *flag = per_item_select ? &p.route_cnt[pair] : &p.sel_ready[pair];
            const uint32_t target = per_item_select ? uint32_t(p.n_rc) : 1u;
            while (ld_shared(flag) < target) {
                __builtin_amdgcn_s_sleep(1);
                if (++n > kSpinLimit) { flag_error(p, kErrSpinTimeout); ok = false; break; }
            }
        }
        sm.bcast[2] = ok;
    }
    __syncthreads();
    int n_loser = 0;
    int S = -1;
    if (sm.bcast[2]) {
        if (per_item_select) {
            rank_candidates<T, D, G>(p, sm, pair, j, m_b, tid, n_loser);
            S = Z.sel[j];
            if (tid == 0 && p.sel_out) p.sel_out[size_t(pair) * p.k + j] = S;
        } else if (p.mode == kModeFused) {
            const int32_t *rec = reinterpret_cast<const int32_t *>(&p.zrec[size_t(pair) * p.k + j]);
            S = ld_shared(rec);
        } else {
            S = p.sel_in[size_t(pair) * p.k + j];
        }
    }
    if (tid == 0) {
        int L = 0;
        int64_t off = 0;
        if (S >= m_b) { flag_error(p, kErrSelRange); S = -1; }
        if (S >= 0) {
            L = p.span_len[size_t(b) * p.M_max + S];
            off = p.block_off[(size_t(b) * p.Hkv + g) * p.M_max + S];
            const int64_t bytes = (2 * int64_t(L) * r + 2 * r + 2 * int64_t(r) * D) * T::kBytes;
            if (L < 1 || off < 0 || (off & 15) || off + bytes > p.factors_bytes) {
                flag_error(p, kErrBlockRange);
                S = -1;
            }
        }
        sm.bcast[4] = S;
        sm.bcast[5] = L;
        sm.bcast[6] = int32_t(off & 0xFFFFFFFF);
        sm.bcast[7] = int32_t(off >> 32);
    }
    __syncthreads();
    S = sm.bcast[4];
    const int L = sm.bcast[5];
    const int64_t off = int64_t(uint32_t(sm.bcast[6])) | (int64_t(sm.bcast[7]) << 32);
    const int slot = p.slot_zoom0 + j;
    float acc[G][GE::VEC];
    acc_zero<T, D, G>(acc);

    constexpr int VEC = GE::VEC;
    constexpr int RV = GE::RV;
    constexpr int NVT = (kMaxTopK * RV + NT - 1) / NT;   // Vt vectors per thread at r = 64
    const int RU = r * T::kBytes / 16;                  // vectors per U row
    const unsigned char *UK = p.factors + off;
    const unsigned char *sK = UK + size_t(L) * r * T::kBytes;
    const unsigned char *VtK = sK + size_t(r) * T::kBytes;
    const unsigned char *UV = VtK + size_t(r) * D * T::kBytes;
    const unsigned char *sV = UV + size_t(L) * r * T::kBytes;
    const unsigned char *VtV = sV + size_t(r) * T::kBytes;
    const int ucol = tid % RU;                          // fixed per thread (NT % RU == 0)
    int nb_max = (8 * NT) / RU;
    if (nb_max > kZoomBlock) nb_max = kZoomBlock;
    const int nb0 = min(nb_max, L);

    // issue: Vt_K, Vt_V (row i, column c) and the first token block of U_K, U_V
    uint4 vk[NVT], vvt[NVT], uk[8], uv[8];
    if (S >= 0) {
#pragma unroll
        for (int u = 0; u < NVT; ++u) {
            const int vi = tid + NT * u;
            if (vi < r * RV) {
                vk[u] = ld16(VtK + size_t(vi / RV) * GE::RB + (vi % RV) * 16);
                vvt[u] = ld16(VtV + size_t(vi / RV) * GE::RB + (vi % RV) * 16);
            }
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int tok = (tid + NT * u) / RU;
            if (tok < nb0) {
                uk[u] = ld16(UK + size_t(tok) * r * T::kBytes + ucol * 16);
                uv[u] = ld16(UV + size_t(tok) * r * T::kBytes + ucol * 16);
            }
        }
        if (tid < r) {
            Z.sig[0][tid] = T::load1(sK, tid);
            Z.sig[1][tid] = T::load1(sV, tid);
        }
    }

    // losing candidates of this item: coarse entries (v_bar rows, routing scores)
    if (n_loser > 0) {
        constexpr int NJL = (kLoserWin + GE::RPP - 1) / GE::RPP;
        const unsigned char *sv = reinterpret_cast<const unsigned char *>(p.sum_v) +
                                  (size_t(b) * p.Hkv + g) * size_t(p.M_max) * GE::RB;
        const int nl = min(n_loser, kLoserWin);
        uint4 lv[NJL];
#pragma unroll
        for (int jj = 0; jj < NJL; ++jj) {
            const int row = rgrp + GE::RPP * jj;
            if (row < nl) lv[jj] = ld16(sv + size_t(Z.loser[row]) * GE::RB + col * 16);
        }
        if (tid < G)
            for (int i = nl; i < kLoserWin; ++i) Z.lw[tid][i] = -INFINITY;
        __syncthreads();
        online_fold(&Z.lw[0][0], kLoserWin, nl, G, sm.m_run, sm.l_run, sm.scale_old, tid);
        __syncthreads();
        acc_rows<T, D, G, NJL>(acc, lv, &Z.lw[0][0], kLoserWin, nl, rgrp);
    }

    if (S >= 0) {
        __syncthreads();
        // w[h][i] = scale*log2e * sigma_K[i] * (Vt_K[i] . q_h)
#pragma unroll
        for (int u = 0; u < NVT; ++u) {
            const int vi = tid + NT * u;
            const int row = vi / RV, c = vi % RV;
            float part[G];
#pragma unroll
            for (int hl = 0; hl < G; ++hl) part[hl] = 0.0f;
            if (vi < r * RV) {
                float f[VEC];
                T::unpack(vk[u], f);
#pragma unroll
                for (int hl = 0; hl < G; ++hl)
#pragma unroll
                    for (int e = 0; e < VEC; ++e) part[hl] += Z.qf[hl][c * VEC + e] * f[e];
            }
#pragma unroll
            for (int o = 1; o < RV; o <<= 1)
#pragma unroll
                for (int hl = 0; hl < G; ++hl) part[hl] += __shfl_xor(part[hl], o, 64);
            if (vi < r * RV && c == 0)
#pragma unroll
                for (int hl = 0; hl < G; ++hl)
                    Z.w[hl][row] = part[hl] * Z.sig[0][row] * p.scale_log2;
        }
        __syncthreads();

        // token blocks: scores via U_K, online softmax, y = p^T U_V accumulated per lane
        float yacc[G][VEC];
#pragma unroll
        for (int hl = 0; hl < G; ++hl)
#pragma unroll
            for (int e = 0; e < VEC; ++e) yacc[hl][e] = 0.0f;
        const int wave = tid >> 6, lane = tid & 63;
        for (int t0 = 0; t0 < L; t0 += nb_max) {
            const int nb = min(nb_max, L - t0);
            if (t0 > 0) {
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int tok = (tid + NT * u) / RU;
                    if (tok < nb) {
                        uk[u] = ld16(UK + size_t(t0 + tok) * r * T::kBytes + ucol * 16);
                        uv[u] = ld16(UV + size_t(t0 + tok) * r * T::kBytes + ucol * 16);
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int tok = (tid + NT * u) / RU;
                float part[G];
#pragma unroll
                for (int hl = 0; hl < G; ++hl) part[hl] = 0.0f;
                if (tok < nb) {
                    float f[VEC];
                    T::unpack(uk[u], f);
#pragma unroll
                    for (int hl = 0; hl < G; ++hl)
#pragma unroll
                        for (int e = 0; e < VEC; ++e) part[hl] += f[e] * Z.w[hl][ucol * VEC + e];
                }
                for (int o = 1; o < RU; o <<= 1)
#pragma unroll
                    for (int hl = 0; hl < G; ++hl) part[hl] += __shfl_xor(part[hl], o, 64);
                if (tok < nb && ucol == 0)
#pragma unroll
                    for (int hl = 0; hl < G; ++hl) Z.zs[hl][tok] = part[hl];
            }
            __syncthreads();
            online_fold(&Z.zs[0][0], kZoomBlock, nb, G, sm.m_run, sm.l_run, sm.scale_old, tid);
            __syncthreads();
#pragma unroll
            for (int hl = 0; hl < G; ++hl) {
                const float so = sm.scale_old[hl];
#pragma unroll
                for (int e = 0; e < VEC; ++e) {
                    yacc[hl][e] *= so;
                    acc[hl][e] *= so;
                }
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int tok = (tid + NT * u) / RU;
                if (tok < nb) {
                    float f[VEC];
                    T::unpack(uv[u], f);
#pragma unroll
                    for (int hl = 0; hl < G; ++hl) {
                        const float pw = Z.zs[hl][tok];
#pragma unroll
                        for (int e = 0; e < VEC; ++e) yacc[hl][e] += pw * f[e];
                    }
                }
            }
            __syncthreads();
        }
        // y[h][i]: sum yacc over the lanes sharing ucol, then over the waves
        for (int o = RU; o < 64; o <<= 1)
#pragma unroll
            for (int hl = 0; hl < G; ++hl)
#pragma unroll
                for (int e = 0; e < VEC; ++e) yacc[hl][e] += __shfl_xor(yacc[hl][e], o, 64);
        if (lane < RU)
#pragma unroll
            for (int hl = 0; hl < G; ++hl)
#pragma unroll
                for (int e = 0; e < VEC; ++e) Z.yr[wave][hl][ucol * VEC + e] = yacc[hl][e];
        __syncthreads();
        for (int t = tid; t < G * r; t += NT) {
            const int hl = t / r, i = t % r;
            Z.y[hl][i] = (Z.yr[0][hl][i] + Z.yr[1][hl][i] + Z.yr[2][hl][i] + Z.yr[3][hl][i]) *
                         Z.sig[1][i];
        }
        __syncthreads();
        // o[h][:] += sum_i y~[h][i] Vt_V[i][:]; Vt_V rows of column c sit RV lanes apart,
        // exactly like summary rows
#pragma unroll
        for (int u = 0; u < NVT; ++u) {
            const int vi = tid + NT * u;
            if (vi < r * RV) {
                const int row = vi / RV;
                float f[VEC];
                T::unpack(vvt[u], f);
#pragma unroll
                for (int hl = 0; hl < G; ++hl) {
                    const float y = Z.y[hl][row];
#pragma unroll
                    for (int e = 0; e < VEC; ++e) acc[hl][e] += y * f[e];
                }
            }
        }
    }
    rows_to_red<T, D, G>(sm, acc, tid);
    __syncthreads();
    write_partial<T, D, G>(p, sm, pair, slot, tid);
    stores_done_barrier();
    count_partials<T, D, G>(p, sm, pair, 1u, tid);
}

// ---------------------------------------------------------------------------
// the persistent kernel
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__global__ void __launch_bounds__(NT, 2) sekv_step_kernel(Params p) {
    __shared__ Smem<T, D, G> sm;
    const int tid = threadIdx.x;
    const int n_items = p.end_zoom;
    for (int item = blockIdx.x; item < n_items; item += p.grid) {
        // an opaque copy of the thread index keeps per-thread address arithmetic inside
        // each item instead of alive across the whole loop (register pressure)
        int t;
        asm volatile("v_mov_b32 %0, %1" : "=v"(t) : "v"(tid));
        if (item < p.end_route) {
            route_item<T, D, G>(p, sm, item / p.n_rc, item % p.n_rc, t);
        } else if (item < p.end_anchor) {
            const int i = item - p.end_route;
            anchor_item<T, D, G>(p, sm, i / p.n_ac, i % p.n_ac, t);
        } else {
            const int i = item - p.end_anchor;
            zoom_item<T, D, G>(p, sm, i / p.k, i % p.k, t);
        }
        __syncthreads();
    }
    // shutdown: the last workgroup out zeroes the counters for the next launch
    if (tid == 0) {
        const uint32_t prev = counter_add(&p.hdr->exit_count, 1u);
        sm.bcast[3] = (prev == uint32_t(p.grid - 1));
    }
    __syncthreads();
    if (sm.bcast[3]) {
        const int P = p.B * p.Hkv;
        for (int i = tid; i < P; i += NT) {
            p.route_cnt[i] = 0u;
            p.sel_ready[i] = 0u;
            p.part_cnt[i] = 0u;
        }
        if (tid == 0) {
            p.hdr->ticket = 0u;
            p.hdr->exit_count = 0u;
        }
    }
}

__global__ void zero_kernel(uint4 *p, size_t n16) {
    for (size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n16;
         i += size_t(gridDim.x) * blockDim.x)
        p[i] = make_uint4(0, 0, 0, 0);
}

template <class T, int D, int G>
hipError_t launch_typed(const Params &p, hipStream_t stream) {
    hipLaunchKernelGGL((sekv_step_kernel<T, D, G>), dim3(p.grid), dim3(NT), 0, stream, p);
    return hipGetLastError();
}

template <class T, int D, int G>
int occupancy_typed() {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, sekv_step_kernel<T, D, G>, NT, 0) !=
        hipSuccess)
        return 1;
    return n > 0 ? n : 1;
}

template <class T, int D>
hipError_t launch_g(const Params &p, int group, hipStream_t s) {
    switch (group) {
        case 1: return launch_typed<T, D, 1>(p, s);
        case 2: return launch_typed<T, D, 2>(p, s);
        case 4: return launch_typed<T, D, 4>(p, s);
        case 8: return launch_typed<T, D, 8>(p, s);
    }
    return hipErrorInvalidValue;
}

template <class T, int D>
int occ_g(int group) {
    switch (group) {
        case 1: return occupancy_typed<T, D, 1>();
        case 2: return occupancy_typed<T, D, 2>();
        case 4: return occupancy_typed<T, D, 4>();
        case 8: return occupancy_typed<T, D, 8>();
    }
    return 1;
}

}  // namespace

hipError_t launch_step(const Params &p, int dtype, int head_dim, int group, hipStream_t stream) {
    if (dtype == SEKV_BF16) {
        if (head_dim == 128) return launch_g<BF16, 128>(p, group, stream);
        if (head_dim == 64) return launch_g<BF16, 64>(p, group, stream);
    } else {
        if (head_dim == 128) return launch_g<F32, 128>(p, group, stream);
        if (head_dim == 64) return launch_g<F32, 64>(p, group, stream);
    }
    return hipErrorInvalidValue;
}

int resident_workgroups(int dtype, int head_dim, int group) {
    int per_cu = 1;
    if (dtype == SEKV_BF16) per_cu = head_dim == 128 ? occ_g<BF16, 128>(group) : occ_g<BF16, 64>(group);
    else per_cu = head_dim == 128 ? occ_g<F32, 128>(group) : occ_g<F32, 64>(group);
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return per_cu;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) cus = 1;
    return per_cu * (cus > 0 ? cus : 1);
}

hipError_t launch_zero(void *ptr, size_t bytes, hipStream_t stream) {
    const size_t n16 = bytes / 16;
    if (n16 == 0) return hipSuccess;
    size_t blocks = (n16 + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(zero_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream,
                       reinterpret_cast<uint4 *>(ptr), n16);
    return hipGetLastError();
}

}  // namespace sekv
