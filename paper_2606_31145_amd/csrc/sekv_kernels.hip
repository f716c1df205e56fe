// SeKV decode step for gfx950: one persistent kernel over typed work items.
//
// Work items (per (sequence b, KV head g) "pair"):
//   route   chunk of 128 spans: routing scores in float64 (eq. routing_gate with the
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

// ---------------------------------------------------------------------------
// lane reductions without LDS: DPP row operations inside 16-lane rows and the
// gfx950 permlane swaps across rows.  With both operands equal, permlane16_swap /
// permlane32_swap return the two halves whose sum is the xor-16 / xor-32 butterfly.
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ inline float dpp_mov(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ inline uint32_t dpp_mov_u(uint32_t v) {
    return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppRor4 = 0x124;       // row_ror:4
constexpr int kDppRor8 = 0x128;       // row_ror:8  (= xor 8 inside a row)
constexpr int kDppHalfMirror = 0x141; // row_half_mirror

struct OpSum { __device__ static float f(float a, float b) { return a + b; } };
struct OpMax { __device__ static float f(float a, float b) { return fmaxf(a, b); } };

template <class Op>
__device__ inline float perm16(float v) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return Op::f(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
template <class Op>
__device__ inline float perm32(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return Op::f(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Reduce over the lanes whose index differs only in bits [LO, HI); every lane gets
// the result.  Bit 2 alone (without bits 2 and 3 together) needs bits 0 and 1 reduced.
template <int LO, int HI, class Op = OpSum>
__device__ inline float lane_reduce(float v) {
    static_assert(!(HI == 3 && LO != 0), "bit 2 alone needs bits 0-1 reduced first");
    if constexpr (LO <= 0 && 0 < HI) v = Op::f(v, dpp_mov<kDppXor1>(v));
    if constexpr (LO <= 1 && 1 < HI) v = Op::f(v, dpp_mov<kDppXor2>(v));
    if constexpr (LO <= 2 && 3 < HI) {
        v = Op::f(v, dpp_mov<kDppRor4>(v));
        v = Op::f(v, dpp_mov<kDppRor8>(v));
    } else if constexpr (LO <= 2 && 2 < HI) {
        v = Op::f(v, dpp_mov<kDppHalfMirror>(v));
    } else if constexpr (LO <= 3 && 3 < HI) {
        v = Op::f(v, dpp_mov<kDppRor8>(v));
    }
    if constexpr (LO <= 4 && 4 < HI) v = perm16<Op>(v);
    if constexpr (LO <= 5 && 5 < HI) v = perm32<Op>(v);
    return v;
}

__device__ inline float wave_max(float v) { return lane_reduce<0, 6, OpMax>(v); }
__device__ inline float wave_sum(float v) { return lane_reduce<0, 6, OpSum>(v); }

// Sum over the n lanes of an aligned group of n (n in {1,2,4,8,16}); runtime n.
__device__ inline float group_sum(float v, int n) {
    switch (n) {
        case 1: return v;
        case 2: return lane_reduce<0, 1>(v);
        case 4: return lane_reduce<0, 2>(v);
        case 8: return lane_reduce<0, 3>(v);
        default: return lane_reduce<0, 4>(v);
    }
}
// Sum over the lanes that share lane % n (n in {1,2,4,8,16}); runtime n.
__device__ inline float stride_sum(float v, int n) {
    switch (n) {
        case 1: return lane_reduce<0, 6>(v);
        case 2: return lane_reduce<1, 6>(v);
        case 4: return lane_reduce<2, 6>(v);
        case 8: return lane_reduce<3, 6>(v);
        default: return lane_reduce<4, 6>(v);
    }
}
template <int RV>
__device__ inline float row_sum(float v) {     // sum over an aligned group of RV lanes
    if constexpr (RV == 8) return lane_reduce<0, 3>(v);
    else if constexpr (RV == 16) return lane_reduce<0, 4>(v);
    else return lane_reduce<0, 5>(v);
}
template <int RV>
__device__ inline float col_sum(float v) {     // sum over the lanes sharing lane % RV
    if constexpr (RV == 8) return lane_reduce<3, 6>(v);
    else if constexpr (RV == 16) return lane_reduce<4, 6>(v);
    else return lane_reduce<5, 6>(v);
}

// Value of the lane at index ^ S (bitonic partner), 32-bit.
template <int S>
__device__ inline uint32_t lane_xor(uint32_t v, int lane) {
    if constexpr (S == 1) return dpp_mov_u<kDppXor1>(v);
    else if constexpr (S == 2) return dpp_mov_u<kDppXor2>(v);
    else if constexpr (S == 8) return dpp_mov_u<kDppRor8>(v);
    else if constexpr (S == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
        return (lane & 16) ? r[0] : r[1];
    } else if constexpr (S == 32) {
        const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
        return (lane & 32) ? r[0] : r[1];
    } else {
        return uint32_t(__shfl_xor(int(v), S, 64));
    }
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
        int32_t slen[CR];                                // |S| of the chunk's spans
        int64_t boff[CR];                                // their block offsets
        uint64_t skey[2][64];                            // two sorted halves of the chunk
        uint32_t sidx[2][64];
    };
    struct Anchor {
        float qf[G][D];
        float sc[G][CA];                                 // scores, then weights
    };
    struct Zoom {
        float qf[G][D];
        uint4 cand[kMergeBuf];                           // {key lo, key hi, span, -}
        int32_t loser[kZoomLosers];                      // this item's losing candidates
        float lw[G][kZoomLosers];                        // their base-2 logits, then weights
        float w[G][kMaxTopK];                            // scale*log2e*sigma_K*(Vt_K q)
        float zs[G][kZoomBlock];                         // token scores, then weights
        float yr[4][G][kMaxTopK];                        // per-wave partial sums of p^T U_V
        float y[G][kMaxTopK];                            // (p^T U_V) * sigma_V
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
    for (int hl = 0; hl < G; ++hl)
#pragma unroll
        for (int e = 0; e < GE::VEC; ++e) acc[hl][e] = col_sum<GE::RV>(acc[hl][e]);
    if (lane < GE::RV) {
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
__device__ __forceinline__ void final_merge(const Params &p, Smem<T, D, G> &sm, int pair, int tid) {
    auto &F = sm.u.fin;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    const int ns = p.n_slots;
    const bool use_losers = (p.mode == kModeFused) && p.merger;
    const float *ml = p.part_ml + size_t(pair) * ns * G * 2;
    const float *po = p.part_o + size_t(pair) * ns * G * D;
    constexpr int NOUT = (G * D + NT - 1) / NT;
    // every load first: the (m, l) of all slots to LDS, this thread's o values to registers
    constexpr int kBatch = 32;                          // slots whose o values are in flight
    float ov[NOUT][kBatch];
    for (int i = tid; i < ns * G * 2; i += NT) (&F.ml[0][0][0])[i] = ld_shared(ml + i);
#pragma unroll
    for (int u = 0; u < NOUT; ++u) {
        const int o = tid + NT * u;
        const int hl = o / D, d = o % D;
#pragma unroll
        for (int s = 0; s < kBatch; ++s)
            ov[u][s] = (o < G * D && s < ns) ? ld_shared(po + (size_t(s) * G + hl) * D + d) : 0.0f;
    }
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
#pragma unroll
    for (int u = 0; u < NOUT; ++u) {
        const int o = tid + NT * u;
        if (o >= G * D) continue;
        const int hl = o / D, d = o % D;
        float a = 0.0f;
#pragma unroll
        for (int s = 0; s < kBatch; ++s) {
            const float wgt = (s < ns) ? F.wgt[s][hl] : 0.0f;
            a += (wgt != 0.0f) ? wgt * ov[u][s] : 0.0f;
        }
        for (int s = kBatch; s < ns; ++s) {              // rare: more slots than the batch
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
__device__ __forceinline__ void merge_selection(const Params &p, Smem<T, D, G> &sm, int pair, int tid) {
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
__device__ __forceinline__ void losers_partial(const Params &p, Smem<T, D, G> &sm, int pair, int tid) {
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
__device__ __forceinline__ void route_item(const Params &p, Smem<T, D, G> &sm, int pair, int chunk, int tid) {
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
    const int wave = tid >> 6, lane = tid & 63;
    constexpr int NJ = (CR + GE::RPP - 1) / GE::RPP;

    // 1. issue the loads routing needs: summary keys (-> LDS), query, ln|S|, and
    //    |S| / block offsets for the candidate records
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
    if (tid < CR) {
        R.excl[tid] = 0;
        if (!attend && tid < nv) {
            R.slen[tid] = p.span_len[size_t(b) * p.M_max + s0 + tid];
            R.boff[tid] = p.block_off[row0 + tid];
        }
    }
    __syncthreads();

    // 2. routing scores: float64, products exact, summed left to right over d,
    //    then (s * scale) + ln|S| as two separately rounded operations.  Each thread
    //    runs two independent chains (same head within a wave, different spans).
    for (int c0 = tid; c0 < G * CR; c0 += 2 * NT) {
        const int c1 = c0 + NT;
        const bool has1 = c1 < G * CR;
        const int h0 = c0 / CR, i0 = c0 % CR;
        const int h1 = has1 ? c1 / CR : h0, i1 = has1 ? c1 % CR : i0;
        double sc0 = -INFINITY, sc1 = -INFINITY;
        if (need_dots) {
            const unsigned char *r0 = R.kb + size_t(i0) * GE::RS;
            const unsigned char *r1 = R.kb + size_t(i1) * GE::RS;
            double a0 = 0.0, a1 = 0.0;
#pragma unroll 2
            for (int c = 0; c < GE::RV; ++c) {
                float f0[GE::VEC], f1[GE::VEC];
                T::unpack(*reinterpret_cast<const uint4 *>(r0 + c * 16), f0);
                T::unpack(*reinterpret_cast<const uint4 *>(r1 + c * 16), f1);
#pragma unroll
                for (int e = 0; e < GE::VEC; ++e) {
                    a0 = __builtin_fma(R.qd[h0][c * GE::VEC + e], double(f0[e]), a0);
                    a1 = __builtin_fma(R.qd[h1][c * GE::VEC + e], double(f1[e]), a1);
                }
            }
            {
#pragma clang fp contract(off)
                const double m0 = a0 * p.scale;
                const double m1 = a1 * p.scale;
                if (i0 < nv) sc0 = m0 + R.lns[i0];
                if (has1 && i1 < nv) sc1 = m1 + R.lns[i1];
            }
        } else {
            const size_t lbase = (size_t(b) * p.Hq + size_t(g) * G) * p.M_max + s0;
            if (i0 < nv) sc0 = double(p.logits_in[lbase + size_t(h0) * p.M_max + i0]);
            if (has1 && i1 < nv) sc1 = double(p.logits_in[lbase + size_t(h1) * p.M_max + i1]);
        }
        R.lg[h0][i0] = sc0;
        if (has1) R.lg[h1][i1] = sc1;
        if (p.logits_out) {
            const size_t lbase = (size_t(b) * p.Hq + size_t(g) * G) * p.M_max;
            if (s0 + i0 < p.M_max) p.logits_out[lbase + size_t(h0) * p.M_max + s0 + i0] = float(sc0);
            if (has1 && s0 + i1 < p.M_max) p.logits_out[lbase + size_t(h1) * p.M_max + s0 + i1] = float(sc1);
        }
    }
    __syncthreads();

    // 3. candidates: waves 0 and 1 each sort 64 (key, span) pairs with a bitonic network;
    //    a span's rank in the chunk is its position plus the number of better entries of
    //    the other half (binary search); the best kc become the chunk's sorted candidates.
    if (!attend) {
        if (wave < 2) {
            const int i = wave * 64 + lane;
            uint64_t key = 0;
            uint32_t idx = kInvalidIdx - uint32_t(i);
            if (i < nv) {
                double x = R.lg[0][i];
                for (int hl = 1; hl < G; ++hl) x = fmax(x, R.lg[hl][i]);
                key = order_key(x);
                idx = uint32_t(s0 + i);
            }
#define SEKV_BITONIC_STEP(STRIDE)                                                          \
            {                                                                              \
                const uint32_t klo = lane_xor<STRIDE>(uint32_t(key), lane);                \
                const uint32_t khi = lane_xor<STRIDE>(uint32_t(key >> 32), lane);          \
                const uint32_t oi = lane_xor<STRIDE>(idx, lane);                           \
                const uint64_t ok = (uint64_t(khi) << 32) | klo;                           \
                const bool lower = (lane & (STRIDE)) == 0;                                 \
                const bool take = (lower == up) ? better(ok, oi, key, idx)                 \
                                                : better(key, idx, ok, oi);                \
                if (take) { key = ok; idx = oi; }                                          \
            }
#pragma unroll
            for (int size = 2; size <= 64; size <<= 1) {
                const bool up = (lane & size) == 0;
                if (size >= 64) SEKV_BITONIC_STEP(32)
                if (size >= 32) SEKV_BITONIC_STEP(16)
                if (size >= 16) SEKV_BITONIC_STEP(8)
                if (size >= 8) SEKV_BITONIC_STEP(4)
                if (size >= 4) SEKV_BITONIC_STEP(2)
                SEKV_BITONIC_STEP(1)
            }
#undef SEKV_BITONIC_STEP
            R.skey[wave][lane] = key;
            R.sidx[wave][lane] = idx;
        }
        __syncthreads();
        const int kc = min(p.kc, nv);
        if (wave < 2) {
            const uint64_t key = R.skey[wave][lane];
            const uint32_t idx = R.sidx[wave][lane];
            const int other = 1 - wave;
            int lo = 0, hi = 64;
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (better(R.skey[other][mid], R.sidx[other][mid], key, idx)) lo = mid + 1;
                else hi = mid;
            }
            const int rank = lane + lo;
            if (idx < 0x80000000u && rank < kc) {
                const int li = int(idx) - s0;
                const size_t ci = (size_t(pair) * p.n_rc + chunk) * p.kc + rank;
                st_shared(&p.cand_key[ci], key);
                st_shared(&p.cand_idx[ci], int32_t(idx));
                st_shared(&p.cand_len[ci], R.slen[li]);
                st_shared(&p.cand_off[ci], R.boff[li]);
                for (int hl = 0; hl < G; ++hl) st_shared(&p.cand_lg[ci * G + hl], float(R.lg[hl][li]));
                R.excl[li] = 1;
            }
        }
        if (tid == 0) st_shared(&p.cand_cnt[pair * p.n_rc + chunk], kc);
        // publish the candidates before the coarse partial: zoom items wait on them
        stores_done_barrier();
        if (tid == 0) {
            sm.bcast[1] = 0;
            if (p.merger) {
                const uint32_t prev = counter_add(&p.route_cnt[pair], 1u);
                sm.bcast[1] = (prev == uint32_t(p.n_rc - 1));
            } else {
                (void)counter_add(&p.route_cnt[pair], 1u);     // no return value awaited
            }
        }
        __syncthreads();
    } else {
        if (tid < CR) {
            int ex = 0;
            for (int j = 0; j < p.k; ++j) ex |= (p.sel_in[size_t(pair) * p.k + j] == s0 + tid);
            R.excl[tid] = ex;
        }
        if (tid == 0) sm.bcast[1] = 0;
        __syncthreads();
    }
    const bool merger = sm.bcast[1] != 0;

    // 4. coarse partial over the chunk's remaining spans
    uint32_t n_done = 0;
    uint4 v[NJ];
    if (need_coarse) {
        const unsigned char *src = reinterpret_cast<const unsigned char *>(p.sum_v) + row0 * GE::RB;
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int row = rgrp + GE::RPP * j;
            if (row < nv) v[j] = ld16(src + size_t(row) * GE::RB + col * 16);
        }
    }
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
        n_done = 1;
    }
    if (merger) {
        __syncthreads();
        merge_selection<T, D, G>(p, sm, pair, tid);
        __syncthreads();
        if (p.mode == kModeFused) {
            losers_partial<T, D, G>(p, sm, pair, tid);
            n_done += 1;
        }
    }
    if (n_done) {
        stores_done_barrier();
        count_partials<T, D, G>(p, sm, pair, n_done, tid);
    }
}

// ---------------------------------------------------------------------------
// anchor item: CA full-resolution tokens of a pair
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__device__ __forceinline__ void anchor_item(const Params &p, Smem<T, D, G> &sm, int pair, int chunk, int tid) {
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
        for (int hl = 0; hl < G; ++hl) part[hl] = row_sum<GE::RV>(part[hl]);
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
__device__ __forceinline__ void rank_candidates(const Params &p, Smem<T, D, G> &sm, int pair, int j, int m_b,
                                int tid, int &n_loser) {
    auto &Z = sm.u.zoom;
    const int k = p.k, kc = p.kc;
    const int n_cand = p.n_rc * kc;
    // each thread owns candidates tid and tid + NT: records stay in its registers
    constexpr int OWN = kMergeBuf / NT;
    uint64_t okey[OWN];
    uint32_t oidx[OWN];
    int32_t olen[OWN];
    int64_t ooff[OWN];
    float olg[OWN][G];
#pragma unroll
    for (int u = 0; u < OWN; ++u) {
        const int c = tid + NT * u;
        okey[u] = 0;
        oidx[u] = kInvalidIdx - uint32_t(c);
        olen[u] = 0;
        ooff[u] = 0;
        if (c < n_cand) {
            const int chunk = c / kc, jj = c % kc;
            if (jj < ld_shared(&p.cand_cnt[pair * p.n_rc + chunk])) {
                const size_t ci = (size_t(pair) * p.n_rc + chunk) * kc + jj;
                okey[u] = ld_shared(&p.cand_key[ci]);
                oidx[u] = uint32_t(ld_shared(&p.cand_idx[ci]));
                olen[u] = ld_shared(&p.cand_len[ci]);
                ooff[u] = ld_shared(&p.cand_off[ci]);
#pragma unroll
                for (int hl = 0; hl < G; ++hl) olg[u][hl] = ld_shared(&p.cand_lg[ci * G + hl]);
            }
        }
        Z.cand[c] = make_uint4(uint32_t(okey[u]), uint32_t(okey[u] >> 32), oidx[u], 0);
    }
    if (tid == 0) { sm.bcast[3] = 0; sm.bcast[4] = -1; sm.bcast[5] = 0; sm.bcast[6] = 0; sm.bcast[7] = 0; }
    __syncthreads();
    // rank = number of candidates ahead in (key desc, span asc); LDS reads batched by 8
    int rank[OWN];
    int n_valid_local = 0;
#pragma unroll
    for (int u = 0; u < OWN; ++u) {
        rank[u] = -1;
        const int c = tid + NT * u;
        if (c >= n_cand || oidx[u] >= 0x80000000u) continue;
        ++n_valid_local;
        int rk = 0;
        int o = 0;
        for (; o + 8 <= n_cand; o += 8) {
            uint4 e[8];
#pragma unroll
            for (int w = 0; w < 8; ++w) e[w] = Z.cand[o + w];
#pragma unroll
            for (int w = 0; w < 8; ++w)
                rk += better((uint64_t(e[w].y) << 32) | e[w].x, e[w].z, okey[u], oidx[u]) ? 1 : 0;
        }
        for (; o < n_cand; ++o) {
            const uint4 e = Z.cand[o];
            rk += better((uint64_t(e.y) << 32) | e.x, e.z, okey[u], oidx[u]) ? 1 : 0;
        }
        rank[u] = rk;
        if (rk == j && rk < k && rk < m_b) {        // this item's span
            sm.bcast[4] = int32_t(oidx[u]);
            sm.bcast[5] = olen[u];
            sm.bcast[6] = int32_t(ooff[u] & 0xFFFFFFFF);
            sm.bcast[7] = int32_t(ooff[u] >> 32);
        }
    }
    const float nvl = wave_sum(float(n_valid_local));
    if ((tid & 63) == 0) atomicAdd(&sm.bcast[3], int(nvl));
    __syncthreads();
    // losing candidates of this item: ranks k + j, 2k + j, ...  (deterministic slots)
    const int n_valid = sm.bcast[3];
    const int n_lose_all = max(0, n_valid - k);
    n_loser = (n_lose_all > j) ? (n_lose_all - j + k - 1) / k : 0;
#pragma unroll
    for (int u = 0; u < OWN; ++u) {
        const int rk = rank[u];
        if (rk >= k && ((rk - k) % k) == j) {
            const int slot = (rk - k) / k;
            if (slot < kZoomLosers) {
                Z.loser[slot] = int32_t(oidx[u]);
#pragma unroll
                for (int hl = 0; hl < G; ++hl) Z.lw[hl][slot] = olg[u][hl] * kLog2e;
            }
        }
    }
    __syncthreads();
}

// ---------------------------------------------------------------------------
// zoom item body for one span, RU = 16-byte vectors per factor row U[t][:]
// ---------------------------------------------------------------------------
template <class T, int D, int G, int RU>
__device__ __forceinline__ void zoom_span(const Params &p, Smem<T, D, G> &sm, int pair, int S,
                                          int L, int64_t off, int nl,
                                          float (&acc)[G][T::kVec], int tid) {
    using GE = Geo<T, D>;
    auto &Z = sm.u.zoom;
    constexpr int VEC = GE::VEC;
    constexpr int RV = GE::RV;
    constexpr int NVT = (kMaxTopK * RV + NT - 1) / NT;   // Vt vectors per thread at r = 64
    constexpr int NSV = (G * kMaxTopK + NT - 1) / NT;    // y entries per thread at r = 64
    constexpr int NB = (8 * NT / RU) < kZoomBlock ? (8 * NT / RU) : kZoomBlock;  // tokens/block
    constexpr int NU = NB * RU / NT;                     // U vectors per thread per block
    constexpr int LG_RU = RU == 1 ? 0 : RU == 2 ? 1 : RU == 4 ? 2 : RU == 8 ? 3 : 4;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    const int r = p.r;
    const int rgrp = tid / GE::RV, col = tid % GE::RV;
    const int ucol = tid % RU;
    const int wave = tid >> 6, lane = tid & 63;
    const unsigned char *UK = p.factors + off;
    const unsigned char *sK = UK + size_t(L) * r * T::kBytes;
    const unsigned char *VtK = sK + size_t(r) * T::kBytes;
    const unsigned char *UV = VtK + size_t(r) * D * T::kBytes;
    const unsigned char *sV = UV + size_t(L) * r * T::kBytes;
    const unsigned char *VtV = sV + size_t(r) * T::kBytes;
    const bool zoom = S >= 0;
    const int nb0 = min(NB, L);

    // issue in the order of use: sigmas, Vt_K, losers' value rows, U_K, then U_V.
    // Addresses are clamped into the block, validity is applied where values are used.
    float sk_reg[NVT], sv_reg[NSV];
    uint4 vk[NVT], vvt[NVT], uk[NU], uv[NU];
    constexpr int NJL = (kZoomLosers + GE::RPP - 1) / GE::RPP;
    uint4 lv[NJL];
    if (zoom) {
#pragma unroll
        for (int u = 0; u < NVT; ++u) {
            const int vi = min(tid + NT * u, r * RV - 1);
            sk_reg[u] = T::load1(sK, vi / RV);
        }
#pragma unroll
        for (int u = 0; u < NSV; ++u) sv_reg[u] = T::load1(sV, (tid + NT * u) % r);
#pragma unroll
        for (int u = 0; u < NVT; ++u) {
            const int vi = min(tid + NT * u, r * RV - 1);
            vk[u] = ld16(VtK + size_t(vi / RV) * GE::RB + (vi % RV) * 16);
        }
    }
    if (nl > 0) {
        const unsigned char *sv = reinterpret_cast<const unsigned char *>(p.sum_v) +
                                  (size_t(b) * p.Hkv + g) * size_t(p.M_max) * GE::RB;
#pragma unroll
        for (int jj = 0; jj < NJL; ++jj) {
            const int row = min(rgrp + GE::RPP * jj, nl - 1);
            lv[jj] = ld16(sv + size_t(Z.loser[row]) * GE::RB + col * 16);
        }
        if (tid < G)
            for (int i = nl; i < kZoomLosers; ++i) Z.lw[tid][i] = -INFINITY;
    }
    if (zoom) {
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            const int tok = min((tid + NT * u) / RU, nb0 - 1);
            uk[u] = ld16(UK + size_t(tok) * r * T::kBytes + ucol * 16);
        }
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            const int tok = min((tid + NT * u) / RU, nb0 - 1);
            uv[u] = ld16(UV + size_t(tok) * r * T::kBytes + ucol * 16);
        }
    }
    __syncthreads();

    if (zoom) {
        // w[h][i] = scale*log2e * sigma_K[i] * (Vt_K[i] . q_h)
#pragma unroll
        for (int u = 0; u < NVT; ++u) {
            const int vi = tid + NT * u;
            const int row = vi / RV, c = vi % RV;
            float part[G];
            float f[VEC];
            T::unpack(vk[u], f);
#pragma unroll
            for (int hl = 0; hl < G; ++hl) {
                part[hl] = 0.0f;
#pragma unroll
                for (int e = 0; e < VEC; ++e) part[hl] += Z.qf[hl][c * VEC + e] * f[e];
                part[hl] = row_sum<RV>(part[hl]);
            }
            if (vi < r * RV && c == 0)
#pragma unroll
                for (int hl = 0; hl < G; ++hl) Z.w[hl][row] = part[hl] * sk_reg[u] * p.scale_log2;
        }
        // Vt_V rows take the registers Vt_K has released
#pragma unroll
        for (int u = 0; u < NVT; ++u) {
            const int vi = min(tid + NT * u, r * RV - 1);
            vvt[u] = ld16(VtV + size_t(vi / RV) * GE::RB + (vi % RV) * 16);
        }
    }

    // this item's losing candidates: coarse entries (v_bar rows, routing scores)
    if (nl > 0) {
        online_fold(&Z.lw[0][0], kZoomLosers, nl, G, sm.m_run, sm.l_run, sm.scale_old, tid);
        __syncthreads();
        acc_rows<T, D, G, NJL>(acc, lv, &Z.lw[0][0], kZoomLosers, nl, rgrp);
    }
    if (!zoom) return;
    __syncthreads();

    // token blocks: scores via U_K, online softmax, y = p^T U_V accumulated per lane
    float yacc[G][VEC];
#pragma unroll
    for (int hl = 0; hl < G; ++hl)
#pragma unroll
        for (int e = 0; e < VEC; ++e) yacc[hl][e] = 0.0f;
    for (int t0 = 0; t0 < L; t0 += NB) {
        const int nb = min(NB, L - t0);
        if (t0 > 0) {
#pragma unroll
            for (int u = 0; u < NU; ++u) {
                const int tok = min((tid + NT * u) / RU, nb - 1);
                uk[u] = ld16(UK + size_t(t0 + tok) * r * T::kBytes + ucol * 16);
            }
#pragma unroll
            for (int u = 0; u < NU; ++u) {
                const int tok = min((tid + NT * u) / RU, nb - 1);
                uv[u] = ld16(UV + size_t(t0 + tok) * r * T::kBytes + ucol * 16);
            }
        }
#pragma unroll
        for (int u = 0; u < NU; ++u) {
            const int tok = (tid + NT * u) / RU;
            float f[VEC];
            T::unpack(uk[u], f);
            float part[G];
#pragma unroll
            for (int hl = 0; hl < G; ++hl) {
                part[hl] = 0.0f;
#pragma unroll
                for (int e = 0; e < VEC; ++e) part[hl] += f[e] * Z.w[hl][ucol * VEC + e];
                part[hl] = lane_reduce<0, LG_RU>(part[hl]);
            }
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
        for (int u = 0; u < NU; ++u) {
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
#pragma unroll
    for (int hl = 0; hl < G; ++hl)
#pragma unroll
        for (int e = 0; e < VEC; ++e) yacc[hl][e] = lane_reduce<LG_RU, 6>(yacc[hl][e]);
    if (lane < RU)
#pragma unroll
        for (int hl = 0; hl < G; ++hl)
#pragma unroll
            for (int e = 0; e < VEC; ++e) Z.yr[wave][hl][ucol * VEC + e] = yacc[hl][e];
    __syncthreads();
#pragma unroll
    for (int u = 0; u < NSV; ++u) {
        const int t = tid + NT * u;
        if (t < G * r) {
            const int hl = t / r, i = t % r;
            Z.y[hl][i] = (Z.yr[0][hl][i] + Z.yr[1][hl][i] + Z.yr[2][hl][i] + Z.yr[3][hl][i]) *
                         sv_reg[u];
        }
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

// ---------------------------------------------------------------------------
// zoom item: one selection slot of a pair, attended through the span's factors
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__device__ __forceinline__ void zoom_item(const Params &p, Smem<T, D, G> &sm, int pair, int j, int tid) {
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
    if (sm.bcast[2] && per_item_select) {
        // ranks the pair's candidates; the owner of rank j leaves {span, |S|, offset} in bcast
        rank_candidates<T, D, G>(p, sm, pair, j, m_b, tid, n_loser);
    }
    if (tid == 0) {
        int L = 0;
        int64_t off = 0;
        if (!sm.bcast[2]) {
            S = -1;
        } else if (per_item_select) {
            S = sm.bcast[4];
            L = sm.bcast[5];
            off = int64_t(uint32_t(sm.bcast[6])) | (int64_t(sm.bcast[7]) << 32);
            if (p.sel_out) p.sel_out[size_t(pair) * p.k + j] = S;
        } else {
            if (p.mode == kModeFused) {
                S = ld_shared(reinterpret_cast<const int32_t *>(&p.zrec[size_t(pair) * p.k + j]));
            } else {
                S = p.sel_in[size_t(pair) * p.k + j];
            }
            if (S >= m_b) { flag_error(p, kErrSelRange); S = -1; }
            if (S >= 0) {
                L = p.span_len[size_t(b) * p.M_max + S];
                off = p.block_off[(size_t(b) * p.Hkv + g) * p.M_max + S];
            }
        }
        if (S >= 0) {
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
    const int nl = min(n_loser, kZoomLosers);
    if (S >= 0 || nl > 0) {
        switch (r * T::kBytes / 16) {                   // 16-byte vectors per U row
            case 1: zoom_span<T, D, G, 1>(p, sm, pair, S, L, off, nl, acc, tid); break;
            case 2: zoom_span<T, D, G, 2>(p, sm, pair, S, L, off, nl, acc, tid); break;
            case 4: zoom_span<T, D, G, 4>(p, sm, pair, S, L, off, nl, acc, tid); break;
            case 8: zoom_span<T, D, G, 8>(p, sm, pair, S, L, off, nl, acc, tid); break;
            default: zoom_span<T, D, G, 16>(p, sm, pair, S, L, off, nl, acc, tid); break;
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
