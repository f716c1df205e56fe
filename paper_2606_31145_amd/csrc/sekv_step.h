// SeKV decode step for gfx950: one persistent kernel over typed work items.
//
// Work items (per (sequence b, KV head g) "pair"):
//   route   chunk of 128 spans: routing scores in float64 (eq. routing_gate with the
//           coarse mean key as summary).  It publishes every span's score (the coarse
//           logit) and, when the step selects, the chunk's local top-k as sorted
//           candidate records.  It waits for nothing.
//   share   share slot j of a pair (j < n_zi, n_zi = min(k, about 512 / pairs), at
//           least 1).  While routing runs it attends to its share of the anchor tokens;
//           then it ranks the pair's candidates (Sec. 3.3 budget rule: decreasing routing
//           score, here top-k), takes the spans of ranks j, j + n_zi, ... and attends to
//           their tokens through the factors, K_hat = U diag(sigma) V^T (eq.
//           key_reconstruction), never forming K_hat in memory; while the first factor
//           loads are in flight it folds its share of the summaries, skipping the
//           selected spans, so every span enters the softmax once: zoomed or coarse.
// Each share item leaves one partial (max, sum, weighted value sum per head) in a fixed
// slot; the item that completes a pair merges the slots in order into the output (one
// softmax over the mixed-resolution memory, Sec. 3.3).  No floating-point atomics:
// results are bitwise deterministic.
//
// Data movement: an item issues its global loads up front, as 16-byte vectors mapped
// (row, column) onto the workgroup -- a wave reads 1 KB of contiguous rows per
// instruction -- and keeps them in registers; row sums are lane shuffles inside a row
// plus one cross-wave pass through LDS.
//
// Cross-workgroup protocol.  Routing results travel as tagged words: 32 bits of payload
// and the launch's 32-bit tag in one 64-bit relaxed agent-scope atomic store
// (write-through to the device coherence point on this chip).  A reader polls them with
// relaxed agent-scope atomic loads until every tag it needs is the current launch's, so
// the writer neither waits for its stores nor bumps a counter.  The tag is the
// workspace epoch (1 after initialisation, never 0, which unwritten words hold); the last
// workgroup out advances it.  Partials (and the
// single-merger selection) use counters instead: every wave waits for its stores to
// complete (s_waitcnt vmcnt(0)), the workgroup synchronises, and one thread bumps the
// pair's counter with a relaxed agent-scope atomic; readers load the data only after
// observing the counter.  No fence writes back or invalidates whole L2 caches.
//
// Scheduling: workgroup w takes items w, w + grid, w + 2 grid, ... with grid no larger
// than the number of workgroups the device holds at once.  A routing chunk is computed
// by whichever workgroup first claims it (an atomic exchange of the launch tag into the
// chunk's claim word): its own routing item, or a share item that has polled for the
// pair's candidates kHelpAfter times and then runs every unclaimed chunk of the pair
// itself (help_route) before polling again.  A share item thus only waits for chunks
// held by running workgroups, which never wait, so every wait ends whatever the
// residency (waits are bounded anyway and flag the workspace on timeout).  The last
// workgroup to leave zeroes the counters, so the workspace is ready for the next launch.
#pragma once

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
// A waiting share item starts helping (computing routing chunks nobody has claimed) after
// this many unsuccessful polls, and again every this many polls.
constexpr uint32_t kHelpAfter = 256;
// After this many rounds of help a share item waits without giving up (bounded by
// kSpinLimit, which flags the workspace): every wait of a launch ends.
constexpr int kMaxHelps = 64;
// A share item that starts with the launch holds its first loads back by this many
// s_sleep units (64 cycles each, about 0.4 us) so that the routing items' summary-key
// loads, which the selection waits for, reach memory first.
constexpr int kShareHoldBack = 16;
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

// Phase marks of the diagnostic trace (builds with SEKV_PHASE_TRACE).  Slot 0 of an
// item holds its descriptor: kind (0 route, 1 share) << 60 | XCC id << 48 | workgroup.
enum : int {
    kTrStart = 1, kTrEnd = 2,
    // routing item
    kTrRLoaded = 3, kTrRScored = 4, kTrRSorted = 5, kTrRPublished = 6,
    // share item
    kTrSAnchors = 3, kTrSSelected = 4, kTrSZoomIssued = 5, kTrSZoomMid = 6, kTrSZoomW = 7,
    kTrSZoomTokens = 8, kTrSZoomDone = 9, kTrSCoarse = 10, kTrSPartial = 11, kTrSMerged = 12,
    kTrSPolled = 13,    // the first poll of the candidate records answered
    kTrSPolls = 14,     // a count, not a time: polls until every record was current
};
#ifdef SEKV_PHASE_TRACE
__device__ inline uint32_t xcc_id() {
    uint32_t v;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
    return v & 0xF;
}
#define SEKV_TRACE_BEGIN(P, SM, ITEM)                                                         \
    do {                                                                                      \
        if (threadIdx.x == 0) {                                                               \
            (SM).trace_item = (ITEM);                                                         \
            if ((P).trace) {                                                                  \
                int64_t *tr_ = (P).trace + size_t(ITEM) * kTraceSlots;                        \
                tr_[0] = (int64_t((ITEM) >= (P).end_route) << 60) | (int64_t(xcc_id()) << 48) | \
                         int64_t(blockIdx.x);                                                 \
                tr_[kTrStart] = int64_t(__builtin_amdgcn_s_memrealtime());                    \
            }                                                                                 \
        }                                                                                     \
    } while (0)
#define SEKV_STAMP(P, SM, SLOT)                                                               \
    do {                                                                                      \
        if (threadIdx.x == 0 && (P).trace)                                                    \
            (P).trace[size_t((SM).trace_item) * kTraceSlots + (SLOT)] =                       \
                int64_t(__builtin_amdgcn_s_memrealtime());                                    \
    } while (0)
#define SEKV_NOTE(P, SM, SLOT, V)                                                             \
    do {                                                                                      \
        if (threadIdx.x == 0 && (P).trace)                                                    \
            (P).trace[size_t((SM).trace_item) * kTraceSlots + (SLOT)] = int64_t(V);           \
    } while (0)
#else
#define SEKV_TRACE_BEGIN(P, SM, ITEM) do {} while (0)
#define SEKV_STAMP(P, SM, SLOT) do {} while (0)
#define SEKV_NOTE(P, SM, SLOT, V) do {} while (0)
#endif

// Tagged words: payload in the low half, the launch tag in the high half.
__device__ inline uint64_t tagged(uint32_t tag, uint32_t v) { return (uint64_t(tag) << 32) | v; }
__device__ inline bool tag_is(uint64_t w, uint32_t tag) { return uint32_t(w >> 32) == tag; }
__device__ inline uint64_t pack2(float lo, float hi) {
    return uint64_t(__float_as_uint(lo)) | (uint64_t(__float_as_uint(hi)) << 32);
}
__device__ inline float lo_f(uint64_t w) { return __uint_as_float(uint32_t(w)); }
__device__ inline float hi_f(uint64_t w) { return __uint_as_float(uint32_t(w >> 32)); }

// The span word that travels with a selected span: |S| in bits 0..20, r_K / 4 in bits
// 21..25 and r_V / 4 in bits 26..30 (the retained ranks of its block).  Ranks read from
// the caller's table must be multiples of 16 / element bytes in [that, rank]; otherwise
// both are 0, and the zoom skips the block and flags it like one outside the arena.
template <class T>
__device__ inline int32_t span_word(const Params &p, int32_t L, int32_t table_word) {
    int rk = p.r, rv = p.r;
    if (p.block_rank) {
        rk = int(uint32_t(table_word) & 0xFFFFu);
        rv = int(uint32_t(table_word) >> 16);
        constexpr int gran = 16 / T::kBytes;
        const bool ok = rk >= gran && rk <= p.r && rk % gran == 0 && rv >= gran && rv <= p.r && rv % gran == 0;
        if (!ok) rk = rv = 0;
    }
    return int32_t((uint32_t(L) & 0x1FFFFFu) | (uint32_t(rk >> 2) << 21) | (uint32_t(rv >> 2) << 26));
}
__device__ inline int word_len(int32_t w) { return int(uint32_t(w) & 0x1FFFFFu); }
__device__ inline int word_rk(int32_t w) { return int((uint32_t(w) >> 21) & 31u) << 2; }
__device__ inline int word_rv(int32_t w) { return int((uint32_t(w) >> 26) & 31u) << 2; }

// ---------------------------------------------------------------------------
// shared memory
// ---------------------------------------------------------------------------
template <class T, int D, int G>
struct Smem {
    using GE = Geo<T, D>;
    static constexpr int HPT = (G + 1) / 2;              // routing heads per thread
    static constexpr int NJ = 4;                          // rows per thread in a summary block
    static constexpr int NJA = 8;                         // rows per thread in an anchor block
    static constexpr int AB = NJA * GE::RPP;              // anchor tokens per block
    static constexpr int CB = NJ * GE::RPP;               // summary rows per block
    struct Route {                                       // routing item
        unsigned char kb[CR * GE::RS];                   // summary key rows
        double lns[CR];                                  // ln|S| of the chunk's spans
        double pmax[2][CR];                              // per head group max score
        int32_t slen[CR];                                // |S| of the chunk's spans
        int64_t boff[CR];                                // their block offsets
        uint64_t skey[2][64];                            // two sorted halves of the chunk
        uint32_t sidx[2][64];
    };
    struct Share {                                       // share item
        float qf[G][D];
        uint32_t qb[G][D / 2];                           // the same query, bf16 pairs (bf16 storage)
        float sc[G][AB];                                 // anchor scores, then weights
        float cw[G][CB];                                 // summary logits, then weights
        uint4 cand[kMergeBuf];                           // {~span, key lo, key hi, -}
        uint32_t rk[NT];                                 // partial ranks (two scanners)
        int32_t sel[kMaxTopK];                           // the pair's selected spans
        int4 zi[kMaxTopK];                               // {span, |S|, offset lo, hi} per rank
        float w[G][kMaxTopK];                            // scale*log2e*sigma_K*(Vt_K q)
        float zs[G][kZoomBlock];                         // token scores, then weights
        float yr[4][G][kMaxTopK];                        // per-wave partial sums of p^T U_V
        float y[G][kMaxTopK];                            // (p^T U_V) * sigma_V
    };
    struct Merge {                                       // single-merger selection
        uint64_t key[kMergeBuf];
        uint32_t idx[kMergeBuf];
        int32_t sel[kMaxTopK];
    };
    struct Final {                                       // softmax merge
        float m[kMaxTopK][G], l[kMaxTopK][G];
        float wgt[kMaxTopK][G];
        float L[G];
    };
    union {
        Route route;
        Share share;
        Merge merge;
        Final fin;
    } u;
    float red[4][G][D];                                  // per-wave row sums
    float m_run[G], l_run[G], scale_old[G];              // online softmax state
    int32_t bcast[8];
#ifdef SEKV_PHASE_TRACE
    int trace_item;
#endif
};

// part[h] = sum over the values of 16-byte vector c of a row times query row h: packed
// bf16 dot products (exact products, fp32 sums) for bf16 storage, fp32 FMAs for fp32.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
template <class T, int D, int G>
__device__ inline void query_dot(const Smem<T, D, G> &sm, const uint4 &v, int c, float (&part)[G]) {
    const auto &Z = sm.u.share;
    if constexpr (T::kBytes == 2) {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int hl = 0; hl < G; ++hl) {
            float a = 0.0f;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w[i]),
                                                    __builtin_bit_cast(bf16x2_t, Z.qb[hl][c * 4 + i]), a, false);
            part[hl] = a;
        }
    } else {
        float f[T::kVec];
        T::unpack(v, f);
#pragma unroll
        for (int hl = 0; hl < G; ++hl) {
            part[hl] = 0.0f;
#pragma unroll
            for (int e = 0; e < T::kVec; ++e) part[hl] += Z.qf[hl][c * T::kVec + e] * f[e];
        }
    }
}

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

// Write the partial of share slot `slot`: (m, l) from the online state; o = the 4 wave
// rows of red, as float pairs.
template <class T, int D, int G>
__device__ inline void write_partial(const Params &p, Smem<T, D, G> &sm, int pair, int slot,
                                     int tid) {
    constexpr int NO = G * D / 2;
    const size_t base = size_t(pair) * p.n_zi + slot;
    if (tid < G) st_shared(&p.part_ml[base * G + tid], pack2(sm.m_run[tid], sm.l_run[tid]));
    uint64_t *po = p.part_o + base * NO;
    for (int o2 = tid; o2 < NO; o2 += NT) {
        const int hl = (2 * o2) / D, d = (2 * o2) % D;
        const float v0 = sm.red[0][hl][d] + sm.red[1][hl][d] + sm.red[2][hl][d] + sm.red[3][hl][d];
        const float v1 = sm.red[0][hl][d + 1] + sm.red[1][hl][d + 1] + sm.red[2][hl][d + 1] +
                         sm.red[3][hl][d + 1];
        st_shared(&po[o2], pack2(v0, v1));
    }
}

// Add acc, summed over this wave's rows, into the wave's row of sm.red after scaling that
// row by pend (the rescale factors of the folds since the previous flush); pend becomes 1.
// Each wave touches only its own row, so no synchronisation is needed here.
template <class T, int D, int G>
__device__ inline void acc_flush(Smem<T, D, G> &sm, float (&acc)[G][T::kVec], float (&pend)[G],
                                 int tid) {
    using GE = Geo<T, D>;
    const int lane = tid & 63, wave = tid >> 6;
#pragma unroll
    for (int hl = 0; hl < G; ++hl)
#pragma unroll
        for (int e = 0; e < GE::VEC; ++e) acc[hl][e] = col_sum<GE::RV>(acc[hl][e]);
    if (lane < GE::RV) {
#pragma unroll
        for (int hl = 0; hl < G; ++hl)
#pragma unroll
            for (int e = 0; e < GE::VEC; ++e) {
                float &r = sm.red[wave][hl][lane * GE::VEC + e];
                r = r * pend[hl] + acc[hl][e];
            }
    }
#pragma unroll
    for (int hl = 0; hl < G; ++hl) pend[hl] = 1.0f;
}

// Multiply the pending rescale factors by those of the fold that just finished.
template <int G>
__device__ inline void pend_fold(float (&pend)[G], const float *so) {
#pragma unroll
    for (int hl = 0; hl < G; ++hl) pend[hl] *= so[hl];
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
    const int ns = p.n_zi;
    constexpr int NO = G * D / 2;                       // float pairs per slot
    constexpr int NP = (NO + NT - 1) / NT;              // float pairs per thread
    constexpr int kBatch = 16;                          // slots whose values are in flight
    const uint64_t *ml = p.part_ml + size_t(pair) * ns * G;
    const uint64_t *po = p.part_o + size_t(pair) * ns * NO;
    // every load first: (m, l) of all slots to LDS, this thread's o values to registers
    for (int i = tid; i < ns * G; i += NT) {
        const uint64_t w = ld_shared(ml + i);
        F.m[i / G][i % G] = lo_f(w);
        F.l[i / G][i % G] = hi_f(w);
    }
    uint64_t ov[NP][kBatch];
#pragma unroll
    for (int u = 0; u < NP; ++u) {
        const int o2 = min(tid + NT * u, NO - 1);
#pragma unroll
        for (int s = 0; s < kBatch; ++s) ov[u][s] = ld_shared(po + size_t(min(s, ns - 1)) * NO + o2);
    }
    __syncthreads();
    const int wave = tid >> 6, lane = tid & 63;
    for (int hl = wave; hl < G; hl += 4) {
        float mx = -INFINITY;
        for (int s = lane; s < ns; s += 64)
            if (F.l[s][hl] > 0.0f) mx = fmaxf(mx, F.m[s][hl]);
        mx = wave_max(mx);
        float lsum = 0.0f;
        for (int s = lane; s < ns; s += 64) {
            float wgt = 0.0f;
            if (F.l[s][hl] > 0.0f) {
                wgt = exp2f(F.m[s][hl] - mx);
                lsum += wgt * F.l[s][hl];
            }
            F.wgt[s][hl] = wgt;
        }
        lsum = wave_sum(lsum);
        if (lane == 0) F.L[hl] = lsum;
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < NP; ++u) {
        const int o2 = tid + NT * u;
        if (o2 >= NO) continue;
        const int hl = (2 * o2) / D, d = (2 * o2) % D;
        float a0 = 0.0f, a1 = 0.0f;
#pragma unroll
        for (int s = 0; s < kBatch; ++s) {
            const float wgt = (s < ns) ? F.wgt[s][hl] : 0.0f;
            if (wgt != 0.0f) {
                a0 += wgt * lo_f(ov[u][s]);
                a1 += wgt * hi_f(ov[u][s]);
            }
        }
        for (int s = kBatch; s < ns; ++s) {              // more slots than the batch
            const float wgt = F.wgt[s][hl];
            const uint64_t v = ld_shared(po + size_t(s) * NO + o2);
            if (wgt != 0.0f) {
                a0 += wgt * lo_f(v);
                a1 += wgt * hi_f(v);
            }
        }
        const float L = F.L[hl];
        const float r0 = (L > 0.0f) ? a0 / L : 0.0f;
        const float r1 = (L > 0.0f) ? a1 / L : 0.0f;
        const size_t oi = (size_t(b) * p.Hq + size_t(g) * G + hl) * D + d;
        if (p.out_f32) {
            *reinterpret_cast<float2 *>(reinterpret_cast<float *>(p.out) + oi) = make_float2(r0, r1);
        } else {
            *reinterpret_cast<uint32_t *>(reinterpret_cast<uint16_t *>(p.out) + oi) =
                uint32_t(f32_to_bf16_rne(r0)) | (uint32_t(f32_to_bf16_rne(r1)) << 16);
        }
    }
}

// Shutdown of a launch, by the last workgroup out: zero the counters and advance the epoch
// (0 marks unwritten words).
__device__ inline void shutdown(const Params &p, uint32_t tag, int tid) {
    const int P = p.B * p.Hkv;
    for (int i = tid; i < P; i += NT) {
        p.route_cnt[i] = 0u;
        p.sel_ready[i] = 0u;
        p.part_cnt[i] = 0u;
    }
    if (tid == 0) {
        p.hdr->exit_count = 0u;
        st_shared(&p.hdr->epoch, tag + 1u == 0u ? 1u : tag + 1u);
    }
}

// Count one finished partial of `pair` (written, stores completed by every wave); the
// item completing the pair merges.  In the workgroup's last item (`leave`) the workgroup
// also counts itself out here, once the partial's count has returned (so every counter it
// touches is final), and the round trip of that count overlaps the merge; the last
// workgroup out shuts the launch down.  After this point the workgroup reads only untagged
// partials, so the shutdown may overlap another workgroup's merge.
template <class T, int D, int G>
__device__ inline void count_partial(const Params &p, Smem<T, D, G> &sm, int pair, int tid, bool leave,
                                     uint32_t tag) {
    if (tid == 0) {
        const uint32_t prev = counter_add(&p.part_cnt[pair], 1u);
        sm.bcast[0] = (prev + 1u == uint32_t(p.n_zi));
    }
    __syncthreads();
    uint32_t out = 0u;
    if (leave && tid == 0) out = counter_add(&p.hdr->exit_count, 1u);
    if (sm.bcast[0]) final_merge<T, D, G>(p, sm, pair, tid);
    if (leave) {
        if (tid == 0) sm.bcast[3] = (out == uint32_t(p.grid - 1));
        __syncthreads();
        if (sm.bcast[3]) shutdown(p, tag, tid);
    }
    __syncthreads();
}

// ---------------------------------------------------------------------------
// selection by a single merger (route mode, or more than kMergeBuf candidates).  Runs
// in the last route item of the pair, after every route item's records are complete.
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__device__ __forceinline__ void merge_selection(const Params &p, Smem<T, D, G> &sm, int pair, int tid) {
    auto &M = sm.u.merge;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    const int k = p.k;
    int m_b = p.n_spans[b];
    m_b = m_b < 0 ? 0 : (m_b > p.M_max ? p.M_max : m_b);
    const int n_cand = p.n_cand;
    const size_t FS = size_t(p.B) * p.Hkv * size_t(n_cand);
    const uint64_t *rec = p.cand + size_t(pair) * n_cand;
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
                const uint32_t ci = uint32_t(ld_shared(rec + kCandIdx * FS + c));
                if (ci < 0x80000000u) {
                    key = (uint64_t(uint32_t(ld_shared(rec + kCandKeyHi * FS + c))) << 32) |
                          uint32_t(ld_shared(rec + kCandKeyLo * FS + c));
                    idx = ci;
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
                const size_t bi = (size_t(b) * p.Hkv + g) * p.M_max + s;
                L = span_word<T>(p, p.span_len[size_t(b) * p.M_max + s], p.block_rank ? p.block_rank[bi] : 0);
                off = p.block_off[bi];
            }
            int32_t *zr = reinterpret_cast<int32_t *>(&p.zrec[size_t(pair) * k + j]);
            st_shared(zr + 0, s);
            st_shared(zr + 1, L);
            st_shared(zr + 2, int32_t(off & 0xFFFFFFFF));
            st_shared(zr + 3, int32_t(off >> 32));
        }
    }
    stores_done_barrier();
    if (p.mode == kModeFused && tid == 0) st_shared(&p.sel_ready[pair], 1u);
}

// Compile-time loop: f(IC<I>{}) for I in [B, E).
template <int V> struct IC { static constexpr int value = V; };
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (B < E) {
        f(IC<B>{});
        static_for<B + 1, E>(f);
    }
}

// ---------------------------------------------------------------------------
// float64 FMA chains with the query broadcast by DPP: lane l of every 16-lane row holds
// q[d] for d = 16 m + l in qv[m]; `v_fmac_f64` with row_newbcast:n reads lane n of the
// lane's own row, so each FMA takes the query value of column d straight from a
// register.  One 16-byte key vector (VEC consecutive columns starting at column N0,
// N0 % 16 + VEC <= 16) is folded into the HPT chains a[u] += q_u[d] * k[e], column by
// column, in increasing d: the same left-to-right sum as a plain loop.  A DPP source
// must not be written by a VALU instruction in the two preceding wait states; the
// s_nop at the top of every block guarantees it whatever the compiler placed before.
// ---------------------------------------------------------------------------
template <int HPT, int VEC, int N0>
__device__ __forceinline__ void dpp_fma_block(double (&a)[HPT], const double (&q)[HPT], const double (&k)[VEC]) {
    if constexpr (HPT == 1 && VEC == 4) {
        asm("s_nop 1\n\t"
            "v_fmac_f64_dpp %0, %1, %2 row_newbcast:%6 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %1, %3 row_newbcast:%7 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %1, %4 row_newbcast:%8 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %1, %5 row_newbcast:%9 row_mask:0xf bank_mask:0xf\n\t"
            : "+v"(a[0])
            : "v"(q[0]), "v"(k[0]), "v"(k[1]), "v"(k[2]), "v"(k[3]), "n"(N0 + 0), "n"(N0 + 1), "n"(N0 + 2), "n"(N0 + 3));
    }
    else if constexpr (HPT == 1 && VEC == 8) {
        asm("s_nop 1\n\t"
            "v_fmac_f64_dpp %0, %1, %2 row_newbcast:%10 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %1, %3 row_newbcast:%11 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %1, %4 row_newbcast:%12 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %1, %5 row_newbcast:%13 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %1, %6 row_newbcast:%14 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %1, %7 row_newbcast:%15 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %1, %8 row_newbcast:%16 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %1, %9 row_newbcast:%17 row_mask:0xf bank_mask:0xf\n\t"
            : "+v"(a[0])
            : "v"(q[0]), "v"(k[0]), "v"(k[1]), "v"(k[2]), "v"(k[3]), "v"(k[4]), "v"(k[5]), "v"(k[6]), "v"(k[7]), "n"(N0 + 0), "n"(N0 + 1), "n"(N0 + 2), "n"(N0 + 3), "n"(N0 + 4), "n"(N0 + 5), "n"(N0 + 6), "n"(N0 + 7));
    }
    else if constexpr (HPT == 2 && VEC == 4) {
        asm("s_nop 1\n\t"
            "v_fmac_f64_dpp %0, %2, %4 row_newbcast:%8 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %3, %4 row_newbcast:%8 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %2, %5 row_newbcast:%9 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %3, %5 row_newbcast:%9 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %2, %6 row_newbcast:%10 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %3, %6 row_newbcast:%10 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %2, %7 row_newbcast:%11 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %3, %7 row_newbcast:%11 row_mask:0xf bank_mask:0xf\n\t"
            : "+v"(a[0]), "+v"(a[1])
            : "v"(q[0]), "v"(q[1]), "v"(k[0]), "v"(k[1]), "v"(k[2]), "v"(k[3]), "n"(N0 + 0), "n"(N0 + 1), "n"(N0 + 2), "n"(N0 + 3));
    }
    else if constexpr (HPT == 2 && VEC == 8) {
        asm("s_nop 1\n\t"
            "v_fmac_f64_dpp %0, %2, %4 row_newbcast:%12 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %3, %4 row_newbcast:%12 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %2, %5 row_newbcast:%13 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %3, %5 row_newbcast:%13 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %2, %6 row_newbcast:%14 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %3, %6 row_newbcast:%14 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %2, %7 row_newbcast:%15 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %3, %7 row_newbcast:%15 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %2, %8 row_newbcast:%16 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %3, %8 row_newbcast:%16 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %2, %9 row_newbcast:%17 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %3, %9 row_newbcast:%17 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %2, %10 row_newbcast:%18 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %3, %10 row_newbcast:%18 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %2, %11 row_newbcast:%19 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %3, %11 row_newbcast:%19 row_mask:0xf bank_mask:0xf\n\t"
            : "+v"(a[0]), "+v"(a[1])
            : "v"(q[0]), "v"(q[1]), "v"(k[0]), "v"(k[1]), "v"(k[2]), "v"(k[3]), "v"(k[4]), "v"(k[5]), "v"(k[6]), "v"(k[7]), "n"(N0 + 0), "n"(N0 + 1), "n"(N0 + 2), "n"(N0 + 3), "n"(N0 + 4), "n"(N0 + 5), "n"(N0 + 6), "n"(N0 + 7));
    }
    else if constexpr (HPT == 4 && VEC == 4) {
        asm("s_nop 1\n\t"
            "v_fmac_f64_dpp %0, %4, %8 row_newbcast:%12 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %5, %8 row_newbcast:%12 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %2, %6, %8 row_newbcast:%12 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %3, %7, %8 row_newbcast:%12 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %4, %9 row_newbcast:%13 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %5, %9 row_newbcast:%13 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %2, %6, %9 row_newbcast:%13 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %3, %7, %9 row_newbcast:%13 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %4, %10 row_newbcast:%14 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %5, %10 row_newbcast:%14 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %2, %6, %10 row_newbcast:%14 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %3, %7, %10 row_newbcast:%14 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %4, %11 row_newbcast:%15 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %5, %11 row_newbcast:%15 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %2, %6, %11 row_newbcast:%15 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %3, %7, %11 row_newbcast:%15 row_mask:0xf bank_mask:0xf\n\t"
            : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3])
            : "v"(q[0]), "v"(q[1]), "v"(q[2]), "v"(q[3]), "v"(k[0]), "v"(k[1]), "v"(k[2]), "v"(k[3]), "n"(N0 + 0), "n"(N0 + 1), "n"(N0 + 2), "n"(N0 + 3));
    }
    else if constexpr (HPT == 4 && VEC == 8) {
        asm("s_nop 1\n\t"
            "v_fmac_f64_dpp %0, %4, %8 row_newbcast:%16 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %5, %8 row_newbcast:%16 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %2, %6, %8 row_newbcast:%16 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %3, %7, %8 row_newbcast:%16 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %4, %9 row_newbcast:%17 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %5, %9 row_newbcast:%17 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %2, %6, %9 row_newbcast:%17 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %3, %7, %9 row_newbcast:%17 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %4, %10 row_newbcast:%18 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %5, %10 row_newbcast:%18 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %2, %6, %10 row_newbcast:%18 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %3, %7, %10 row_newbcast:%18 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %4, %11 row_newbcast:%19 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %5, %11 row_newbcast:%19 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %2, %6, %11 row_newbcast:%19 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %3, %7, %11 row_newbcast:%19 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %4, %12 row_newbcast:%20 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %5, %12 row_newbcast:%20 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %2, %6, %12 row_newbcast:%20 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %3, %7, %12 row_newbcast:%20 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %4, %13 row_newbcast:%21 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %5, %13 row_newbcast:%21 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %2, %6, %13 row_newbcast:%21 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %3, %7, %13 row_newbcast:%21 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %4, %14 row_newbcast:%22 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %5, %14 row_newbcast:%22 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %2, %6, %14 row_newbcast:%22 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %3, %7, %14 row_newbcast:%22 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %0, %4, %15 row_newbcast:%23 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %1, %5, %15 row_newbcast:%23 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %2, %6, %15 row_newbcast:%23 row_mask:0xf bank_mask:0xf\n\t"
            "v_fmac_f64_dpp %3, %7, %15 row_newbcast:%23 row_mask:0xf bank_mask:0xf\n\t"
            : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3])
            : "v"(q[0]), "v"(q[1]), "v"(q[2]), "v"(q[3]), "v"(k[0]), "v"(k[1]), "v"(k[2]), "v"(k[3]), "v"(k[4]), "v"(k[5]), "v"(k[6]), "v"(k[7]), "n"(N0 + 0), "n"(N0 + 1), "n"(N0 + 2), "n"(N0 + 3), "n"(N0 + 4), "n"(N0 + 5), "n"(N0 + 6), "n"(N0 + 7));
    }
    else {
        static_assert(HPT == 1 || HPT == 2 || HPT == 4, "heads per thread");
    }
}

// ---------------------------------------------------------------------------
// route item: one chunk of CR spans of a pair
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__device__ __forceinline__ void route_item(const Params &p, Smem<T, D, G> &sm, int pair, int chunk,
                                           uint32_t tag, int tid, bool claimed = false) {
    using GE = Geo<T, D>;
    constexpr int HPT = Smem<T, D, G>::HPT;
    auto &R = sm.u.route;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    int m_b = p.n_spans[b];
    m_b = m_b < 0 ? 0 : (m_b > p.M_max ? p.M_max : m_b);
    const int s0 = chunk * CR;
    const int nv = max(0, min(CR, m_b - s0));
    const bool select = (p.mode != kModeAttend);       // candidates for the selection
    const bool publish = (p.mode != kModeRoute);       // coarse logits for the share items
    const size_t row0 = (size_t(b) * p.Hkv + g) * size_t(p.M_max) + s0;
    const int rgrp = tid / GE::RV, col = tid % GE::RV;
    const int wave = tid >> 6, lane = tid & 63;
    constexpr int NJ = (CR + GE::RPP - 1) / GE::RPP;

    // 0. claim the chunk: the claim word holds the tag of the launch that claimed it.  The
    //    result is needed only once the loads below are in: a chunk a waiting share item
    //    has already taken over (see help_route) is left to it.
    uint32_t prev_claim = tag;
    if (!claimed && tid == 0)
        prev_claim = __hip_atomic_exchange(&p.claim[size_t(pair) * p.n_rc + chunk], tag, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
    // 1. loads: summary keys (-> LDS), query (-> registers, float64), ln|S|, and
    //    |S| / block offsets for the candidate records.  Every load is issued before any
    //    value is used; addresses are clamped to the chunk's rows inside the arrays, so
    //    none waits for n_spans (validity is applied where the values are used).
    const int nr = min(CR, p.M_max - s0);               // rows of this chunk in the arrays
    double qv[D / 16][HPT];
    {
        const unsigned char *src = reinterpret_cast<const unsigned char *>(p.sum_k) + row0 * GE::RB;
        uint4 kv[NJ];
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int row = min(rgrp + GE::RPP * j, nr - 1);
            kv[j] = ld16(src + size_t(row) * GE::RB + col * 16);
        }
        // the query of the thread's head group: lane l of each 16-lane row holds
        // q_u[16 m + l] in qv[m][u]
        const int l16 = lane & 15, hgq = tid / CR;
        float qr[D / 16][HPT];
#pragma unroll
        for (int m = 0; m < D / 16; ++m)
#pragma unroll
            for (int u = 0; u < HPT; ++u) {
                const int h = min(hgq * HPT + u, G - 1);
                qr[m][u] = T::load1(p.q, (size_t(b) * p.Hq + size_t(g) * G + h) * D + m * 16 + l16);
            }
        const int ti = min(tid, nr - 1);
        const double lns = p.span_logsize[size_t(b) * p.M_max + s0 + ti];
        int32_t slen = 0, srank = 0;
        int64_t boff = 0;
        if (select) {
            slen = p.span_len[size_t(b) * p.M_max + s0 + ti];
            boff = p.block_off[row0 + ti];
            if (p.block_rank) srank = p.block_rank[row0 + ti];
        }
#pragma unroll
        for (int m = 0; m < D / 16; ++m)
#pragma unroll
            for (int u = 0; u < HPT; ++u) qv[m][u] = (hgq * HPT + u < G) ? double(qr[m][u]) : 0.0;
        if (tid < CR) {
            R.lns[tid] = lns;
            R.slen[tid] = span_word<T>(p, slen, srank);
            R.boff[tid] = boff;
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int row = rgrp + GE::RPP * j;
            if (row < nr) *reinterpret_cast<uint4 *>(R.kb + size_t(row) * GE::RS + col * 16) = kv[j];
        }
    }
    if (tid == 0) sm.bcast[5] = claimed || prev_claim != tag;
    __syncthreads();
    SEKV_STAMP(p, sm, kTrRLoaded);
    if (!sm.bcast[5]) return;                           // another workgroup runs this chunk

    // 2. routing scores: float64, products exact, summed left to right over d, then
    //    (s * scale) + ln|S| as two separately rounded operations.  Thread (span i, head
    //    group hg) runs HPT chains that share each converted key element; the head group
    //    is uniform per wave and the query comes from registers by DPP broadcast.
    const int i = tid % CR, hg = tid / CR;
    double sc[HPT];
    {
        double a[HPT];
#pragma unroll
        for (int u = 0; u < HPT; ++u) a[u] = 0.0;
        const unsigned char *rowp = R.kb + size_t(i) * GE::RS;
        static_for<0, GE::RV>([&](auto cc) {
            constexpr int c = decltype(cc)::value;
            constexpr int d0 = c * GE::VEC;
            float f[GE::VEC];
            T::unpack(*reinterpret_cast<const uint4 *>(rowp + c * 16), f);
            double kd[GE::VEC];
#pragma unroll
            for (int e = 0; e < GE::VEC; ++e) kd[e] = double(f[e]);
            double qq[HPT];
#pragma unroll
            for (int u = 0; u < HPT; ++u) qq[u] = qv[d0 / 16][u];
            dpp_fma_block<HPT, GE::VEC, d0 % 16>(a, qq, kd);
        });
        {
#pragma clang fp contract(off)
#pragma unroll
            for (int u = 0; u < HPT; ++u) {
                const double m = a[u] * p.scale;
                sc[u] = (i < nv) ? m + R.lns[i] : -INFINITY;
            }
        }
    }
    // 3. per (head, span) outputs: the tagged base-2 logit for the share items, the
    //    natural-unit logit for the caller
#pragma unroll
    for (int u = 0; u < HPT; ++u) {
        const int h = hg * HPT + u;
        if (h >= G) continue;
        if (publish && i < nv)
            st_shared(&p.tlg[(size_t(pair) * G + h) * p.M_max + s0 + i],
                      tagged(tag, __float_as_uint(float(sc[u] * kLog2eD))));
        if (p.logits_out && s0 + i < p.M_max)
            p.logits_out[(size_t(b) * p.Hq + size_t(g) * G + h) * p.M_max + s0 + i] = float(sc[u]);
    }
    SEKV_STAMP(p, sm, kTrRScored);
    if (!select) return;
    {
        double mx = -INFINITY;
#pragma unroll
        for (int u = 0; u < HPT; ++u)
            if (hg * HPT + u < G) mx = fmax(mx, sc[u]);
        R.pmax[hg][i] = mx;
    }
    __syncthreads();

    // 4. candidates: waves 0 and 1 each sort 64 (key, span) pairs with a bitonic network;
    //    a span's rank in the chunk is its position plus the number of better entries of
    //    the other half (binary search); the best kc become the chunk's candidate records.
    if (wave < 2) {
        const int ii = wave * 64 + lane;
        uint64_t key = 0;
        uint32_t idx = kInvalidIdx - uint32_t(ii);
        if (ii < nv) {
            key = order_key(fmax(R.pmax[0][ii], R.pmax[1][ii]));
            idx = uint32_t(s0 + ii);
        }
#define SEKV_BITONIC_STEP(STRIDE)                                                          \
        {                                                                                  \
            const uint32_t klo = lane_xor<STRIDE>(uint32_t(key), lane);                    \
            const uint32_t khi = lane_xor<STRIDE>(uint32_t(key >> 32), lane);              \
            const uint32_t oi = lane_xor<STRIDE>(idx, lane);                               \
            const uint64_t ok = (uint64_t(khi) << 32) | klo;                               \
            const bool lower = (lane & (STRIDE)) == 0;                                     \
            const bool take = (lower == up) ? better(ok, oi, key, idx)                     \
                                            : better(key, idx, ok, oi);                    \
            if (take) { key = ok; idx = oi; }                                              \
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
    SEKV_STAMP(p, sm, kTrRSorted);
    const int kc = p.kc;
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
        if (rank < kc) {
            // every position of every chunk is written each launch (invalid entries too),
            // so a reader never has to know which ones exist
            const bool valid = idx < 0x80000000u;
            const int li = valid ? int(idx) - s0 : 0;
            const int32_t len = valid ? R.slen[li] : 0;
            const uint64_t off = valid ? uint64_t(R.boff[li]) : 0;
            const size_t FS = size_t(p.B) * p.Hkv * size_t(p.n_cand);
            uint64_t *rec = p.cand + size_t(pair) * p.n_cand + size_t(chunk) * kc + rank;
            st_shared(rec + kCandKeyHi * FS, tagged(tag, valid ? uint32_t(key >> 32) : 0u));
            st_shared(rec + kCandKeyLo * FS, tagged(tag, valid ? uint32_t(key) : 0u));
            st_shared(rec + kCandIdx * FS, tagged(tag, valid ? idx : kInvalidIdx));
            st_shared(rec + kCandLen * FS, tagged(tag, uint32_t(len)));
            st_shared(rec + kCandOffLo * FS, tagged(tag, uint32_t(off)));
            st_shared(rec + kCandOffHi * FS, tagged(tag, uint32_t(off >> 32)));
        }
    }
    SEKV_STAMP(p, sm, kTrRPublished);
    if (p.merger) {
        // single merger: the last route item of the pair (counted after its records are
        // complete) selects for the whole pair
        stores_done_barrier();
        if (tid == 0) {
            const uint32_t prev = counter_add(&p.route_cnt[pair], 1u);
            sm.bcast[1] = (prev == uint32_t(p.n_rc - 1));
        }
        __syncthreads();
        if (sm.bcast[1]) merge_selection<T, D, G>(p, sm, pair, tid);
    }
}

// ---------------------------------------------------------------------------
// share item pieces
// ---------------------------------------------------------------------------
// Rows rgrp + RPP*j (j < NJ) of a block of n rows; addresses are clamped to the last
// row, so every vector is loaded (validity is applied where the values are used).
template <class T, int D, int NJ>
__device__ inline void load_rows(uint4 (&v)[NJ], const unsigned char *base, int n, int rgrp, int col) {
    using GE = Geo<T, D>;
    if (n <= 0) return;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int row = min(rgrp + GE::RPP * j, n - 1);
        v[j] = ld16(base + size_t(row) * GE::RB + col * 16);
    }
}

// One block of na anchor tokens, in two halves so that the next block's keys can load
// while this block's values are used: the scores (into Z.sc), then the online softmax
// and the weighted values (into sm.red).
template <class T, int D, int G, int NJ>
__device__ inline void anchor_scores(const Params &p, Smem<T, D, G> &sm, const uint4 (&kr)[NJ], int na,
                                     int rgrp, int col) {
    using GE = Geo<T, D>;
    auto &Z = sm.u.share;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        const int row = rgrp + GE::RPP * j;
        float part[G];
        query_dot<T, D, G>(sm, kr[j], col, part);
#pragma unroll
        for (int hl = 0; hl < G; ++hl) part[hl] = row_sum<GE::RV>(part[hl]);
        if (col == 0 && row < na)
#pragma unroll
            for (int hl = 0; hl < G; ++hl) Z.sc[hl][row] = part[hl] * p.scale_log2;
    }
    __syncthreads();
}

template <class T, int D, int G, int NJ>
__device__ inline void anchor_values(Smem<T, D, G> &sm, const uint4 (&vr)[NJ], int na, float (&pend)[G],
                                     int rgrp, int tid) {
    using GE = Geo<T, D>;
    constexpr int AB = Smem<T, D, G>::AB;
    auto &Z = sm.u.share;
    online_fold(&Z.sc[0][0], AB, na, G, sm.m_run, sm.l_run, sm.scale_old, tid);
    __syncthreads();
    pend_fold<G>(pend, sm.scale_old);
    float acc[G][GE::VEC];
    acc_zero<T, D, G>(acc);
    acc_rows<T, D, G, NJ>(acc, vr, &Z.sc[0][0], AB, na, rgrp);
    acc_flush<T, D, G>(sm, acc, pend, tid);
    __syncthreads();
}

// One block of nc summary rows starting at span c0; Z.cw holds their base-2 logits.
// Spans among the pair's k selected ones (Z.sel) are skipped: they are zoomed.
template <class T, int D, int G, int NJ>
__device__ inline void coarse_block(Smem<T, D, G> &sm, const uint4 (&cv)[NJ], int c0, int nc,
                                    int k, float (&pend)[G], int rgrp, int tid) {
    using GE = Geo<T, D>;
    constexpr int CB = Smem<T, D, G>::CB;
    static_assert(CB <= NT, "one thread per summary row");
    auto &Z = sm.u.share;
    if (tid < nc) {
        bool ex = false;
        for (int t = 0; t < k; ++t) ex |= (Z.sel[t] == c0 + tid);
        if (ex)
#pragma unroll
            for (int hl = 0; hl < G; ++hl) Z.cw[hl][tid] = -INFINITY;
    }
    __syncthreads();
    online_fold(&Z.cw[0][0], CB, nc, G, sm.m_run, sm.l_run, sm.scale_old, tid);
    __syncthreads();
    pend_fold<G>(pend, sm.scale_old);
    float acc[G][GE::VEC];
    acc_zero<T, D, G>(acc);
    acc_rows<T, D, G, NJ>(acc, cv, &Z.cw[0][0], CB, nc, rgrp);
    acc_flush<T, D, G>(sm, acc, pend, tid);
    __syncthreads();
}

// Base-2 logits of summary rows [c0, c0 + nc) into Z.cw: one polling attempt on this
// launch's tagged words (returns whether every tag was current), or the caller's logits.
template <class T, int D, int G>
__device__ inline bool coarse_logits(const Params &p, Smem<T, D, G> &sm, int pair, int c0, int nc,
                                     uint32_t tag, int tid) {
    constexpr int CB = Smem<T, D, G>::CB;
    auto &Z = sm.u.share;
    bool ok = true;
    if (p.logits_in) {
        const int b = pair / p.Hkv, g = pair % p.Hkv;
        for (int t = tid; t < G * CB; t += NT) {
            const int hl = t / CB, i = t % CB;
            if (i < nc)
                Z.cw[hl][i] = p.logits_in[(size_t(b) * p.Hq + size_t(g) * G + hl) * p.M_max + c0 + i] * kLog2e;
        }
        return true;
    }
    for (int t = tid; t < G * CB; t += NT) {
        const int hl = t / CB, i = t % CB;
        if (i < nc) {
            const uint64_t w = ld_shared(&p.tlg[(size_t(pair) * G + hl) * p.M_max + c0 + i]);
            ok &= tag_is(w, tag);
            Z.cw[hl][i] = lo_f(w);
        }
    }
    return ok;
}

// Poll until the logits of summary block [c0, c0 + nc) are this launch's.  Returns true
// when the wait has lasted kHelpAfter polls (the share item then gives up for help_route).
template <class T, int D, int G>
__device__ inline bool wait_coarse_logits(const Params &p, Smem<T, D, G> &sm, int pair, int c0,
                                          int nc, uint32_t tag, int tid, bool may_give_up) {
    for (uint32_t it = 0;; ++it) {
        const bool ok = coarse_logits<T, D, G>(p, sm, pair, c0, nc, tag, tid);
        if (__syncthreads_and(ok)) return false;
        if (it >= kSpinLimit) {
            if (tid == 0) flag_error(p, kErrSpinTimeout);
            return false;
        }
        if (may_give_up && it >= kHelpAfter) return true;
        __builtin_amdgcn_s_sleep(2);
    }
}

// A share item whose wait has lasted kHelpAfter polls gives up (share_item returns true)
// and its workgroup runs every routing chunk of the pair that no workgroup has claimed yet
// (a chunk's owner may not be resident: other kernels can hold the compute units), then
// runs the share item again from the start.  Claimed chunks belong to running workgroups,
// which never wait, so every wait ends whatever the residency.
template <class T, int D, int G>
__device__ __forceinline__ void help_route(const Params &p, Smem<T, D, G> &sm, int pair, uint32_t tag, int tid) {
    for (int c = 0; c < p.n_rc; ++c) {
        __syncthreads();
        if (tid == 0) {
            uint32_t *w = &p.claim[size_t(pair) * p.n_rc + c];
            sm.bcast[6] = ld_shared(w) != tag &&
                          __hip_atomic_exchange(w, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != tag;
        }
        __syncthreads();
        if (sm.bcast[6]) route_item<T, D, G>(p, sm, pair, c, tag, tid, true);
    }
    __syncthreads();
}

constexpr int kOwn = kMergeBuf / NT;                   // candidates per thread when ranking

// One polling attempt on the pair's candidate records; thread tid owns candidates tid
// and tid + NT.  Returns whether every tag was current.
__device__ inline bool load_candidates(const Params &p, int pair, uint32_t tag, uint64_t (&okey)[kOwn],
                                       uint32_t (&oidx)[kOwn], int32_t (&olen)[kOwn],
                                       int64_t (&ooff)[kOwn], int tid) {
    const size_t FS = size_t(p.B) * p.Hkv * size_t(p.n_cand);
    const uint64_t *rec = p.cand + size_t(pair) * p.n_cand;
    bool ok = true;
#pragma unroll
    for (int u = 0; u < kOwn; ++u) {
        const int c = tid + NT * u;
        okey[u] = 0;
        oidx[u] = kInvalidIdx;
        olen[u] = 0;
        ooff[u] = 0;
        if (c < p.n_cand) {
            uint64_t w[kCandFields];
#pragma unroll
            for (int f = 0; f < kCandFields; ++f) w[f] = ld_shared(rec + f * FS + c);
#pragma unroll
            for (int f = 0; f < kCandFields; ++f) ok &= tag_is(w[f], tag);
            okey[u] = (uint64_t(uint32_t(w[kCandKeyHi])) << 32) | uint32_t(w[kCandKeyLo]);
            oidx[u] = uint32_t(w[kCandIdx]);
            olen[u] = int32_t(uint32_t(w[kCandLen]));
            ooff[u] = int64_t(uint64_t(uint32_t(w[kCandOffLo])) | (uint64_t(uint32_t(w[kCandOffHi])) << 32));
        }
    }
    return ok;
}

// rk += 1 if (key_o, ~idx_o) > (key_c, ~idx_c) as 96-bit unsigned numbers, i.e. if
// candidate o is ahead of candidate c in (key desc, span asc): the borrow out of
// mine - other.  Words are {~idx, key lo, key hi}.
__device__ __forceinline__ void count_ahead(uint32_t &rk, const uint4 &o, uint32_t m0, uint32_t m1,
                                            uint32_t m2) {
    uint32_t t;
    asm("v_sub_co_u32 %0, vcc, %2, %3\n\t"
        "v_subb_co_u32 %0, vcc, %4, %5, vcc\n\t"
        "v_subb_co_u32 %0, vcc, %6, %7, vcc\n\t"
        "v_addc_co_u32 %1, vcc, 0, %1, vcc"
        : "=&v"(t), "+v"(rk)
        : "v"(m0), "v"(o.x), "v"(m1), "v"(o.y), "v"(m2), "v"(o.z)
        : "vcc");
}

// Rank the pair's candidates (LDS): rank = number of candidates ahead in (key desc,
// span asc).  Ranks below k fill Z.sel and Z.zi ({span, |S|, offset}).  Up to NT/2
// candidates, two threads scan half the list each.
template <class T, int D, int G>
__device__ __forceinline__ void rank_candidates(const Params &p, Smem<T, D, G> &sm, int m_b,
                                                const uint64_t (&okey)[kOwn], const uint32_t (&oidx)[kOwn],
                                                const int32_t (&olen)[kOwn], const int64_t (&ooff)[kOwn],
                                                int tid) {
    auto &Z = sm.u.share;
    const int k = p.k, n_cand = p.n_cand;
#pragma unroll
    for (int u = 0; u < kOwn; ++u) {
        const int c = tid + NT * u;
        if (c < n_cand) Z.cand[c] = make_uint4(~oidx[u], uint32_t(okey[u]), uint32_t(okey[u] >> 32), 0);
    }
    __syncthreads();
    const bool split = n_cand <= NT / 2;
    if (split) {
        // thread c and c + NT/2 rank candidate c over the two halves of the list
        const int c = tid % (NT / 2), half = tid / (NT / 2);
        const int o0 = half ? n_cand / 2 : 0, o1 = half ? n_cand : n_cand / 2;
        uint32_t rk = 0;
        if (c < n_cand) {
            const uint4 me = Z.cand[c];
            int o = o0;
            for (; o + 8 <= o1; o += 8) {
                uint4 e[8];
#pragma unroll
                for (int w = 0; w < 8; ++w) e[w] = Z.cand[o + w];
#pragma unroll
                for (int w = 0; w < 8; ++w) count_ahead(rk, e[w], me.x, me.y, me.z);
            }
            for (; o < o1; ++o) count_ahead(rk, Z.cand[o], me.x, me.y, me.z);
        }
        Z.rk[tid] = rk;
        __syncthreads();
        if (tid < n_cand && oidx[0] < 0x80000000u) {
            const int r = int(Z.rk[tid] + Z.rk[tid + NT / 2]);
            if (r < k && r < m_b) {
                Z.sel[r] = int32_t(oidx[0]);
                Z.zi[r] = make_int4(int32_t(oidx[0]), olen[0], int32_t(ooff[0] & 0xFFFFFFFF),
                                    int32_t(ooff[0] >> 32));
            }
        }
    } else {
#pragma unroll
        for (int u = 0; u < kOwn; ++u) {
            const int c = tid + NT * u;
            if (c >= n_cand || oidx[u] >= 0x80000000u) continue;
            const uint32_t m0 = ~oidx[u], m1 = uint32_t(okey[u]), m2 = uint32_t(okey[u] >> 32);
            uint32_t rk = 0;
            int o = 0;
            for (; o + 8 <= n_cand; o += 8) {
                uint4 e[8];
#pragma unroll
                for (int w = 0; w < 8; ++w) e[w] = Z.cand[o + w];
#pragma unroll
                for (int w = 0; w < 8; ++w) count_ahead(rk, e[w], m0, m1, m2);
            }
            for (; o < n_cand; ++o) count_ahead(rk, Z.cand[o], m0, m1, m2);
            if (int(rk) < k && int(rk) < m_b) {
                Z.sel[rk] = int32_t(oidx[u]);
                Z.zi[rk] = make_int4(int32_t(oidx[u]), olen[u], int32_t(ooff[u] & 0xFFFFFFFF),
                                     int32_t(ooff[u] >> 32));
            }
        }
    }
    __syncthreads();
}

// ---------------------------------------------------------------------------
// zoom of one span through its factors, RU = 16-byte vectors per factor row U[t][:].
// `mid` runs once the first factor loads are issued: work that needs none of them.
// ---------------------------------------------------------------------------
template <class T, int D, int G, int RU, bool RANKED, class Mid>
__device__ __forceinline__ void zoom_span(const Params &p, Smem<T, D, G> &sm, int L, int rk, int rv,
                                          int64_t off, float (&pend)[G], int tid, Mid &&mid) {
    using GE = Geo<T, D>;
    auto &Z = sm.u.share;
    constexpr int VEC = GE::VEC;
    constexpr int RV = GE::RV;
    constexpr int R = RU * 16 / T::kBytes;               // rank of the factors
    constexpr int NVT = (R * RV + NT - 1) / NT;          // Vt vectors per thread
    constexpr int NSV = (G * R + NT - 1) / NT;           // y entries per thread
    constexpr int NB = (8 * NT / RU) < kZoomBlock ? (8 * NT / RU) : kZoomBlock;  // tokens/block
    constexpr int NU = NB * RU / NT;                     // U vectors per thread per block
    constexpr int LG_RU = RU == 1 ? 0 : RU == 2 ? 1 : RU == 4 ? 2 : RU == 8 ? 3 : 4;
    const int rgrp = tid / GE::RV, col = tid % GE::RV;
    const int ucol = tid % RU;
    const int wave = tid >> 6, lane = tid & 63;
    // The block keeps r_K <= R key components and r_V <= R value components: rows,
    // columns and sigmas past them are not loaded and count as zero, so they add nothing
    // to the scores and values (the dropped components of Sec. 3.2).  Without a rank
    // table every block has R of each (compile-time, so the masks fold away).
    if constexpr (RANKED) {
        rk = __builtin_amdgcn_readfirstlane(rk);
        rv = __builtin_amdgcn_readfirstlane(rv);
    } else {
        rk = R;
        rv = R;
    }
    const int ruk = rk * T::kBytes / 16, ruv = rv * T::kBytes / 16;
    const unsigned char *UK = p.factors + off;
    const unsigned char *sK = UK + size_t(L) * rk * T::kBytes;
    const unsigned char *VtK = sK + size_t(rk) * T::kBytes;
    const unsigned char *UV = VtK + size_t(rk) * D * T::kBytes;
    const unsigned char *sV = UV + size_t(L) * rv * T::kBytes;
    const unsigned char *VtV = sV + size_t(rv) * T::kBytes;
    const int nb0 = min(NB, L);
    const uint4 zero4 = make_uint4(0u, 0u, 0u, 0u);

    // issue in the order of use: sigmas, Vt_K, U_K, then (after `mid`) U_V.  Addresses
    // are clamped into the block, validity is applied where values are used.
    float sk_reg[NVT], sv_reg[NSV];
    uint4 vk[NVT], vvt[NVT], uk[NU], uv[NU];
#pragma unroll
    for (int u = 0; u < NVT; ++u) {
        const int vi = min(tid + NT * u, R * RV - 1);
        sk_reg[u] = vi / RV < rk ? T::load1(sK, vi / RV) : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < NSV; ++u) {
        const int i = (tid + NT * u) % R;
        sv_reg[u] = i < rv ? T::load1(sV, i) : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < NVT; ++u) {
        const int vi = min(tid + NT * u, R * RV - 1);
        vk[u] = vi / RV < rk ? ld16(VtK + size_t(vi / RV) * GE::RB + (vi % RV) * 16) : zero4;
    }
#pragma unroll
    for (int u = 0; u < NU; ++u) {
        const int tok = min((tid + NT * u) / RU, nb0 - 1);
        uk[u] = ucol < ruk ? ld16(UK + size_t(tok) * rk * T::kBytes + ucol * 16) : zero4;
    }
    SEKV_STAMP(p, sm, kTrSZoomIssued);
    mid();
    SEKV_STAMP(p, sm, kTrSZoomMid);
#pragma unroll
    for (int u = 0; u < NU; ++u) {
        const int tok = min((tid + NT * u) / RU, nb0 - 1);
        uv[u] = ucol < ruv ? ld16(UV + size_t(tok) * rv * T::kBytes + ucol * 16) : zero4;
    }

    // w[h][i] = scale*log2e * sigma_K[i] * (Vt_K[i] . q_h).  No barrier first: Z.w was
    // last read by an earlier zoom, which has passed several barriers since, and the
    // query rows (Z.qf / Z.qb) were written at the start of the item.
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
        if (vi < R * RV && c == 0)
#pragma unroll
            for (int hl = 0; hl < G; ++hl) Z.w[hl][row] = part[hl] * sk_reg[u] * p.scale_log2;
    }
    // Vt_V rows take the registers Vt_K has released
#pragma unroll
    for (int u = 0; u < NVT; ++u) {
        const int vi = min(tid + NT * u, R * RV - 1);
        vvt[u] = vi / RV < rv ? ld16(VtV + size_t(vi / RV) * GE::RB + (vi % RV) * 16) : zero4;
    }

    __syncthreads();
    SEKV_STAMP(p, sm, kTrSZoomW);

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
                uk[u] = ucol < ruk ? ld16(UK + size_t(t0 + tok) * rk * T::kBytes + ucol * 16) : zero4;
            }
#pragma unroll
            for (int u = 0; u < NU; ++u) {
                const int tok = min((tid + NT * u) / RU, nb - 1);
                uv[u] = ucol < ruv ? ld16(UV + size_t(t0 + tok) * rv * T::kBytes + ucol * 16) : zero4;
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
            for (int e = 0; e < VEC; ++e) yacc[hl][e] *= so;
        }
        pend_fold<G>(pend, sm.scale_old);
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
        if (t0 + NB < L) __syncthreads();               // Z.zs and scale_old are reused
    }
    SEKV_STAMP(p, sm, kTrSZoomTokens);
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
        if (t < G * R) {
            const int hl = t / R, i = t % R;
            Z.y[hl][i] = (Z.yr[0][hl][i] + Z.yr[1][hl][i] + Z.yr[2][hl][i] + Z.yr[3][hl][i]) *
                         sv_reg[u];
        }
    }
    __syncthreads();
    // o[h][:] += sum_i y~[h][i] Vt_V[i][:]; Vt_V rows of column c sit RV lanes apart,
    // exactly like summary rows
    float acc[G][VEC];
    acc_zero<T, D, G>(acc);
#pragma unroll
    for (int u = 0; u < NVT; ++u) {
        const int vi = tid + NT * u;
        if (vi < R * RV) {
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
    acc_flush<T, D, G>(sm, acc, pend, tid);
    SEKV_STAMP(p, sm, kTrSZoomDone);
}

// ---------------------------------------------------------------------------
// share item: anchors share, selection slot j, summaries share of one pair
// ---------------------------------------------------------------------------
// Returns true when a wait lasted kHelpAfter polls: the caller then helps with routing
// (help_route) and runs the item again from the start.
template <class T, int D, int G>
__device__ __forceinline__ bool share_item(const Params &p, Smem<T, D, G> &sm, int pair, int j,
                                           uint32_t tag, int tid, bool first, bool may_give_up, bool leave) {
    using GE = Geo<T, D>;
    using SM = Smem<T, D, G>;
    constexpr int NJ = SM::NJ, NJA = SM::NJA, AB = SM::AB, CB = SM::CB;
    auto &Z = sm.u.share;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    const int k = p.k, r = p.r, nz = p.n_zi;
    // this item's shares: contiguous ranges of the anchor and span index spaces up to
    // the maxima, so the first loads need no table value; the sequence's own counts
    // (n_anchors, n_spans) mask rows where the values are used
    // anchors go to the slots that start with the launch (j < n_early): they fold them
    // while routing runs, and later slots reach their selection and zoom sooner
    const int ne = p.n_early;
    const int as = (p.A_max + ne - 1) / ne;
    const int a_lo = j < ne ? min(p.A_max, j * as) : p.A_max, a_hi = min(p.A_max, a_lo + as);
    const int cs = (p.M_max + nz - 1) / nz;
    const int c_lo = min(p.M_max, j * cs), c_hi = min(p.M_max, c_lo + cs);
    const int rgrp = tid / GE::RV, col = tid % GE::RV;
    const size_t pr = size_t(b) * p.Hkv + g;
    const unsigned char *ak = reinterpret_cast<const unsigned char *>(p.anchor_k) + pr * p.A_max * GE::RB;
    const unsigned char *av = reinterpret_cast<const unsigned char *>(p.anchor_v) + pr * p.A_max * GE::RB;
    const unsigned char *sv = reinterpret_cast<const unsigned char *>(p.sum_v) + pr * p.M_max * GE::RB;

    if (first && p.end_route > 0) __builtin_amdgcn_s_sleep(kShareHoldBack);
    // 1. loads that depend on nothing: the first anchor block, the first summary block
    //    (values only; its logits come from routing), the query
    uint4 kr[NJA], vr[NJA], cv[NJ];
    load_rows<T, D, NJA>(kr, ak + size_t(a_lo) * GE::RB, min(AB, a_hi - a_lo), rgrp, col);
    load_rows<T, D, NJA>(vr, av + size_t(a_lo) * GE::RB, min(AB, a_hi - a_lo), rgrp, col);
    load_rows<T, D, NJ>(cv, sv + size_t(c_lo) * GE::RB, min(CB, c_hi - c_lo), rgrp, col);
    int m_b = p.n_spans[b];
    m_b = m_b < 0 ? 0 : (m_b > p.M_max ? p.M_max : m_b);
    int An = p.n_anchors[b];
    An = An < 0 ? 0 : (An > p.A_max ? p.A_max : An);
    for (int i = tid; i < G * D; i += NT) {
        const int hl = i / D, d = i % D;
        Z.qf[hl][d] = T::load1(p.q, (size_t(b) * p.Hq + size_t(g) * G + hl) * D + d);
    }
    if constexpr (T::kBytes == 2) {
        const uint32_t *q2 = reinterpret_cast<const uint32_t *>(p.q) + (size_t(b) * p.Hq + size_t(g) * G) * (D / 2);
        for (int i = tid; i < G * D / 2; i += NT) Z.qb[i / (D / 2)][i % (D / 2)] = q2[i];
    }
    online_reset(G, sm.m_run, sm.l_run, sm.scale_old, tid);
    for (int t = tid; t < kMaxTopK; t += NT) { Z.sel[t] = -1; Z.zi[t] = make_int4(-1, 0, 0, 0); }
    for (int i = tid; i < 4 * G * D; i += NT) (&sm.red[0][0][0])[i] = 0.0f;
    __syncthreads();
    // valid rows of the prefetched blocks
    const int nc0 = max(0, min(min(CB, c_hi - c_lo), m_b - c_lo));
    // the weighted value sums live in sm.red (one row per wave); pend holds the rescale
    // factors not yet applied to them
    float pend[G];
#pragma unroll
    for (int hl = 0; hl < G; ++hl) pend[hl] = 1.0f;

    // 2. the anchor share, while routing runs elsewhere; the next block's keys load
    //    while this block's values are used, its values while the next scores are taken
    for (int a0 = a_lo; a0 < a_hi && a0 < An; a0 += AB) {
        const int na = min(min(AB, a_hi - a0), An - a0);
        const int a1 = a0 + AB;
        const int na1 = (a1 < a_hi && a1 < An) ? min(min(AB, a_hi - a1), An - a1) : 0;
        anchor_scores<T, D, G, NJA>(p, sm, kr, na, rgrp, col);
        load_rows<T, D, NJA>(kr, ak + size_t(a1) * GE::RB, na1, rgrp, col);
        anchor_values<T, D, G, NJA>(sm, vr, na, pend, rgrp, tid);
        load_rows<T, D, NJA>(vr, av + size_t(a1) * GE::RB, na1, rgrp, col);
    }

    SEKV_STAMP(p, sm, kTrSAnchors);
    // 3. the selection (Z.sel, this slot's span in bcast) and the first block's logits
    const bool per_item = (p.mode == kModeFused) && !p.merger;
    if (per_item) {
        uint64_t okey[kOwn];
        uint32_t oidx[kOwn];
        int32_t olen[kOwn];
        int64_t ooff[kOwn];
        bool done = false;
        for (uint32_t it = 0;; ++it) {
            bool ok = load_candidates(p, pair, tag, okey, oidx, olen, ooff, tid);
            ok &= coarse_logits<T, D, G>(p, sm, pair, c_lo, nc0, tag, tid);
            const bool all = __syncthreads_and(ok);
            if (it == 0) SEKV_STAMP(p, sm, kTrSPolled);
            if (all) {
                SEKV_NOTE(p, sm, kTrSPolls, it + 1);
                done = true;
                break;
            }
            if (it >= kSpinLimit) {
                if (tid == 0) flag_error(p, kErrSpinTimeout);
                break;
            }
            if (may_give_up && it >= kHelpAfter) return true;
            __builtin_amdgcn_s_sleep(2);
        }
        if (done) rank_candidates<T, D, G>(p, sm, m_b, okey, oidx, olen, ooff, tid);
        if (tid < k && tid % nz == j && p.sel_out) p.sel_out[size_t(pair) * k + tid] = Z.sel[tid];
    } else {
        if (p.mode == kModeFused) {
            // single merger: wait for the pair's selection records
            for (uint32_t it = 0;; ++it) {
                if (tid == 0) sm.bcast[2] = ld_shared(&p.sel_ready[pair]) != 0u ? 1 : 0;
                __syncthreads();
                if (sm.bcast[2]) break;
                if (it >= kSpinLimit) {
                    if (tid == 0) flag_error(p, kErrSpinTimeout);
                    break;
                }
                if (may_give_up && it >= kHelpAfter) return true;
                __builtin_amdgcn_s_sleep(2);
            }
            if (sm.bcast[2] && tid < k) {
                const int32_t *zr = reinterpret_cast<const int32_t *>(&p.zrec[size_t(pair) * k + tid]);
                const int s = ld_shared(zr);
                Z.sel[tid] = s;
                if (tid % nz == j) Z.zi[tid] = make_int4(s, ld_shared(zr + 1), ld_shared(zr + 2), ld_shared(zr + 3));
            }
        } else if (tid < k) {
            // the caller's selection
            int s = p.sel_in[size_t(pair) * k + tid];
            if (s >= m_b) { flag_error(p, kErrSelRange); s = -1; }
            Z.sel[tid] = s;
            if (tid % nz == j && s >= 0) {
                const int64_t off = p.block_off[pr * p.M_max + s];
                const int32_t w = span_word<T>(p, p.span_len[size_t(b) * p.M_max + s],
                                               p.block_rank ? p.block_rank[pr * p.M_max + s] : 0);
                Z.zi[tid] = make_int4(s, w, int32_t(off & 0xFFFFFFFF), int32_t(off >> 32));
            }
        }
        if (nc0 > 0) {
            if (wait_coarse_logits<T, D, G>(p, sm, pair, c_lo, nc0, tag, tid, may_give_up)) return true;
        } else {
            __syncthreads();
        }
    }
    SEKV_STAMP(p, sm, kTrSSelected);
    // the zoomed spans' blocks must lie inside the factor arena
    if (tid < k && tid % nz == j) {
        const int4 zi = Z.zi[tid];
        if (zi.x >= 0) {
            const int L = word_len(zi.y), rk = word_rk(zi.y), rv = word_rv(zi.y);
            const int64_t off = int64_t(uint32_t(zi.z)) | (int64_t(zi.w) << 32);
            const int64_t bytes = (int64_t(L) + 1 + D) * (rk + rv) * T::kBytes;
            if (L < 1 || rk == 0 || rv == 0 || off < 0 || (off & 15) || off + bytes > p.factors_bytes) {
                flag_error(p, kErrBlockRange);
                Z.zi[tid].x = -1;
            }
        }
    }
    __syncthreads();

    // 4. zoom the slot's spans (ranks j, j + n_zi, ...).  With one span, the first
    //    summary block is folded while its factor loads are in flight; with several,
    //    it is folded first, so its rows are not held in registers across the zooms.
    auto coarse0 = [&]() {
        if (nc0 > 0) coarse_block<T, D, G, NJ>(sm, cv, c_lo, nc0, k, pend, rgrp, tid);
    };
    auto zoom_ranked = [&](auto ranked_c, int32_t w, int64_t off, int tid, auto &&mid) {
        constexpr bool RANKED = decltype(ranked_c)::value;
        // 16-byte vectors per U row at the largest rank: 8..64 gives 1..8 (bf16) or 2..16
        // (f32); the block's own ranks r_K, r_V <= r travel in the span word
        const int ru = r * T::kBytes / 16;
        const int L = word_len(w), rk = word_rk(w), rv = word_rv(w);
        if constexpr (T::kBytes == 2) {
            switch (ru) {
                case 1: zoom_span<T, D, G, 1, RANKED>(p, sm, L, rk, rv, off, pend, tid, mid); break;
                case 2: zoom_span<T, D, G, 2, RANKED>(p, sm, L, rk, rv, off, pend, tid, mid); break;
                case 4: zoom_span<T, D, G, 4, RANKED>(p, sm, L, rk, rv, off, pend, tid, mid); break;
                default: zoom_span<T, D, G, 8, RANKED>(p, sm, L, rk, rv, off, pend, tid, mid); break;
            }
        } else {
            switch (ru) {
                case 2: zoom_span<T, D, G, 2, RANKED>(p, sm, L, rk, rv, off, pend, tid, mid); break;
                case 4: zoom_span<T, D, G, 4, RANKED>(p, sm, L, rk, rv, off, pend, tid, mid); break;
                case 8: zoom_span<T, D, G, 8, RANKED>(p, sm, L, rk, rv, off, pend, tid, mid); break;
                default: zoom_span<T, D, G, 16, RANKED>(p, sm, L, rk, rv, off, pend, tid, mid); break;
            }
        }
    };
    auto zoom_one = [&](int32_t w, int64_t off, int tid, auto &&mid) {
        if (p.block_rank) zoom_ranked(IC<1>{}, w, off, tid, mid);
        else zoom_ranked(IC<0>{}, w, off, tid, mid);
    };
    if (j + nz >= k) {
        const int4 zi = Z.zi[j < kMaxTopK ? j : 0];
        if (j < k && zi.x >= 0)
            zoom_one(zi.y, int64_t(uint32_t(zi.z)) | (int64_t(zi.w) << 32), tid, coarse0);
        else
            coarse0();
    } else {
        coarse0();
        for (int rk = j; rk < k; rk += nz) {
            // an opaque copy of the thread index keeps the zoom's per-thread address
            // arithmetic inside the loop rather than hoisted and alive across it
            int t;
            asm volatile("v_mov_b32 %0, %1" : "=v"(t) : "v"(tid));
            const int4 zi = Z.zi[rk];
            if (zi.x >= 0) zoom_one(zi.y, int64_t(uint32_t(zi.z)) | (int64_t(zi.w) << 32), t, [] {});
        }
    }
    // 5. the rest of the summary share (several blocks only when k is small)
    for (int c0 = c_lo + CB; c0 < c_hi && c0 < m_b; c0 += CB) {
        const int nc = min(min(CB, c_hi - c0), m_b - c0);
        load_rows<T, D, NJ>(cv, sv + size_t(c0) * GE::RB, nc, rgrp, col);
        if (wait_coarse_logits<T, D, G>(p, sm, pair, c0, nc, tag, tid, may_give_up)) return true;
        coarse_block<T, D, G, NJ>(sm, cv, c0, nc, k, pend, rgrp, tid);
    }
    __syncthreads();
    SEKV_STAMP(p, sm, kTrSCoarse);
    write_partial<T, D, G>(p, sm, pair, j, tid);
    stores_done_barrier();
    SEKV_STAMP(p, sm, kTrSPartial);
    count_partial<T, D, G>(p, sm, pair, tid, leave, tag);
    SEKV_STAMP(p, sm, kTrSMerged);
    return false;
}

// ---------------------------------------------------------------------------
// the persistent kernel
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__global__ void __launch_bounds__(NT, G == 8 ? 1 : 2) sekv_step_kernel(Params p) {
    __shared__ Smem<T, D, G> sm;
    const int tid = threadIdx.x;
    // the tag of this launch's published words, used as loaded: its first use is when
    // an item publishes or polls, so the load overlaps the first item's own loads
    const uint32_t tag = ld_shared(&p.hdr->epoch);
    const int n_items = p.end_share;
    // Workgroup w takes items w, w + grid, ...: routing items first (they never wait),
    // then share items, which wait only for routing chunks and take over any chunk whose
    // owner has not started (help_route), so no wait depends on residency.
    int helps = 0;                                      // help rounds of the current item
    bool left = false;                                  // counted out in its last share item
    for (int item = blockIdx.x; item < n_items;) {
        // an opaque copy of the thread index keeps per-thread address arithmetic inside
        // each item instead of alive across the whole loop (register pressure)
        int t;
        asm volatile("v_mov_b32 %0, %1" : "=v"(t) : "v"(tid));
        SEKV_TRACE_BEGIN(p, sm, item);
        if (item < p.end_route) {
            route_item<T, D, G>(p, sm, item / p.n_rc, item % p.n_rc, tag, t);
        } else {
            const int i = item - p.end_route;                // slot-major
            const int P = p.B * p.Hkv;
            const bool leave = item + p.grid >= n_items;
            if (share_item<T, D, G>(p, sm, i % P, i / P, tag, t, item == int(blockIdx.x) && helps == 0,
                                    helps < kMaxHelps, leave)) {
                help_route<T, D, G>(p, sm, i % P, tag, t);
                ++helps;
                continue;                                    // the same item again
            }
            left = leave;
        }
        SEKV_STAMP(p, sm, kTrEnd);
        __syncthreads();
        helps = 0;
        item += p.grid;
    }
    // a workgroup whose last item was a routing item (or that had none) counts itself out
    // here; the last workgroup out zeroes the counters and advances the epoch
    if (!left) {
        if (tid == 0) {
            const uint32_t prev = counter_add(&p.hdr->exit_count, 1u);
            sm.bcast[3] = (prev == uint32_t(p.grid - 1));
        }
        __syncthreads();
        if (sm.bcast[3]) shutdown(p, tag, tid);
    }
}

}  // namespace
}  // namespace sekv
