// SeKV decode step for gfx950: one persistent kernel over typed work items.
//
// Work items (per (sequence b, KV head g) "pair"):
//   route   chunk of 64 spans: routing scores in float64 (eq. routing_gate with the
//           coarse mean key as summary), local top-k candidates, and -- fused mode --
//           the coarse softmax partial of the chunk's non-candidate spans, so each
//           summary row (k_bar, v_bar) is read from HBM once.  The last route item of a
//           pair merges the candidates into the pair's selection (Sec. 3.3 budget rule)
//           and adds the coarse partial of the candidates that lost.
//   anchor  chunk of 128 full-resolution tokens: softmax partial.
//   zoom    one selected span: its keys/values are U diag(sigma) V^T (eq.
//           key_reconstruction); scores and the value sum are taken through the
//           factors so no reconstructed token is ever written to memory.
// Every partial (max, sum, weighted value sum) lands in a fixed slot; the item that
// completes a pair's last slot merges them in slot order into the output (one softmax
// over the mixed-resolution memory, Sec. 3.3).  No floating-point atomics: results are
// bitwise deterministic.
//
// Scheduling: items [0, S) are taken statically by workgroups [0, S) where S counts
// only items that never wait; the rest are handed out by an atomic ticket.  A zoom
// item waits for its pair's selection, which is produced by route items whose index is
// lower than any ticket, hence already running: the wait always ends (it is bounded
// anyway and flags the workspace on timeout).  The last workgroup to leave zeroes the
// counters, so the workspace is ready for the next launch.
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
// cross-workgroup signalling (agent scope)
// ---------------------------------------------------------------------------
__device__ inline uint32_t atomic_add_acqrel(uint32_t *p, uint32_t v) {
    return __hip_atomic_fetch_add(p, v, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline uint32_t atomic_add_relaxed(uint32_t *p, uint32_t v) {
    return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline uint32_t load_acquire(const uint32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void store_release(uint32_t *p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void fence_acquire() { __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent"); }
__device__ inline void fence_release() { __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent"); }
__device__ inline void flag_error(const Params &p, int32_t bit) {
    __hip_atomic_fetch_or(&p.hdr->error, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
// shared memory
// ---------------------------------------------------------------------------
template <class T, int D, int G>
struct Smem {
    static constexpr int kRowS = D * T::kBytes + 16;     // padded LDS row stride
    struct Rows {                                        // route / summary / anchor items
        union { double qd[G][D]; float qf[G][D]; } q;    // query: float64 (routing) / float32
        unsigned char kb[CR * kRowS];                    // key rows
        unsigned char vb[CR * kRowS];                    // value rows
        double lg[G][CR];                                // routing scores, natural units
        float lw[G][CR];                                 // scores, base-2 units (-inf = excluded)
        float pw[G][CR];                                 // exp2(lw - running max)
        int32_t excl[CR];                                // excluded span / loser index
    };
    struct Zoom {                                        // zoom item
        float qf[G][D];
        unsigned char vt[kMaxTopK * kRowS];              // Vt_V rows
        float zs[G][kZoomBlock];                         // token scores, then weights
        float w[G][kMaxTopK];                            // scale*log2e*sigma_K*(Vt_K q)
        float y[G][kMaxTopK];                            // (p^T U_V) * sigma_V
        float red[4][G][kMaxTopK];                       // per-wave partial sums of y
        float sig[2][kMaxTopK];                          // sigma_K, sigma_V
    };
    struct Merge {                                       // selection merge
        uint64_t key[kMergeBuf];
        uint32_t idx[kMergeBuf];
        int32_t sel[kMaxTopK];
    };
    struct Final {                                       // softmax merge
        float wgt[kMergeBuf][G];
        float M[G], L[G];
    };
    union {
        Rows rows;
        Zoom zoom;
        Merge merge;
        Final fin;
    } u;
    float m_run[G], l_run[G], scale_old[G];              // online softmax state
    int32_t bcast[4];
};

// ---------------------------------------------------------------------------
// helpers on LDS rows
// ---------------------------------------------------------------------------
template <class T, int D>
__device__ inline void copy_rows_to_lds(unsigned char *dst, const unsigned char *src, int nrows,
                                        int tid) {
    constexpr int RV = D * T::kBytes / 16;             // 16-byte vectors per row
    constexpr int RS = D * T::kBytes + 16;
    for (int v = tid; v < nrows * RV; v += NT) {
        const int row = v / RV, col = v % RV;
        *reinterpret_cast<uint4 *>(dst + size_t(row) * RS + col * 16) =
            ld16(src + size_t(row) * (D * T::kBytes) + col * 16);
    }
}

template <class T, int D>
__device__ inline float lds_elem(const unsigned char *rows, int row, int col) {
    constexpr int RS = D * T::kBytes + 16;
    return T::load1(rows + size_t(row) * RS, col);
}

// Online coarse accumulation of one batch of <= CR rows held in LDS (vb, lw).
// Each thread owns outputs o = tid + NT*u (head o / D, dim o % D), accumulated in acc[].
template <class T, int D, int G>
__device__ inline void online_batch(Smem<T, D, G> &sm, int nrows, float *acc, int tid) {
    auto &R = sm.u.rows;
    const int wave = tid >> 6, lane = tid & 63;
    for (int hl = wave; hl < G; hl += 4) {
        float x = (lane < nrows) ? R.lw[hl][lane] : -INFINITY;
        const float mb = wave_max(x);
        const float mo = sm.m_run[hl];
        const float mn = fmaxf(mo, mb);
        const float pw = (mn == -INFINITY) ? 0.0f : safe_exp2(x - mn);
        if (lane < CR) R.pw[hl][lane] = pw;
        const float lb = wave_sum(pw);
        if (lane == 0) {
            const float so = (mn == -INFINITY) ? 1.0f : safe_exp2(mo - mn);
            sm.scale_old[hl] = so;
            sm.l_run[hl] = sm.l_run[hl] * so + lb;
            sm.m_run[hl] = mn;
        }
    }
    __syncthreads();
    constexpr int NOUT = (G * D + NT - 1) / NT;
#pragma unroll
    for (int u = 0; u < NOUT; ++u) {
        const int o = tid + NT * u;
        if (o < G * D) {
            const int hl = o / D, d = o % D;
            float a = acc[u] * sm.scale_old[hl];
            for (int i = 0; i < nrows; ++i) a += R.pw[hl][i] * lds_elem<T, D>(R.vb, i, d);
            acc[u] = a;
        }
    }
    __syncthreads();
}

template <class T, int D, int G>
__device__ inline void online_reset(Smem<T, D, G> &sm, float *acc, int tid) {
    auto &R = sm.u.rows;
    if (tid < G) { sm.m_run[tid] = -INFINITY; sm.l_run[tid] = 0.0f; sm.scale_old[tid] = 1.0f; }
    constexpr int NOUT = (G * D + NT - 1) / NT;
#pragma unroll
    for (int u = 0; u < NOUT; ++u) acc[u] = 0.0f;
    __syncthreads();
}

// Write a finished partial (m, l in LDS state; o in acc) to its slot.
template <class T, int D, int G>
__device__ inline void write_partial(const Params &p, Smem<T, D, G> &sm, int pair, int slot,
                                     const float *acc, int tid) {
    auto &R = sm.u.rows;
    const size_t base = (size_t(pair) * p.n_slots + slot) * G;
    if (tid < G) {
        p.part_ml[(base + tid) * 2 + 0] = sm.m_run[tid];
        p.part_ml[(base + tid) * 2 + 1] = sm.l_run[tid];
    }
    constexpr int NOUT = (G * D + NT - 1) / NT;
#pragma unroll
    for (int u = 0; u < NOUT; ++u) {
        const int o = tid + NT * u;
        if (o < G * D) p.part_o[base * D + o] = acc[u];
    }
}

// ---------------------------------------------------------------------------
// final softmax merge of one pair (slot order fixed => deterministic)
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__device__ void final_merge(const Params &p, Smem<T, D, G> &sm, int pair, int tid) {
    auto &F = sm.u.fin;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    const int ns = p.n_slots;
    const bool use_losers = (p.mode == kModeFused);
    const float *ml = p.part_ml + size_t(pair) * ns * G * 2;
    const int wave = tid >> 6, lane = tid & 63;
    for (int hl = wave; hl < G; hl += 4) {
        float mx = -INFINITY;
        for (int s = lane; s < ns; s += 64) {
            if (s == p.slot_losers && !use_losers) continue;
            if (ml[(s * G + hl) * 2 + 1] > 0.0f) mx = fmaxf(mx, ml[(s * G + hl) * 2]);
        }
        mx = wave_max(mx);
        float lsum = 0.0f;
        for (int s = lane; s < ns; s += 64) {
            float wgt = 0.0f;
            const bool on = !(s == p.slot_losers && !use_losers);
            if (on && ml[(s * G + hl) * 2 + 1] > 0.0f) {
                wgt = exp2f(ml[(s * G + hl) * 2] - mx);
                lsum += wgt * ml[(s * G + hl) * 2 + 1];
            }
            F.wgt[s][hl] = wgt;
        }
        // fixed-order sum over lanes (deterministic for a given ns)
        lsum = wave_sum(lsum);
        if (lane == 0) { F.M[hl] = mx; F.L[hl] = lsum; }
    }
    __syncthreads();
    const float *po = p.part_o + size_t(pair) * ns * G * D;
    constexpr int NOUT = (G * D + NT - 1) / NT;
#pragma unroll
    for (int u = 0; u < NOUT; ++u) {
        const int o = tid + NT * u;
        if (o < G * D) {
            const int hl = o / D, d = o % D;
            float a = 0.0f;
            for (int s = 0; s < ns; ++s) {
                const float wgt = F.wgt[s][hl];
                if (wgt != 0.0f) a += wgt * po[(size_t(s) * G + hl) * D + d];
            }
            const float L = F.L[hl];
            const float r = (L > 0.0f) ? a / L : 0.0f;
            const size_t oi = (size_t(b) * p.Hq + size_t(g) * G + hl) * D + d;
            if (p.out_f32) reinterpret_cast<float *>(p.out)[oi] = r;
            else reinterpret_cast<uint16_t *>(p.out)[oi] = f32_to_bf16_rne(r);
        }
    }
}

// Count one finished partial of `pair`; the item completing the pair merges.
template <class T, int D, int G>
__device__ inline void finish_partial(const Params &p, Smem<T, D, G> &sm, int pair, int n_parts,
                                      int tid) {
    __syncthreads();
    if (tid == 0) {
        fence_release();
        const uint32_t prev = atomic_add_acqrel(&p.part_cnt[pair], 1u);
        sm.bcast[0] = (prev == uint32_t(n_parts - 1));
    }
    __syncthreads();
    if (sm.bcast[0]) {
        fence_acquire();
        final_merge<T, D, G>(p, sm, pair, tid);
    }
    __syncthreads();
}

// ---------------------------------------------------------------------------
// selection merge: the last route item of a pair orders all candidates
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__device__ inline void bitonic_sort_lds(Smem<T, D, G> &sm, int tid) {
    auto &M = sm.u.merge;
    for (int size = 2; size <= kMergeBuf; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int t = tid; t < kMergeBuf / 2; t += NT) {
                const int i = (t / stride) * 2 * stride + (t % stride);
                const int j = i + stride;
                const bool up = (i & size) == 0;        // up: better elements first
                const uint64_t ki = M.key[i], kj = M.key[j];
                const uint32_t ii = M.idx[i], ij = M.idx[j];
                const bool swap = up ? better(kj, ij, ki, ii) : better(ki, ii, kj, ij);
                if (swap) { M.key[i] = kj; M.idx[i] = ij; M.key[j] = ki; M.idx[j] = ii; }
            }
            __syncthreads();
        }
    }
}

template <class T, int D, int G>
__device__ void merge_selection(const Params &p, Smem<T, D, G> &sm, int pair, int tid) {
    auto &M = sm.u.merge;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    const int k = p.k;
    int m_b = p.n_spans[b];
    m_b = m_b < 0 ? 0 : (m_b > p.M_max ? p.M_max : m_b);
    const int kc = p.kc;
    const int n_cand = p.n_rc * kc;
    constexpr int kHead = kMaxTopK;                       // running best occupies [0, 64)
    constexpr int kFill = kMergeBuf - kMaxTopK;
    for (int i = tid; i < kMergeBuf; i += NT) { M.key[i] = 0; M.idx[i] = kInvalidIdx - i; }
    __syncthreads();
    for (int base = 0; base < n_cand; base += kFill) {
        for (int i = tid; i < kFill; i += NT) {
            const int c = base + i;
            uint64_t key = 0;
            uint32_t idx = kInvalidIdx - (kHead + i);
            if (c < n_cand) {
                const int chunk = c / kc, j = c % kc;
                const int cnt = __hip_atomic_load(&p.cand_cnt[pair * p.n_rc + chunk],
                                                  __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (j < cnt) {
                    const size_t ci = (size_t(pair) * p.n_rc + chunk) * kc + j;
                    key = p.cand_key[ci];
                    idx = uint32_t(p.cand_idx[ci]);
                }
            }
            M.key[kHead + i] = key;
            M.idx[kHead + i] = idx;
        }
        __syncthreads();
        bitonic_sort_lds<T, D, G>(sm, tid);
        // keep the best k; invalidate [k, 64) so they cannot re-enter
        for (int i = tid; i < kHead; i += NT)
            if (i >= k) { M.key[i] = 0; M.idx[i] = kInvalidIdx - i; }
        __syncthreads();
    }
    const int take = k < m_b ? k : m_b;
    for (int j = tid; j < k; j += NT) {
        const int s = (j < take && M.idx[j] < 0x80000000u) ? int(M.idx[j]) : -1;
        M.sel[j] = s;
        if (p.sel_out) p.sel_out[size_t(pair) * k + j] = s;
        if (p.mode == kModeFused) p.sel_ws[size_t(pair) * k + j] = s;
    }
    __syncthreads();
    if (p.mode == kModeFused && tid == 0) {
        fence_release();
        store_release(&p.sel_ready[pair], 1u);
    }
}

// Coarse partial over the candidates that lost the selection (fused mode).
template <class T, int D, int G>
__device__ void losers_partial(const Params &p, Smem<T, D, G> &sm, int pair, int tid) {
    auto &R = sm.u.rows;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    const int k = p.k, kc = p.kc;
    // selection (from workspace; this workgroup wrote it)
    __shared__ int32_t sel_l[kMaxTopK];
    for (int j = tid; j < kMaxTopK; j += NT) sel_l[j] = (j < k) ? p.sel_ws[size_t(pair) * k + j] : -1;
    __syncthreads();
    constexpr int NOUT = (G * D + NT - 1) / NT;
    float acc[NOUT];
    online_reset<T, D, G>(sm, acc, tid);
    const unsigned char *sv = reinterpret_cast<const unsigned char *>(p.sum_v) +
                              (size_t(b) * p.Hkv + g) * size_t(p.M_max) * D * T::kBytes;
    const int n_cand = p.n_rc * kc;
    for (int base = 0; base < n_cand; base += CR) {
        // gather up to CR losers of this candidate window
        if (tid < CR) {
            const int c = base + tid;
            int idx = -1;
            if (c < n_cand) {
                const int chunk = c / kc, j = c % kc;
                const int cnt = p.cand_cnt[pair * p.n_rc + chunk];
                if (j < cnt) {
                    const size_t ci = (size_t(pair) * p.n_rc + chunk) * kc + j;
                    idx = p.cand_idx[ci];
                    bool chosen = false;
                    for (int q = 0; q < k; ++q) chosen |= (sel_l[q] == idx);
                    if (chosen) idx = -1;
                    else
                        for (int hl = 0; hl < G; ++hl)
                            R.lw[hl][tid] = p.cand_lg[ci * G + hl] * kLog2e;
                }
            }
            R.excl[tid] = idx;
            if (idx < 0)
                for (int hl = 0; hl < G; ++hl) R.lw[hl][tid] = -INFINITY;
        }
        __syncthreads();
        // rows: v_bar of each loser (zero rows for empty slots are never weighted)
        constexpr int RV = D * T::kBytes / 16;
        constexpr int RS = D * T::kBytes + 16;
        for (int v = tid; v < CR * RV; v += NT) {
            const int row = v / RV, col = v % RV;
            const int idx = R.excl[row];
            uint4 val = make_uint4(0, 0, 0, 0);
            if (idx >= 0) val = ld16(sv + size_t(idx) * D * T::kBytes + col * 16);
            *reinterpret_cast<uint4 *>(R.vb + size_t(row) * RS + col * 16) = val;
        }
        __syncthreads();
        online_batch<T, D, G>(sm, CR, acc, tid);
    }
    write_partial<T, D, G>(p, sm, pair, p.slot_losers, acc, tid);
}

// ---------------------------------------------------------------------------
// route / summary item: one chunk of CR spans of a pair
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__device__ void route_item(const Params &p, Smem<T, D, G> &sm, int pair, int chunk, int tid) {
    auto &R = sm.u.rows;
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

    // 1. stage query (float64) and summary rows
    if (need_dots) {
        for (int i = tid; i < G * D; i += NT) {
            const int hl = i / D, d = i % D;
            R.q.qd[hl][d] = double(T::load1(p.q, (size_t(b) * p.Hq + size_t(g) * G + hl) * D + d));
        }
        copy_rows_to_lds<T, D>(R.kb, reinterpret_cast<const unsigned char *>(p.sum_k) +
                                         row0 * D * T::kBytes, nv, tid);
    }
    if (need_coarse)
        copy_rows_to_lds<T, D>(R.vb, reinterpret_cast<const unsigned char *>(p.sum_v) +
                                         row0 * D * T::kBytes, nv, tid);
    __syncthreads();

    // 2. routing scores: float64, products exact, summed left to right over d,
    //    then (s * scale) + ln|S| as two separately rounded operations.
    for (int t = tid; t < G * CR; t += NT) {
        const int hl = t / CR, i = t % CR;
        double sc = -INFINITY;
        if (i < nv) {
            if (need_dots) {
                constexpr int VEC = T::kVec;
                constexpr int RS = D * T::kBytes + 16;
                const unsigned char *row = R.kb + size_t(i) * RS;
                double acc = 0.0;
#pragma unroll 4
                for (int c = 0; c < D / VEC; ++c) {
                    float f[VEC];
                    T::unpack(*reinterpret_cast<const uint4 *>(row + c * 16), f);
#pragma unroll
                    for (int e = 0; e < VEC; ++e) acc = __builtin_fma(R.q.qd[hl][c * VEC + e], double(f[e]), acc);
                }
                {
#pragma clang fp contract(off)
                    const double scaled = acc * p.scale;
                    sc = scaled + p.span_logsize[size_t(b) * p.M_max + s0 + i];
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

    // 3. exclusions: local top-k candidates (route/fused) or the given selection (attend)
    if (!attend) {
        // one wave sorts the chunk's CR = 64 (key, idx) pairs with a bitonic network
        if (tid < 64) {
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
            // lane j holds the j-th best
            const int kc = min(p.kc, nv);
            R.excl[i] = 0;
            __builtin_amdgcn_wave_barrier();
            if (i < kc) {
                const size_t ci = (size_t(pair) * p.n_rc + chunk) * p.kc + i;
                p.cand_key[ci] = key;
                p.cand_idx[ci] = int32_t(idx);
                const int li = int(idx) - s0;
                for (int hl = 0; hl < G; ++hl) p.cand_lg[ci * G + hl] = float(R.lg[hl][li]);
            }
            if (i == 0) p.cand_cnt[pair * p.n_rc + chunk] = kc;
            __builtin_amdgcn_wave_barrier();
            if (i < kc) R.excl[int(idx) - s0] = 1;
        }
    } else {
        if (tid < CR) {
            int ex = 0;
            for (int j = 0; j < p.k; ++j) ex |= (p.sel_in[size_t(pair) * p.k + j] == s0 + tid);
            R.excl[tid] = ex;
        }
    }
    __syncthreads();

    // 4. coarse partial over the chunk's remaining spans
    if (need_coarse) {
        for (int t = tid; t < G * CR; t += NT) {
            const int hl = t / CR, i = t % CR;
            R.lw[hl][i] = (i < nv && !R.excl[i]) ? float(R.lg[hl][i] * kLog2eD) : -INFINITY;
        }
        constexpr int NOUT = (G * D + NT - 1) / NT;
        float acc[NOUT];
        online_reset<T, D, G>(sm, acc, tid);
        online_batch<T, D, G>(sm, nv, acc, tid);
        write_partial<T, D, G>(p, sm, pair, p.slot_route0 + chunk, acc, tid);
    }

    // 5. the last route item of the pair merges the candidates into the selection
    if (!attend) {
        __syncthreads();
        if (tid == 0) {
            fence_release();
            const uint32_t prev = atomic_add_acqrel(&p.route_cnt[pair], 1u);
            sm.bcast[1] = (prev == uint32_t(p.n_rc - 1));
        }
        __syncthreads();
        if (sm.bcast[1]) {
            fence_acquire();
            merge_selection<T, D, G>(p, sm, pair, tid);
            __syncthreads();
            if (p.mode == kModeFused) {
                losers_partial<T, D, G>(p, sm, pair, tid);
            }
        }
        __syncthreads();
        if (p.mode == kModeFused) {
            const int n_parts = p.n_ac + p.n_rc + 1 + p.k;
            // this chunk's coarse partial, plus the losers partial if this item merged
            finish_partial<T, D, G>(p, sm, pair, n_parts, tid);
            if (sm.bcast[1]) finish_partial<T, D, G>(p, sm, pair, n_parts, tid);
        }
    } else {
        finish_partial<T, D, G>(p, sm, pair, p.n_ac + p.n_rc + p.k, tid);
    }
}

// ---------------------------------------------------------------------------
// anchor item: kAnchorChunk full-resolution tokens of a pair, in batches of CR rows
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__device__ void anchor_item(const Params &p, Smem<T, D, G> &sm, int pair, int chunk, int tid) {
    auto &R = sm.u.rows;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    int A = p.n_anchors[b];
    A = A < 0 ? 0 : (A > p.A_max ? p.A_max : A);
    const int a0 = chunk * kAnchorChunk;
    const int na = max(0, min(kAnchorChunk, A - a0));
    for (int i = tid; i < G * D; i += NT) {
        const int hl = i / D, d = i % D;
        R.q.qf[hl][d] = T::load1(p.q, (size_t(b) * p.Hq + size_t(g) * G + hl) * D + d);
    }
    constexpr int NOUT = (G * D + NT - 1) / NT;
    float acc[NOUT];
    online_reset<T, D, G>(sm, acc, tid);
    const size_t base = ((size_t(b) * p.Hkv + g) * size_t(p.A_max) + a0) * D * T::kBytes;
    const unsigned char *ak = reinterpret_cast<const unsigned char *>(p.anchor_k) + base;
    const unsigned char *av = reinterpret_cast<const unsigned char *>(p.anchor_v) + base;
    for (int t0 = 0; t0 < na; t0 += CR) {
        const int nb = min(CR, na - t0);
        copy_rows_to_lds<T, D>(R.kb, ak + size_t(t0) * D * T::kBytes, nb, tid);
        copy_rows_to_lds<T, D>(R.vb, av + size_t(t0) * D * T::kBytes, nb, tid);
        __syncthreads();
        for (int t = tid; t < G * CR; t += NT) {
            const int hl = t / CR, i = t % CR;
            float s = -INFINITY;
            if (i < nb) {
                constexpr int VEC = T::kVec;
                constexpr int RS = D * T::kBytes + 16;
                const unsigned char *row = R.kb + size_t(i) * RS;
                float a = 0.0f;
#pragma unroll 4
                for (int c = 0; c < D / VEC; ++c) {
                    float f[VEC];
                    T::unpack(*reinterpret_cast<const uint4 *>(row + c * 16), f);
#pragma unroll
                    for (int e = 0; e < VEC; ++e) a += R.q.qf[hl][c * VEC + e] * f[e];
                }
                s = a * p.scale_log2;
            }
            R.lw[hl][i] = s;
        }
        __syncthreads();
        online_batch<T, D, G>(sm, nb, acc, tid);
    }
    write_partial<T, D, G>(p, sm, pair, chunk, acc, tid);
    const int n_parts = (p.mode == kModeFused) ? p.n_ac + p.n_rc + 1 + p.k : p.n_ac + p.n_rc + p.k;
    finish_partial<T, D, G>(p, sm, pair, n_parts, tid);
}

// ---------------------------------------------------------------------------
// zoom item: one selected span, attended through its factors
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__device__ void zoom_item(const Params &p, Smem<T, D, G> &sm, int pair, int j, int tid) {
    auto &Z = sm.u.zoom;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    const int r = p.r;
    // which span
    if (tid == 0) {
        int S;
        if (p.mode == kModeFused) {
            uint32_t n = 0;
            while (load_acquire(&p.sel_ready[pair]) == 0u) {
                __builtin_amdgcn_s_sleep(2);
                if (++n > kSpinLimit) { flag_error(p, kErrSpinTimeout); break; }
            }
            S = __hip_atomic_load(&p.sel_ws[size_t(pair) * p.k + j], __ATOMIC_RELAXED,
                                  __HIP_MEMORY_SCOPE_AGENT);
            if (n > kSpinLimit) S = -1;
        } else {
            S = p.sel_in[size_t(pair) * p.k + j];
        }
        int m_b = p.n_spans[b];
        m_b = m_b < 0 ? 0 : (m_b > p.M_max ? p.M_max : m_b);
        if (S >= m_b) { flag_error(p, kErrSelRange); S = -1; }
        int L = 0;
        int64_t off = 0;
        if (S >= 0) {
            L = p.span_len[size_t(b) * p.M_max + S];
            off = p.block_off[(size_t(b) * p.Hkv + g) * p.M_max + S];
            const int64_t bytes = (2 * int64_t(L) * r + 2 * r + 2 * int64_t(r) * D) * T::kBytes;
            if (L < 1 || off < 0 || (off & 15) || off + bytes > p.factors_bytes) {
                flag_error(p, kErrBlockRange);
                S = -1;
            }
        }
        sm.bcast[0] = S;
        sm.bcast[1] = L;
        sm.bcast[2] = int32_t(off & 0xFFFFFFFF);
        sm.bcast[3] = int32_t(off >> 32);
    }
    if (p.mode == kModeFused) fence_acquire();
    __syncthreads();
    const int S = sm.bcast[0];
    const int L = sm.bcast[1];
    const int64_t off = int64_t(uint32_t(sm.bcast[2])) | (int64_t(sm.bcast[3]) << 32);
    __syncthreads();

    constexpr int NOUT = (G * D + NT - 1) / NT;
    float acc[NOUT];
    online_reset<T, D, G>(sm, acc, tid);
    const int slot = p.slot_zoom0 + j;
    if (S >= 0) {
        constexpr int VEC = T::kVec;
        constexpr int RV = D * T::kBytes / 16;          // vectors per d-row
        constexpr int RS = D * T::kBytes + 16;
        const int RU = r * T::kBytes / 16;              // vectors per U row
        const unsigned char *UK = p.factors + off;
        const unsigned char *sK = UK + size_t(L) * r * T::kBytes;
        const unsigned char *VtK = sK + size_t(r) * T::kBytes;
        const unsigned char *UV = VtK + size_t(r) * D * T::kBytes;
        const unsigned char *sV = UV + size_t(L) * r * T::kBytes;
        const unsigned char *VtV = sV + size_t(r) * T::kBytes;

        // stage q (float), sigmas, and Vt_V rows (into kb) for the final projection
        for (int i = tid; i < G * D; i += NT) {
            const int hl = i / D, d = i % D;
            Z.qf[hl][d] = T::load1(p.q, (size_t(b) * p.Hq + size_t(g) * G + hl) * D + d);
        }
        if (tid < r) {
            Z.sig[0][tid] = T::load1(sK, tid);
            Z.sig[1][tid] = T::load1(sV, tid);
        }
        copy_rows_to_lds<T, D>(Z.vt, VtV, r, tid);
        __syncthreads();

        // w[h][i] = scale*log2e * sigma_K[i] * (Vt_K[i] . q_h)
        for (int v0 = 0; v0 < r * RV; v0 += NT) {
            const int v = v0 + tid;
            float part[G];
#pragma unroll
            for (int hl = 0; hl < G; ++hl) part[hl] = 0.0f;
            const int row = v / RV, col = v % RV;
            if (v < r * RV) {
                float f[VEC];
                T::unpack(ld16(VtK + size_t(row) * D * T::kBytes + col * 16), f);
#pragma unroll
                for (int hl = 0; hl < G; ++hl)
#pragma unroll
                    for (int e = 0; e < VEC; ++e) part[hl] += Z.qf[hl][col * VEC + e] * f[e];
            }
#pragma unroll
            for (int o = 1; o < RV; o <<= 1)
#pragma unroll
                for (int hl = 0; hl < G; ++hl) part[hl] += __shfl_xor(part[hl], o, 64);
            if (v < r * RV && col == 0)
#pragma unroll
                for (int hl = 0; hl < G; ++hl) Z.w[hl][row] = part[hl] * Z.sig[0][row] * p.scale_log2;
        }
        __syncthreads();

        // token blocks: scores via U_K, online softmax, y accumulation via U_V
        float yacc[G][VEC];
#pragma unroll
        for (int hl = 0; hl < G; ++hl)
#pragma unroll
            for (int e = 0; e < VEC; ++e) yacc[hl][e] = 0.0f;
        const int col = tid % RU;                       // fixed per thread (NT % RU == 0)
        int nb_max = (8 * NT) / RU;
        if (nb_max > kZoomBlock) nb_max = kZoomBlock;
        const int wave = tid >> 6, lane = tid & 63;
        for (int t0 = 0; t0 < L; t0 += nb_max) {
            const int nb = min(nb_max, L - t0);
            uint4 uv[8];
            {
                uint4 uk[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int tok = (tid + NT * u) / RU;
                    if (tok < nb) uk[u] = ld16(UK + (size_t(t0 + tok) * r) * T::kBytes + col * 16);
                }
                // scores of the block's tokens
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
                            for (int e = 0; e < VEC; ++e) part[hl] += f[e] * Z.w[hl][col * VEC + e];
                    }
                    for (int o = 1; o < RU; o <<= 1)
#pragma unroll
                        for (int hl = 0; hl < G; ++hl) part[hl] += __shfl_xor(part[hl], o, 64);
                    if (tok < nb && col == 0)
#pragma unroll
                        for (int hl = 0; hl < G; ++hl) Z.zs[hl][tok] = part[hl];
                }
            }
            // value-side rows: in flight while the block's softmax weights are formed
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int tok = (tid + NT * u) / RU;
                if (tok < nb) uv[u] = ld16(UV + (size_t(t0 + tok) * r) * T::kBytes + col * 16);
            }
            __syncthreads();
            // block max and weights (wave hl handles head hl)
            for (int hl = wave; hl < G; hl += 4) {
                float mx = -INFINITY;
                for (int t = lane; t < nb; t += 64) mx = fmaxf(mx, Z.zs[hl][t]);
                mx = wave_max(mx);
                const float mo = sm.m_run[hl];
                const float mn = fmaxf(mo, mx);
                float ls = 0.0f;
                for (int t = lane; t < nb; t += 64) {
                    const float w = exp2f(Z.zs[hl][t] - mn);
                    Z.zs[hl][t] = w;
                    ls += w;
                }
                ls = wave_sum(ls);
                if (lane == 0) {
                    const float so = safe_exp2(mo - mn);
                    sm.scale_old[hl] = so;
                    sm.l_run[hl] = sm.l_run[hl] * so + ls;
                    sm.m_run[hl] = mn;
                }
            }
            __syncthreads();
#pragma unroll
            for (int hl = 0; hl < G; ++hl) {
                const float so = sm.scale_old[hl];
#pragma unroll
                for (int e = 0; e < VEC; ++e) yacc[hl][e] *= so;
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int v = tid + NT * u;
                const int tok = v / RU;
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
        // reduce yacc over the lanes sharing `col` (lane ^ RU, 2RU, ... within a wave)
        for (int o = RU; o < 64; o <<= 1)
#pragma unroll
            for (int hl = 0; hl < G; ++hl)
#pragma unroll
                for (int e = 0; e < VEC; ++e) yacc[hl][e] += __shfl_xor(yacc[hl][e], o, 64);
        if (lane < RU)
#pragma unroll
            for (int hl = 0; hl < G; ++hl)
#pragma unroll
                for (int e = 0; e < VEC; ++e) Z.red[wave][hl][col * VEC + e] = yacc[hl][e];
        __syncthreads();
        for (int t = tid; t < G * r; t += NT) {
            const int hl = t / r, i = t % r;
            const float y = Z.red[0][hl][i] + Z.red[1][hl][i] + Z.red[2][hl][i] + Z.red[3][hl][i];
            Z.y[hl][i] = y * Z.sig[1][i];
        }
        __syncthreads();
        // o[h][d] = sum_i y~[h][i] Vt_V[i][d]
#pragma unroll
        for (int u = 0; u < NOUT; ++u) {
            const int o = tid + NT * u;
            if (o < G * D) {
                const int hl = o / D, d = o % D;
                float a = 0.0f;
                for (int i = 0; i < r; ++i) a += Z.y[hl][i] * lds_elem<T, D>(Z.vt, i, d);
                acc[u] = a;
            }
        }
        (void)RS;
    }
    write_partial<T, D, G>(p, sm, pair, slot, acc, tid);
    const int n_parts = (p.mode == kModeFused) ? p.n_ac + p.n_rc + 1 + p.k : p.n_ac + p.n_rc + p.k;
    finish_partial<T, D, G>(p, sm, pair, n_parts, tid);
}

// ---------------------------------------------------------------------------
// the persistent kernel
// ---------------------------------------------------------------------------
template <class T, int D, int G>
__global__ void __launch_bounds__(NT, 2) sekv_step_kernel(Params p) {
    __shared__ Smem<T, D, G> sm;
    const int tid = threadIdx.x;
    const int n_items = p.end_zoom;
    // items that never wait are taken statically by the first workgroups
    const int n_static = min(p.grid, p.end_anchor);
    int item;
    if (int(blockIdx.x) < n_static) {
        item = blockIdx.x;
    } else {
        if (tid == 0) sm.bcast[2] = n_static + int(atomic_add_relaxed(&p.hdr->ticket, 1u));
        __syncthreads();
        item = sm.bcast[2];
        __syncthreads();
    }
    while (item < n_items) {
        if (item < p.end_route) {
            route_item<T, D, G>(p, sm, item / p.n_rc, item % p.n_rc, tid);
        } else if (item < p.end_anchor) {
            const int i = item - p.end_route;
            anchor_item<T, D, G>(p, sm, i / p.n_ac, i % p.n_ac, tid);
        } else {
            const int i = item - p.end_anchor;
            zoom_item<T, D, G>(p, sm, i / p.k, i % p.k, tid);
        }
        __syncthreads();
        if (tid == 0) sm.bcast[2] = n_static + int(atomic_add_relaxed(&p.hdr->ticket, 1u));
        __syncthreads();
        item = sm.bcast[2];
        __syncthreads();
    }
    // shutdown: the last workgroup out zeroes the counters for the next launch
    if (tid == 0) {
        const uint32_t prev = atomic_add_acqrel(&p.hdr->exit_count, 1u);
        sm.bcast[3] = (prev == uint32_t(p.grid - 1));
    }
    __syncthreads();
    if (sm.bcast[3]) {
        fence_acquire();
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
