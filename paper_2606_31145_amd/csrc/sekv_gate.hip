// Learned-routing selection for gfx950: the paper's own zoom decision.
//
//   q'_h  = W_h q_h                                   (Sec. 3.2 eq. query_projection)
//   x_h,S = q'_h . Kbar_h,S / sqrt(d') + ln|S|        (eq. routing_gate, before the sigmoid)
//   z_h,S = [x_h,S > ln(tau_h / (1 - tau_h))]         (Sec. 3.3 eq. zoom_decision; the sigmoid
//                                                      is strictly increasing)
// A span is a candidate of its (sequence, KV head) pair when any query head of the group
// votes for it; candidates are expanded in decreasing order of the largest voting gate
// (ties to the lower span index) while the expanded token count stays within the budget
// and the count within k (the budget cap of Sec. 3.3).
//
// Floating point, so that the selection is exact: q' is summed over d in float64 in
// index order (products of stored values are exact) and rounded once to float32; the
// gate's dot product is summed over d' in float64 in index order (float32 x stored
// products are exact); then one rounded multiply by 1/sqrt(d') and one rounded add of
// ln|S|, never contracted.
//
// Work: one workgroup per (pair, chunk of cr spans).  It projects the group's queries,
// scores its spans (one thread per span, all heads of the group in that thread, so the
// span's key needs no cross-thread step), ranks the chunk's spans in LDS (each entry
// counts the entries ahead of it: key descending, then index ascending) and publishes
// its best k as candidate records.  The last chunk of a pair to finish -- counted after
// its records are stored -- ranks the pair's candidates and applies the cap.  Nothing
// waits, so the launch completes whatever the residency.
#include "sekv_step.h"

namespace sekv {
namespace {

constexpr int GT = 256;                     // threads per workgroup
constexpr int kGateMaxD = 128;

constexpr int kSurv = (kGateMaxG * kGateMaxD + kGateMaxG * kGateMaxDr) * 8 / 16;

struct GateSmem {
    union {
        struct {
            double q64[kGateMaxG][kGateMaxD];   // the group's queries, widened
            double qp[kGateMaxG][kGateMaxDr];   // projected queries (float32 values)
        };
        uint4 surv[kSurv];                      // block survivors of the chunk ranking
    };
    uint4 ent[kGateMaxCand];                // entries {~span, key lo, key hi, |S|}
    uint4 top[64];                          // the best k of them, in expansion order
    int last;
};

// Expansion order: larger key first, then lower span index.  Every entry of a list has
// its own (key, index) -- entries without a vote have key 0 and a unique index, padding
// key 0 and an index with the top bit set -- so ranks are distinct.  Entries are stored
// as {~index, key lo, key hi, |S|}: (key, index) pairs then compare as the 96-bit numbers
// {key hi, key lo, ~index}, and the borrow out of mine - other says whether the other
// entry is ahead (count_ahead).

// Number of entries of list[0, n) ahead of me (four independent counts for ILP).
__device__ inline uint32_t rank_in(const uint4 *list, int n, const uint4 &me) {
    uint32_t r[4] = {0u, 0u, 0u, 0u};
    int o = 0;
    for (; o + 8 <= n; o += 8) {
        uint4 e[8];
#pragma unroll
        for (int w = 0; w < 8; ++w) e[w] = list[o + w];
#pragma unroll
        for (int w = 0; w < 8; ++w) count_ahead(r[w & 3], e[w], me.x, me.y, me.z);
    }
    for (; o < n; ++o) count_ahead(r[0], list[o], me.x, me.y, me.z);
    return r[0] + r[1] + r[2] + r[3];
}

// The k best entries of ent[0, n) into top[0, k), in expansion order.  When n is a
// multiple of 64 and the blocks' survivors fit `surv` (n_surv entries), each 64-entry
// block first keeps its own best k (a global top-k entry is among its block's top k),
// so the final ranking runs over (n / 64) k entries instead of n.
__device__ void top_k(const uint4 *ent, int n, uint4 *surv, int n_surv, uint4 *top, int k, int tid) {
    const bool filter = k < 64 && n % 64 == 0 && (n / 64) * k <= n_surv && n > 64;
    const uint4 *list = ent;
    int m = n;
    if (filter) {
        for (int i = tid; i < n; i += GT) {
            const uint4 me = ent[i];
            const int blk = i / 64;
            const uint32_t r = rank_in(ent + blk * 64, 64, me);
            if (r < uint32_t(k)) surv[blk * k + r] = me;
        }
        __syncthreads();
        list = surv;
        m = (n / 64) * k;
    }
    for (int i = tid; i < m; i += GT) {
        const uint4 me = list[i];
        const uint32_t r = rank_in(list, m, me);
        if (r < uint32_t(k)) top[r] = me;
    }
    __syncthreads();
}

template <class T>
__global__ void __launch_bounds__(GT) gate_kernel(GateParams p) {
    __shared__ GateSmem sm;
    const int tid = threadIdx.x;
    const int pair = blockIdx.x / p.n_rc, chunk = blockIdx.x % p.n_rc;
    const int b = pair / p.Hkv, g = pair % p.Hkv;
    const int G = p.G, d = p.d, dr = p.dr, k = p.k;
    const int s0 = chunk * p.cr;
    int m_b = p.n_spans[b];
    m_b = m_b < 0 ? 0 : (m_b > p.M_max ? p.M_max : m_b);

    constexpr int NWV = kGateMaxD * T::kBytes / 16;     // 16-byte vectors of a W row (max)
    constexpr int NKV = kGateMaxDr * T::kBytes / 16;    // ... of a routing-summary row (max)
    constexpr int HB = T::kBytes == 2 ? 4 : 2;          // summary rows in flight per thread
    const int nwv = d * T::kBytes / 16, nkv = dr * T::kBytes / 16;
    const unsigned char *kr0 = static_cast<const unsigned char *>(p.sum_route);

    // Every load that depends on nothing is issued first: the group's queries, this
    // thread's first projection row, the routing-summary rows of its first span.
    for (int i = tid; i < G * d; i += GT) {
        const int hl = i / d, j = i % d;
        sm.q64[hl][j] = double(T::load1(p.q, (size_t(b) * p.Hq + size_t(g) * G + hl) * d + j));
    }
    uint4 wv[NWV];
    if (tid < G * dr) {
        const unsigned char *w = static_cast<const unsigned char *>(p.proj) +
                                 ((size_t(g) * G) * dr + tid) * d * T::kBytes;
#pragma unroll
        for (int v = 0; v < NWV; ++v)
            if (v < nwv) wv[v] = ld16(w + v * 16);
    }
    // rows (span S, heads hl0 .. hl0 + HB - 1) of the routing summaries
    uint4 kv[HB][NKV];
    auto load_rows = [&](int S, int hl0) {
#pragma unroll
        for (int u = 0; u < HB; ++u) {
            if (hl0 + u < G) {
                const size_t row = (size_t(b) * p.Hq + size_t(g) * G + hl0 + u) * p.M_max + S;
#pragma unroll
                for (int v = 0; v < NKV; ++v)
                    if (v < nkv) kv[u][v] = ld16(kr0 + row * dr * T::kBytes + v * 16);
            }
        }
    };
    if (tid < p.cr && s0 + tid < m_b) load_rows(s0 + tid, 0);
    __syncthreads();

    // 1. q' = W q per head: float64 in index order, one rounding to float32
    for (int o = tid; o < G * dr; o += GT) {
        const int hl = o / dr, i = o % dr;
        if (o != tid) {                                     // more outputs than threads
            const unsigned char *w = static_cast<const unsigned char *>(p.proj) +
                                     ((size_t(g) * G + hl) * dr + i) * d * T::kBytes;
#pragma unroll
            for (int v = 0; v < NWV; ++v)
                if (v < nwv) wv[v] = ld16(w + v * 16);
        }
        double s = 0.0;
#pragma unroll
        for (int v = 0; v < NWV; ++v) {
            if (v < nwv) {
                float f[T::kVec];
                T::unpack(wv[v], f);
#pragma unroll
                for (int e = 0; e < T::kVec; ++e) s = fma(double(f[e]), sm.q64[hl][v * T::kVec + e], s);
            }
        }
        sm.qp[hl][i] = double(float(s));
    }
    __syncthreads();

    // 2. gates of this chunk's spans: thread t takes spans s0 + t, s0 + t + GT, ...; HB
    //    heads at a time, their dot products as independent float64 chains
    for (int t = tid; t < p.cr; t += GT) {
        const int S = s0 + t;
        uint64_t key = 0;
        int32_t len = 0;
        if (S < p.M_max) {
            const bool live = S < m_b;
            const double lns = live ? p.span_logsize[size_t(b) * p.M_max + S] : 0.0;
            bool vote = false;
            double best = 0.0;
            for (int hl0 = 0; hl0 < G; hl0 += HB) {
                if (live && (hl0 > 0 || t != tid)) load_rows(S, hl0);
                double sd[HB];
#pragma unroll
                for (int u = 0; u < HB; ++u) sd[u] = 0.0;
                if (live) {
#pragma unroll
                    for (int v = 0; v < NKV; ++v) {
                        if (v < nkv) {
#pragma unroll
                            for (int u = 0; u < HB; ++u) {
                                if (hl0 + u < G) {
                                    float f[T::kVec];
                                    T::unpack(kv[u][v], f);
#pragma unroll
                                    for (int e = 0; e < T::kVec; ++e)
                                        sd[u] = fma(sm.qp[hl0 + u][v * T::kVec + e], double(f[e]), sd[u]);
                                }
                            }
                        }
                    }
                }
#pragma unroll
                for (int u = 0; u < HB; ++u) {
                    const int hl = hl0 + u;
                    if (hl >= G) break;
                    const int h = g * G + hl;
                    double x = -INFINITY;
                    if (live) {
                        {
#pragma clang fp contract(off)
                            const double m = sd[u] * p.scale_r;
                            x = m + lns;
                        }
                        if (x > p.thr[h]) {
                            best = vote ? fmax(best, x) : x;
                            vote = true;
                        }
                    }
                    if (p.gate_out) p.gate_out[(size_t(b) * p.Hq + h) * p.M_max + S] = x;
                }
            }
            if (vote) {
                key = order_key(best);
                len = p.span_len[size_t(b) * p.M_max + S];
            }
        }
        sm.ent[t] = make_uint4(~(S < p.M_max ? uint32_t(S) : 0x80000000u | uint32_t(S)), uint32_t(key),
                               uint32_t(key >> 32), uint32_t(len));
    }
    __syncthreads();
    if (k <= 0) return;
    top_k(sm.ent, p.cr, sm.surv, kSurv, sm.top, k, tid);

    // 3. publish the chunk's best k (a chunk holds at least kGateMinChunk >= k spans)
    uint64_t *rec = p.cand + (size_t(pair) * p.n_rc + chunk) * size_t(k) * 2;
    if (tid < k) {
        const uint4 e = sm.top[tid];
        st_shared(rec + 2 * tid, (uint64_t(e.z) << 32) | e.y);
        st_shared(rec + 2 * tid + 1, (uint64_t(e.w) << 32) | e.x);
    }
    stores_done_barrier();
    if (tid == 0) sm.last = counter_add(&p.cnt[pair], 1u) == uint32_t(p.n_rc - 1);
    __syncthreads();
    if (!sm.last) return;

    // 4. the pair's last chunk: rank every candidate, then the budget cap
    const int nc = p.n_rc * k;
    const uint64_t *all = p.cand + size_t(pair) * p.n_rc * size_t(k) * 2;
    for (int i = tid; i < nc; i += GT) {
        const uint64_t kw = ld_shared(all + 2 * i), iw = ld_shared(all + 2 * i + 1);
        sm.ent[i] = make_uint4(uint32_t(iw), uint32_t(kw), uint32_t(kw >> 32), uint32_t(iw >> 32));
    }
    __syncthreads();
    top_k(sm.ent, nc, sm.surv, kSurv, sm.top, k, tid);
    // inclusive prefix of the expanded token counts over the first k entries (k <= 64:
    // one wave).  Votes sort ahead of non-votes (key 0), so the entries within budget
    // form a prefix of the expansion order.
    if (tid < 64) {
        const uint4 e = tid < k ? sm.top[tid] : make_uint4(0u, 0u, 0u, 0u);
        const bool vote = (e.y | e.z) != 0u;
        int64_t run = vote ? int64_t(max(int32_t(e.w), 0)) : 0;
        for (int off = 1; off < 64; off <<= 1) {
            const int64_t v = __shfl_up(run, off, 64);
            if (tid >= off) run += v;
        }
        if (tid < k) {
            const bool keep = vote && run <= p.budget;
            p.sel[size_t(pair) * k + tid] = keep ? int32_t(~e.x) : -1;
        }
    }
    if (tid == 0) st_shared(&p.cnt[pair], 0u);     // ready for the next launch
}

template <class T>
hipError_t launch_gate_typed(const GateParams &p, hipStream_t stream) {
    const unsigned grid = unsigned(p.B * p.Hkv * p.n_rc);
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL(gate_kernel<T>, dim3(grid), dim3(GT), 0, stream, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gate(const GateParams &p, int dtype, hipStream_t stream) {
    if (p.G > kGateMaxG || p.d > kGateMaxD || p.dr > kGateMaxDr || p.cr > kGateMaxCand ||
        p.k > 64 || p.n_rc * (p.k > 0 ? p.k : 1) > kGateMaxCand)
        return hipErrorInvalidValue;
    return dtype == SEKV_BF16 ? launch_gate_typed<BF16>(p, stream) : launch_gate_typed<F32>(p, stream);
}

}  // namespace sekv
