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
// span's key needs no cross-thread step), sorts the chunk in LDS (bitonic, key
// descending then index ascending) and publishes its best k as candidate records.  The
// last chunk of a pair to finish -- counted after its records are stored -- sorts the
// pair's candidates and applies the cap.  Nothing waits, so any residency completes.
#include "sekv_step.h"

namespace sekv {
namespace {

constexpr int GT = 256;                     // threads per workgroup
constexpr int kGateMaxD = 128;

struct GateSmem {
    double q64[kGateMaxG][kGateMaxD];       // the group's queries, widened
    double qp[kGateMaxG][kGateMaxDr];       // projected queries (float32 values)
    uint4 ent[kGateMaxCand];                // sort entries {key lo, key hi, span, |S|}
    int last;
};

// a precedes b: larger key first, then lower span index
__device__ inline bool ahead(const uint4 &a, const uint4 &b) {
    const uint64_t ka = (uint64_t(a.y) << 32) | a.x, kb = (uint64_t(b.y) << 32) | b.x;
    return ka > kb || (ka == kb && a.z < b.z);
}

// Bitonic sort of ent[0, n) (n a power of two) into expansion order.
__device__ void sort_entries(uint4 *ent, int n, int tid) {
    for (int kk = 2; kk <= n; kk <<= 1) {
        for (int j = kk >> 1; j > 0; j >>= 1) {
            for (int i = tid; i < n; i += GT) {
                const int o = i ^ j;
                if (o > i) {
                    const uint4 a = ent[i], b = ent[o];
                    const bool first_half = (i & kk) == 0;
                    if (first_half ? ahead(b, a) : ahead(a, b)) {
                        ent[i] = b;
                        ent[o] = a;
                    }
                }
            }
            __syncthreads();
        }
    }
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

    // 1. the group's queries, then q' = W q per head, float64 in index order, one rounding
    for (int i = tid; i < G * d; i += GT) {
        const int hl = i / d, j = i % d;
        sm.q64[hl][j] = double(T::load1(p.q, (size_t(b) * p.Hq + size_t(g) * G + hl) * d + j));
    }
    __syncthreads();
    for (int o = tid; o < G * dr; o += GT) {
        const int hl = o / dr, i = o % dr;
        const size_t row = (size_t(g) * G + hl) * dr + i;
        const unsigned char *w = static_cast<const unsigned char *>(p.proj) + row * d * T::kBytes;
        double s = 0.0;
        for (int j0 = 0; j0 < d; j0 += T::kVec) {
            float f[T::kVec];
            T::unpack(ld16(w + j0 * T::kBytes), f);
#pragma unroll
            for (int e = 0; e < T::kVec; ++e) s = fma(double(f[e]), sm.q64[hl][j0 + e], s);
        }
        sm.qp[hl][i] = double(float(s));
    }
    __syncthreads();

    // 2. gates of this chunk's spans: thread t takes spans s0 + t, s0 + t + GT, ...
    for (int t = tid; t < p.cr; t += GT) {
        const int S = s0 + t;
        uint64_t key = 0;
        int32_t len = 0;
        if (S < p.M_max) {
            const bool live = S < m_b;
            const double lns = live ? p.span_logsize[size_t(b) * p.M_max + S] : 0.0;
            bool vote = false;
            double best = 0.0;
            for (int hl = 0; hl < G; ++hl) {
                const int h = g * G + hl;
                double x = -INFINITY;
                if (live) {
                    const size_t row = (size_t(b) * p.Hq + h) * p.M_max + S;
                    const unsigned char *kr =
                        static_cast<const unsigned char *>(p.sum_route) + row * dr * T::kBytes;
                    double s = 0.0;
                    for (int i0 = 0; i0 < dr; i0 += T::kVec) {
                        float f[T::kVec];
                        T::unpack(ld16(kr + i0 * T::kBytes), f);
#pragma unroll
                        for (int e = 0; e < T::kVec; ++e) s = fma(sm.qp[hl][i0 + e], double(f[e]), s);
                    }
                    {
#pragma clang fp contract(off)
                        const double m = s * p.scale_r;
                        x = m + lns;
                    }
                    if (x > p.thr[h]) {
                        best = vote ? fmax(best, x) : x;
                        vote = true;
                    }
                }
                if (p.gate_out) p.gate_out[(size_t(b) * p.Hq + h) * p.M_max + S] = x;
            }
            if (vote) {
                key = order_key(best);
                len = p.span_len[size_t(b) * p.M_max + S];
            }
        }
        sm.ent[t] = key ? make_uint4(uint32_t(key), uint32_t(key >> 32), uint32_t(S), uint32_t(len))
                        : make_uint4(0u, 0u, 0xFFFFFFFFu, 0u);
    }
    __syncthreads();
    if (k <= 0) return;
    sort_entries(sm.ent, p.cr, tid);

    // 3. publish the chunk's best k (a chunk holds at least kGateMinChunk >= k spans)
    uint64_t *rec = p.cand + (size_t(pair) * p.n_rc + chunk) * size_t(k) * 2;
    if (tid < k) {
        const uint4 e = sm.ent[tid];
        st_shared(rec + 2 * tid, (uint64_t(e.y) << 32) | e.x);
        st_shared(rec + 2 * tid + 1, (uint64_t(e.w) << 32) | e.z);
    }
    stores_done_barrier();
    if (tid == 0) sm.last = counter_add(&p.cnt[pair], 1u) == uint32_t(p.n_rc - 1);
    __syncthreads();
    if (!sm.last) return;

    // 4. the pair's last chunk: sort every candidate, then the budget cap
    const int nc = p.n_rc * k;
    int n2 = 1;
    while (n2 < nc) n2 <<= 1;
    const uint64_t *all = p.cand + size_t(pair) * p.n_rc * size_t(k) * 2;
    for (int i = tid; i < n2; i += GT) {
        if (i < nc) {
            const uint64_t kw = ld_shared(all + 2 * i), iw = ld_shared(all + 2 * i + 1);
            sm.ent[i] = make_uint4(uint32_t(kw), uint32_t(kw >> 32), uint32_t(iw), uint32_t(iw >> 32));
        } else {
            sm.ent[i] = make_uint4(0u, 0u, 0xFFFFFFFFu, 0u);
        }
    }
    __syncthreads();
    sort_entries(sm.ent, n2, tid);
    // inclusive prefix of the expanded token counts over the first k entries (k <= 64:
    // one wave).  Votes sort ahead of non-votes (key 0), so the entries within budget
    // form a prefix of the expansion order.
    if (tid < 64) {
        const uint4 e = tid < k ? sm.ent[tid] : make_uint4(0u, 0u, 0xFFFFFFFFu, 0u);
        const bool vote = (e.x | e.y) != 0u;
        int64_t run = vote ? int64_t(max(int32_t(e.w), 0)) : 0;
        for (int off = 1; off < 64; off <<= 1) {
            const int64_t v = __shfl_up(run, off, 64);
            if (tid >= off) run += v;
        }
        if (tid < k) {
            const bool keep = vote && run <= p.budget;
            p.sel[size_t(pair) * k + tid] = keep ? int32_t(e.z) : -1;
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
