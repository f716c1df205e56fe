// Pinned-host tier: host-to-device moves of the selected factor blocks.
//
// tier_gather_kernel plans on the device: it reads the sequence's selection and tables
// from device memory, gives selection slot (g, j) the fixed staging slot (g, j), and
// copies the block through the arena's device mapping; nothing waits on the host, so a
// tiered step in this mode can be captured in a graph.  (The host-planned mode moves the
// blocks with hipMemcpyAsync instead; see sekv_api.cpp.)
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sekv_internal.h"

namespace sekv {
namespace {

constexpr int kGT = 256;                                   // threads per workgroup
constexpr int kGV = kGatherChunk / (16 * kGT);             // 16-byte vectors per thread

// Copy bytes [lo, hi) of a block (lo, hi multiples of 16): every load of the chunk is
// issued before its first store.
__device__ inline void copy_chunk(const unsigned char *src, unsigned char *dst, int64_t lo, int64_t hi) {
    const int nv = int((hi - lo) >> 4);
    const uint4 *s = reinterpret_cast<const uint4 *>(src + lo);
    uint4 *d = reinterpret_cast<uint4 *>(dst + lo);
    uint4 v[kGV];
#pragma unroll
    for (int u = 0; u < kGV; ++u) {
        const int i = int(threadIdx.x) + kGT * u;
        v[u] = i < nv ? s[i] : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int u = 0; u < kGV; ++u) {
        const int i = int(threadIdx.x) + kGT * u;
        if (i < nv) d[i] = v[u];
    }
}

// Block bytes of a span of length L with rank r on both sides: U|sigma|Vt for keys and
// values, 16-byte segments (half of it is one side).
__device__ inline int64_t dev_block_bytes(int64_t L, int r, int d, int e) {
    auto a16 = [](int64_t x) { return (x + 15) & ~int64_t(15); };
    return 2 * (a16(L * r * e) + a16(int64_t(r) * e) + a16(int64_t(r) * d * e));
}

__global__ __launch_bounds__(kGT) void tier_gather_kernel(TierGatherArgs a) {
    const int slot = int(blockIdx.x) / a.chunks_per_slot, c = int(blockIdx.x) % a.chunks_per_slot;
    const int g = slot / a.k, j = slot % a.k;
    const int s = a.sel[size_t(g) * a.k + j];
    if (s < 0 || s >= a.M) return;
    const int L = a.span_len[s];
    const int64_t off = a.block_off[size_t(g) * a.M + s];
    int rk = a.r, rv = a.r;
    if (a.block_rank) {
        const uint32_t w = uint32_t(a.block_rank[size_t(g) * a.M + s]);
        rk = int(w & 0xFFFFu);
        rv = int(w >> 16);
    }
    const int gran = 16 / a.elem;
    const bool ranks_ok = rk >= gran && rk <= a.r && rk % gran == 0 && rv >= gran && rv <= a.r && rv % gran == 0;
    const int64_t bytes = dev_block_bytes(L, rk, a.d, a.elem) / 2 + dev_block_bytes(L, rv, a.d, a.elem) / 2;
    if (!ranks_ok || L < 1 || L > a.max_span_len || off < 0 || (off & 15) || off > a.arena_bytes - bytes) {
        // skipped: the attention reads whatever the slot holds, inside staging
        if (c == 0 && threadIdx.x == 0)
            __hip_atomic_fetch_or(a.error, kErrBlockRange, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
    }
    const int64_t dst = a.slot0 + int64_t(slot) * a.slot_bytes;
    if (c == 0 && threadIdx.x == 0) {
        a.stage_off[size_t(g) * a.M + s] = dst;
        __hip_atomic_fetch_add(&a.stats[0], (unsigned long long)bytes, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_fetch_add(&a.stats[1], 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    const int64_t lo = int64_t(c) * kGatherChunk;
    if (lo >= bytes) return;
    const int64_t hi = lo + kGatherChunk < bytes ? lo + kGatherChunk : bytes;
    copy_chunk(a.arena + off, a.staging + dst, lo, hi);
}

__global__ void stats_reset_kernel(unsigned long long *stats, int n) {
    if (int(threadIdx.x) < n) stats[threadIdx.x] = 0;
}

// Layered tier: slot (b, g, j) of the launch, chunk c of its block.
__global__ __launch_bounds__(kGT) void layer_copy_kernel(LayerCopyArgs a) {
    const int slot = int(blockIdx.x) / a.chunks_per_slot, c = int(blockIdx.x) % a.chunks_per_slot;
    const int pg = slot / a.k;                                // b * Hkv + g
    const int b = pg / a.Hkv;
    const int s = a.sel[slot];
    const bool first = c == 0 && threadIdx.x == 0;
    if (a.prefetch && first) a.pf_span[slot] = -1;            // set again below once copied
    if (s < 0 || s >= a.M) return;
    const size_t at = size_t(pg) * a.M + s;
    if (!a.prefetch && a.use_pf) {
        for (int jj = 0; jj < a.k; ++jj)
            if (a.pf_span[size_t(pg) * a.k + jj] == s) {
                if (first) a.stage_off[at] = int64_t(size_t(pg) * a.k + jj) * a.slot_bytes;
                return;
            }
    }
    const int L = a.span_len[size_t(b) * a.M + s];
    const int64_t off = a.block_off[at];
    int rk = a.r, rv = a.r;
    if (a.block_rank) {
        const uint32_t w = uint32_t(a.block_rank[at]);
        rk = int(w & 0xFFFFu);
        rv = int(w >> 16);
    }
    const int gran = 16 / a.elem;
    const bool ranks_ok = rk >= gran && rk <= a.r && rk % gran == 0 && rv >= gran && rv <= a.r && rv % gran == 0;
    const int64_t bytes = dev_block_bytes(L, rk, a.d, a.elem) / 2 + dev_block_bytes(L, rv, a.d, a.elem) / 2;
    if (!ranks_ok || L < 1 || L > a.max_span_len || off < 0 || (off & 15) || off > a.arena_bytes - bytes) {
        if (first) __hip_atomic_fetch_or(a.error, kErrBlockRange, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
    }
    const int64_t dst = (a.prefetch ? 0 : a.miss0) + int64_t(slot) * a.slot_bytes;
    if (first) {
        if (a.prefetch) a.pf_span[slot] = s;
        else a.stage_off[at] = dst;
        unsigned long long *st = a.stats + (a.prefetch ? 2 : 0);
        __hip_atomic_fetch_add(&st[0], (unsigned long long)bytes, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_fetch_add(&st[1], 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    const int64_t lo = int64_t(c) * kGatherChunk;
    if (lo >= bytes) return;
    const int64_t hi = lo + kGatherChunk < bytes ? lo + kGatherChunk : bytes;
    copy_chunk(a.arena + off, a.staging + dst, lo, hi);
}

}  // namespace

hipError_t launch_tier_gather(const TierGatherArgs &a, hipStream_t stream) {
    const int64_t n = int64_t(a.Hkv) * a.k * a.chunks_per_slot;
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(tier_gather_kernel, dim3(unsigned(n)), dim3(kGT), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_stats_reset(unsigned long long *stats, hipStream_t stream) {
    hipLaunchKernelGGL(stats_reset_kernel, dim3(1), dim3(64), 0, stream, stats, 2);
    return hipGetLastError();
}

hipError_t launch_stats_reset4(unsigned long long *stats, hipStream_t stream) {
    hipLaunchKernelGGL(stats_reset_kernel, dim3(1), dim3(64), 0, stream, stats, 4);
    return hipGetLastError();
}

hipError_t launch_layer_copy(const LayerCopyArgs &a, hipStream_t stream) {
    const int64_t n = int64_t(a.B) * a.Hkv * a.k * a.chunks_per_slot;
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(layer_copy_kernel, dim3(unsigned(n)), dim3(kGT), 0, stream, a);
    return hipGetLastError();
}

}  // namespace sekv
