// Pinned-host tier: the host-to-device gather of the selected factor blocks.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sekv_internal.h"

namespace sekv {
namespace {

// Moves the selected factor blocks from host memory (read through its
// device mapping) into device staging.  Each workgroup moves whole chunks of at most
// kGatherChunk bytes, 16-byte aligned at both ends; the chunk table itself sits in
// pinned host memory.  All of a chunk's loads are issued before its first store.
__global__ __launch_bounds__(256) void gather_kernel(const unsigned char *src, unsigned char *dst,
                                                     const GatherChunk *chunks, int n_chunks) {
    constexpr int kV = kGatherChunk / (16 * 256);
    for (int c = blockIdx.x; c < n_chunks; c += gridDim.x) {
        const GatherChunk ch = chunks[c];
        const int nv = int(ch.bytes >> 4);
        const uint4 *s = reinterpret_cast<const uint4 *>(src + ch.src);
        uint4 *d = reinterpret_cast<uint4 *>(dst + ch.dst);
        uint4 v[kV];
#pragma unroll
        for (int u = 0; u < kV; ++u) {
            const int i = int(threadIdx.x) + 256 * u;
            if (i < nv) v[u] = s[i];
        }
#pragma unroll
        for (int u = 0; u < kV; ++u) {
            const int i = int(threadIdx.x) + 256 * u;
            if (i < nv) d[i] = v[u];
        }
    }
}

}  // namespace

hipError_t launch_gather(const void *src, void *dst, const GatherChunk *chunks, int n_chunks,
                         hipStream_t stream) {
    if (n_chunks <= 0) return hipSuccess;
    const int blocks = n_chunks < 1024 ? n_chunks : 1024;
    hipLaunchKernelGGL(gather_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream,
                       static_cast<const unsigned char *>(src), static_cast<unsigned char *>(dst),
                       chunks, n_chunks);
    return hipGetLastError();
}

}  // namespace sekv
