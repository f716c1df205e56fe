// Launch dispatch of the step kernel over its compiled variants, and the workspace
// zero kernel.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sekv_internal.h"

namespace sekv {

// defined in sekv_step_inst.hip, one object per (storage type, head_dim)
hipError_t launch_step_BF16_128(const Params &p, int group, hipStream_t s);
hipError_t launch_step_BF16_64(const Params &p, int group, hipStream_t s);
hipError_t launch_step_F32_128(const Params &p, int group, hipStream_t s);
hipError_t launch_step_F32_64(const Params &p, int group, hipStream_t s);
int occupancy_BF16_128(int group);
int occupancy_BF16_64(int group);
int occupancy_F32_128(int group);
int occupancy_F32_64(int group);

namespace {

// Workspace initialisation: everything zero except the header's epoch, which starts at
// 1 (the first {unused, exit_count, error, epoch} vector).
__global__ void zero_kernel(uint4 *p, size_t n16) {
    for (size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n16;
         i += size_t(gridDim.x) * blockDim.x)
        p[i] = make_uint4(0, 0, 0, i == 0 ? 1u : 0u);
}

}  // namespace

hipError_t launch_step(const Params &p, int dtype, int head_dim, int group, hipStream_t stream) {
    if (dtype == SEKV_BF16) {
        if (head_dim == 128) return launch_step_BF16_128(p, group, stream);
        if (head_dim == 64) return launch_step_BF16_64(p, group, stream);
    } else {
        if (head_dim == 128) return launch_step_F32_128(p, group, stream);
        if (head_dim == 64) return launch_step_F32_64(p, group, stream);
    }
    return hipErrorInvalidValue;
}

int resident_workgroups(int dtype, int head_dim, int group) {
    int per_cu = 1;
    if (dtype == SEKV_BF16) per_cu = head_dim == 128 ? occupancy_BF16_128(group) : occupancy_BF16_64(group);
    else per_cu = head_dim == 128 ? occupancy_F32_128(group) : occupancy_F32_64(group);
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
