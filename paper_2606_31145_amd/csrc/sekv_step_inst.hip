// One storage type and head dimension of the step kernel (SEKV_T, SEKV_D), for the four
// group sizes.  The build compiles this file once per (type, head_dim) pair, so the
// instantiations compile in parallel.
#include "sekv_step.h"

#if !defined(SEKV_T) || !defined(SEKV_D)
#error "build with -DSEKV_T=BF16|F32 -DSEKV_D=64|128"
#endif

#define SEKV_CAT3(a, b, c) a##_##b##_##c
#define SEKV_NAME(fn, t, d) SEKV_CAT3(fn, t, d)

namespace sekv {
namespace {

template <int G>
hipError_t launch_typed(const Params &p, hipStream_t stream) {
    hipLaunchKernelGGL((sekv_step_kernel<SEKV_T, SEKV_D, G>), dim3(p.grid), dim3(kThreads), 0, stream, p);
    return hipGetLastError();
}

template <int G>
int occupancy_typed() {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, sekv_step_kernel<SEKV_T, SEKV_D, G>, kThreads, 0) !=
        hipSuccess)
        return 1;
    return n > 0 ? n : 1;
}

}  // namespace

hipError_t SEKV_NAME(launch_step, SEKV_T, SEKV_D)(const Params &p, int group, hipStream_t s) {
    switch (group) {
        case 1: return launch_typed<1>(p, s);
        case 2: return launch_typed<2>(p, s);
        case 4: return launch_typed<4>(p, s);
        case 8: return launch_typed<8>(p, s);
    }
    return hipErrorInvalidValue;
}

int SEKV_NAME(occupancy, SEKV_T, SEKV_D)(int group) {
    switch (group) {
        case 1: return occupancy_typed<1>();
        case 2: return occupancy_typed<2>();
        case 4: return occupancy_typed<4>();
        case 8: return occupancy_typed<8>();
    }
    return 1;
}

}  // namespace sekv
