// sekv_decode_step_noalloc: the fused decode step with its workspace in a file-scope
// device array, for callers that cannot allocate device memory.
//
// `scratch` is a static device array; in host code its name is only a host-side stand-in
// for the symbol, so the host never passes it to a kernel or a copy.  The first call on
// each device looks up the array's device address there (hipGetSymbolAddress, with that
// device current) and keeps it; every later call on the device uses that address.  The
// step itself is sekv_decode_step's, with the same checks; the library's workspace
// bookkeeping zeroes the array (a kernel on the caller's stream) on its first use and
// whenever the shapes change, so nothing left by an earlier call leaks into a later one.
#include <hip/hip_runtime.h>

#include <mutex>

#include "sekv.h"
#include "sekv_host.h"
#include "sekv_internal.h"

namespace {

constexpr size_t kScratchBytes = size_t(16) << 20;       // SEKV_NOALLOC_MAX_WORKSPACE
static_assert(kScratchBytes == SEKV_NOALLOC_MAX_WORKSPACE, "header and library disagree");
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void *g_ptr[kMaxDevices] = {};

}  // namespace

extern "C" sekv_status sekv_decode_step_noalloc(const sekv_dims *dims, const sekv_cache *cache,
                                                int32_t *sel, void *out, hipStream_t stream) {
    sekv_status st = sekv::check_dims(dims);
    if (st != SEKV_OK) return st;
    const size_t need = sekv_workspace_size(dims);
    if (need > kScratchBytes)
        return sekv::fail(SEKV_ERR_WORKSPACE,
                          "these shapes need a %zu-byte workspace; sekv_decode_step_noalloc holds %zu "
                          "bytes (use sekv_decode_step with a caller workspace)", need, kScratchBytes);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return sekv::fail(SEKV_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices) return sekv::fail(SEKV_ERR_UNSUPPORTED, "device %d", dev);
    void *ptr = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        if (!g_ptr[dev]) {
            void *p = nullptr;
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess || !p)
                return sekv::fail(SEKV_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                                  hipGetErrorString(e));
            g_ptr[dev] = p;
        }
        ptr = g_ptr[dev];
    }
    return sekv::run_fused_step(dims, cache, sel, out, ptr, kScratchBytes, stream);
}
