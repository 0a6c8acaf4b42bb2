// bla_forward_noalloc: bla_forward whose workspace is a fixed device array of this library
// instead of a caller buffer, for callers that cannot allocate device memory.
//
// The array `scratch` is a file-scope __device__ variable: each device that loads the
// library's code object holds its own copy until the process ends.  In host code its name
// is only a host-side stand-in, so the device address of each device's copy is taken once,
// with that device current, through hipGetSymbolAddress, kept in a per-device table, and
// that address is what reaches the kernels.
#include <mutex>

#include <hip/hip_runtime.h>

#include "bla.h"

namespace {

constexpr size_t kScratchBytes = BLA_NOALLOC_SCRATCH_BYTES;
static_assert(kScratchBytes % 256 == 0, "the array is handed out whole, 256-byte aligned");

__device__ __align__(256) char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// Device address of the current device's copy of `scratch` (taken on the first call on that
// device), or nullptr if the runtime cannot provide it.
void* device_scratch()
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
        g_scratch_ptr[dev] = ptr;
    }
    return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

bla_status bla_forward_noalloc(const bla_params* p, const double* T, const void* q, const void* k,
                               const void* v, const float* state_k_in, const float* state_v_in, void* o,
                               float* state_k_out, float* state_v_out, void* stream)
{
    const bla_status st = bla_supported(p);
    if (st != BLA_OK) return st;
    if (bla_workspace_size(p) > kScratchBytes) return BLA_ERR_WORKSPACE;
    void* ws = device_scratch();
    if (!ws) return BLA_ERR_HIP;
    // The forward writes every workspace byte it reads (tables, then summaries), so nothing
    // has to be cleared between calls.
    return bla_forward(p, T, q, k, v, state_k_in, state_v_in, o, state_k_out, state_v_out, ws, kScratchBytes,
                       stream);
}

}  // extern "C"
