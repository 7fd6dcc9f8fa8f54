// mfpsn_backward_no_alloc: the backward of the training step for callers
// that cannot allocate device memory (code under HIP graph capture, tight
// serving loops, harnesses that forbid hipMalloc).  Its workspace is a
// file-scope device array of fixed size instead of a caller-provided buffer.
//
// The array lives once on every GPU the library runs on, until the process
// ends.  Host code never uses the array's name as an address: the first call
// on a device (with that device current) asks the runtime for the array's
// device address with hipGetSymbolAddress and keeps it per device; the
// kernels receive that address like any workspace pointer.
#include <hip/hip_runtime.h>

#include <mutex>

#include "mfpsn.h"

namespace {

// Upper bound of mfpsn_backward_workspace_size that this entry point serves:
// the per-block partial sums of grad_w and grad_b (double, or int64 for
// Q8.8), (k+1)*C values per resident block.
constexpr size_t kScratchBytes = (size_t)MFPSN_NO_ALLOC_WORKSPACE_BYTES;

__device__ __align__(256) double scratch[kScratchBytes / sizeof(double)];

constexpr int kMaxDevices = 64;
std::mutex scratch_mutex;
void* scratch_ptr[kMaxDevices] = {};

// Device address of this device's scratch array, looked up once per device.
int scratch_for_current_device(void** out)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0)
        return MFPSN_ERR_HIP;
    if (dev >= kMaxDevices)
        return MFPSN_ERR_HIP;
    std::lock_guard<std::mutex> lock(scratch_mutex);
    if (scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
            return MFPSN_ERR_HIP;
        scratch_ptr[dev] = p;
    }
    *out = scratch_ptr[dev];
    return MFPSN_OK;
}

}  // namespace

extern "C" int mfpsn_backward_no_alloc(const mfpsn_desc* desc, const void* x, const void* grad_spikes, const void* h,
                                       const void* sg, const int8_t* sign, const int8_t* shift, const void* bias,
                                       const void* v_th_c, void* grad_x, void* grad_w, void* grad_b, void* grad_vth,
                                       void* stream)
{
    size_t need = 0;
    int st = mfpsn_backward_workspace_size(desc, &need);
    if (st != MFPSN_OK)
        return st;
    if (need > kScratchBytes)
        return MFPSN_ERR_WORKSPACE;
    void* ws = nullptr;
    if (need > 0) {
        st = scratch_for_current_device(&ws);
        if (st != MFPSN_OK)
            return st;
    }
    return mfpsn_backward(desc, x, grad_spikes, h, sg, sign, shift, bias, v_th_c, grad_x, grad_w, grad_b, grad_vth,
                          ws, need > 0 ? kScratchBytes : 0, stream);
}
