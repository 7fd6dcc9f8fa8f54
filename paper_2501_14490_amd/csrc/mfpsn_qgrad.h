// Internal interface of the quantizer-gradient kernel (mfpsn_qgrad.hip) for
// the C-ABI layer.  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace mfpsn {

hipError_t launch_quantizer_grad(const float* w, const int8_t* shift, int32_t lo, int32_t hi, const float* g,
                                 int64_t count, int32_t mode, float* out, hipStream_t stream);

}  // namespace mfpsn
