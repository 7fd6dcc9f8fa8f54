// Internal interface of the layer-chaining kernel (mfpsn_chain.hip) for the
// C-ABI layer.  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace mfpsn {

hipError_t launch_spikes_to_input(const uint8_t* spikes, int64_t count, int32_t dtype, void* x, hipStream_t stream);

}  // namespace mfpsn
