// Internal interface of the streaming-inference kernel (mfpsn_stream.hip)
// for the C-ABI layer.  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "mfpsn.h"
#include "mfpsn_internal.h"

namespace mfpsn {

struct StreamArgs {
    int64_t M;           // columns per time step, N*C*S
    int32_t C, S, k, d;
    int32_t R;           // ring slots, (k-1)*d + 1
    int32_t slot;        // t mod R: the slot x_t is stored in
    int32_t m_max;       // min(k-1, t/d): taps looking back more than t steps are left out
    int64_t rows[MFPSN_MAX_K];  // element offset of the ring row of time t - m*d (slot mod R) for
                                // m < k; rows[0] is x_t's slot
    int32_t shift_lo, shift_hi;
    float v_th;
    int32_t v_th_q;
    const void* x_t;     // [N][C][S]
    void* ring;          // [R][N][C][S]
    const int8_t* sign;  // [C][k]
    const int8_t* shift; // [C][k]
    const void* bias;    // float[C] or int32[C]
    uint8_t* spikes;     // [N][C][S]
    void* h_t;           // nullable, float or int32 [N][C][S]
};

hipError_t launch_stream_step(const StreamArgs& a, int dtype, hipStream_t stream);

}  // namespace mfpsn
