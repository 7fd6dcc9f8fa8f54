// Internal interface of the time-last kernels (mfpsn_tl.hip: forward and
// backward) for the C-ABI layer.  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace mfpsn {

constexpr int kTlWaves = 4;                 // waves per block
constexpr int kTlMaxHalo = 2048;            // longest history tl_fwd_kernel stages in LDS
constexpr int kTlColsMaxT = 64;             // longest column of the lane-per-column kernels
constexpr int kTlBwdSeg = 256;              // time steps per segment of the zero-window segment kernels
constexpr int kTlBwdSegLong = 1024;         // the same for histories (k-1) d above 64
constexpr int kTlBwdMaxSpan = 1024;         // longest history (k-1) d of the zero-window segment kernels

struct TlArgs {
    const void* x;          // [N][C][S][T] storage type
    const int8_t* sign;     // [C][k]
    const int8_t* shift;    // [C][k]
    const void* bias;       // float[C] or int32[C]
    uint8_t* spikes;        // [N][C][S][T]
    void* h_out;            // nullable, float or int32 [N][C][S][T]
    int64_t M;              // columns, N*C*S
    int32_t T, C, S, k, d;
    int32_t steps_per_lane; // 1 or 4: segments of 64 or 256 time steps (seg = 0)
    int32_t seg;            // > 0: segment length of tl_seg_fwd_kernel (T > kTlColsMaxT, history <= kTlBwdMaxSpan)
    int32_t nseg;           // segments per column, ceil(T / seg), else ceil(T / (64 * steps_per_lane))
    int32_t halo;           // LDS history slots per wave (0: taps read from global memory)
    int32_t shift_lo, shift_hi;
    float v_th;
    int32_t v_th_q;
    float fast_lo, fast_hi; // range of |x| in which the exponent-add tap is exact
    uint32_t tdiv;          // floor(2^32 / T) + 1 (T >= 2; 0 when T = 1): e / T = umulhi(e, tdiv) for e < 64 T
    int32_t vec_x;          // x is aligned for 4-element vector loads
    int32_t vec_s;          // spikes are 16-byte aligned
};

hipError_t launch_forward_time_last(const TlArgs& a, int dtype, hipStream_t stream);

// Backward in the time-last layout
struct TlBwdArgs {
    const void* x;          // [N][C][S][T] storage type
    const void* g;          // grad_spikes, [N][C][S][T] storage type
    const int8_t* sign;     // [C][k]
    const int8_t* shift;    // [C][k]
    const void* bias;       // float[C] or int32[C]
    void* grad_x;           // [N][C][S][T] float, bfloat16 bits or int32
    void* acc;              // [k+1][C] double (float data) or int64 (Q8.8): grad_w rows, then grad_b
    int64_t M;              // columns, N*C*S
    int32_t T, C, S, k, d;
    int32_t shift_lo, shift_hi;
    float v_th;
    int32_t v_th_q;
    int32_t sg;             // surrogate kind
    float alpha;
    float fast_lo, fast_hi; // range of |x| and |dH| in which the exponent-add tap is exact
    uint32_t tdiv;          // as TlArgs::tdiv (0 when T = 1)
    int32_t vec_x;          // x and g aligned for 4-element vector loads
    int32_t seg;            // time steps per segment (T > kTlColsMaxT): kTlBwdSeg or kTlBwdSegLong
    int32_t nseg;           // segments per column, ceil(T / seg)
};

// Zeroes acc, runs the backward, which adds into acc; the caller finalizes
// acc into grad_w and grad_b.
hipError_t launch_backward_time_last(const TlBwdArgs& a, int dtype, hipStream_t stream);

// One storage type's launchers, each in its own translation unit
void tl_forward_f32(const TlArgs& a, hipStream_t st);
void tl_forward_bf16(const TlArgs& a, hipStream_t st);
void tl_forward_q88(const TlArgs& a, hipStream_t st);
void tl_backward_f32(const TlBwdArgs& a, hipStream_t st);
void tl_backward_bf16(const TlBwdArgs& a, hipStream_t st);
void tl_backward_q88(const TlBwdArgs& a, hipStream_t st);

}  // namespace mfpsn
