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
constexpr int kTlSegMaxBlocks = 8192;       // most blocks of the persistent segment backward

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
    void* part;             // [slots][k+1] of the same type: each block's (T <= kTlColsMaxT) or
                            // wave's sums of one group of columns, at slot (block or wave) + group
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
    int64_t chunk;          // segments per wave of the segment backward (set by its launcher)
};

// Slots of partial sums the backward writes to TlBwdArgs::part.  The columns
// fall into groups whose sums are wanted (the (n, c) rows of S columns for
// T <= kTlColsMaxT, whose blocks take 64 columns each; the channels' runs
// of N*S*nseg segments for the segment kernel, whose waves take `chunk`
// segments each).  Both cut the same sequence into consecutive pieces, so
// the (block, group) pairs that share a column have distinct sums block +
// group, fewer than blocks + groups.
inline int64_t tl_bwd_slots(int64_t M, int32_t T, int32_t C, int32_t N, int64_t nseg)
{
    if (M == 0 || T == 0)
        return 0;
    if (T <= kTlColsMaxT)
        return (M + 63) / 64 + (int64_t)N * C;
    int64_t blocks = (M * nseg + kTlWaves - 1) / kTlWaves;
    blocks = blocks < kTlSegMaxBlocks ? blocks : kTlSegMaxBlocks;
    return blocks * kTlWaves + C;
}

// Runs the backward, which writes its partial sums to a.part, then adds
// each channel's slots in a fixed order into acc (so grad_w and grad_b do
// not change from call to call); the caller finalizes acc into grad_w and
// grad_b.
hipError_t launch_backward_time_last(const TlBwdArgs& a, int dtype, hipStream_t stream);

// One storage type's launchers, each in its own translation unit
void tl_forward_f32(const TlArgs& a, hipStream_t st);
void tl_forward_bf16(const TlArgs& a, hipStream_t st);
void tl_forward_q88(const TlArgs& a, hipStream_t st);
// (the backward launchers return the columns per block, or segments per
// wave, of the kernel they launched)
int64_t tl_backward_f32(const TlBwdArgs& a, hipStream_t st);
int64_t tl_backward_bf16(const TlBwdArgs& a, hipStream_t st);
int64_t tl_backward_q88(const TlBwdArgs& a, hipStream_t st);

}  // namespace mfpsn
