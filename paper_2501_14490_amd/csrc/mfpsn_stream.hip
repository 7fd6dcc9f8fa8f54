// gfx950 kernel of the step-by-step (streaming) inference of the mul-free
// channel-wise Parallel Spiking Neuron (arXiv 2501.14490): one time step of
// the charge (Sec. 4.2, Eq. mfdpsn_charge) and fire (Eq. mfdpsn_fire) per
// launch, for inputs that arrive one step at a time.
//
// The neuron keeps the inputs of its receptive field, (k-1)*d + 1 time steps,
// in a caller-owned history ring [R][N][C][S]: the input of time tau lives in
// slot tau mod R.  A launch stores x_t in its slot and evaluates
//   H_t = sum_{i : t-(k-1-i)d >= 0} sign[c,i] * 2^-shift[c,i] * x[t-(k-1-i)d] + bias[c]
// with the terms in ascending tap order from +0 (float: exact exponent move
// by v_ldexp_f32, then a sign flip; Q8.8: arithmetic right shift, then
// negation), bias last, so that a run over t = 0..T-1 reproduces the
// whole-sequence forward bit for bit.  The step is memory-bound: each column
// reads its new input and up to k-1 older ones and writes one ring entry and
// one spike byte (and optionally H).  One lane per column; adjacent lanes own
// adjacent columns, so every access of a wave is one contiguous row segment.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfpsn_stream.h"

namespace mfpsn {
namespace {

constexpr int kStreamThreads = 256;

template <int DT> struct StreamIO;
template <> struct StreamIO<kF32> {
    using T = float;
    __device__ static float value(float v) { return v; }
};
template <> struct StreamIO<kBF16> {
    using T = uint16_t;
    __device__ static float value(uint16_t v) { return __builtin_bit_cast(float, (uint32_t)v << 16); }
};
template <> struct StreamIO<kQ88> {
    using T = int16_t;
    __device__ static int32_t value(int16_t v) { return v; }
};

template <int DT>
__global__ __launch_bounds__(kStreamThreads) void stream_kernel(StreamArgs a)
{
    using ST = typename StreamIO<DT>::T;
    const ST* __restrict__ x_t = (const ST*)a.x_t;
    ST* __restrict__ ring = (ST*)a.ring;
    // M * 4 < 2^31 (checked on the host), so column indices are 32-bit
    const uint32_t M = (uint32_t)a.M;
    const uint32_t stride = gridDim.x * kStreamThreads;
    for (uint32_t col = blockIdx.x * kStreamThreads + threadIdx.x; col < M; col += stride) {
        const int c = (int)((col / (uint32_t)a.S) % (uint32_t)a.C);
        const ST xn = x_t[col];
        ring[(size_t)a.slot * M + col] = xn;
        // taps i = k-1-m look back m*d steps; m > m_max reads before time 0
        if constexpr (DT == kQ88) {
            int32_t acc = ((const int32_t*)a.bias)[c];
            for (int m = a.m_max; m >= 0; --m) {
                const int i = a.k - 1 - m;
                int sl = a.slot - m * a.d;
                sl += sl < 0 ? a.R : 0;
                const int32_t v = m == 0 ? (int32_t)xn : (int32_t)ring[(size_t)sl * M + col];
                int s = a.shift[c * a.k + i];
                s = s < a.shift_lo ? a.shift_lo : (s > a.shift_hi ? a.shift_hi : s);
                const int32_t y = v >> s;
                acc += a.sign[c * a.k + i] < 0 ? -y : y;
            }
            a.spikes[col] = acc >= a.v_th_q ? 1 : 0;
            if (a.h_t != nullptr)
                ((int32_t*)a.h_t)[col] = acc;
        } else {
            float acc = 0.0f;
            for (int m = a.m_max; m >= 0; --m) {
                const int i = a.k - 1 - m;
                int sl = a.slot - m * a.d;
                sl += sl < 0 ? a.R : 0;
                const float v = StreamIO<DT>::value(m == 0 ? xn : ring[(size_t)sl * M + col]);
                int s = a.shift[c * a.k + i];
                s = s < a.shift_lo ? a.shift_lo : (s > a.shift_hi ? a.shift_hi : s);
                float y = ldexpf(v, -s);
                if (a.sign[c * a.k + i] < 0)
                    y = -y;
                acc = acc + y;
            }
            const float h = acc + ((const float*)a.bias)[c];
            a.spikes[col] = h >= a.v_th ? 1 : 0;
            if (a.h_t != nullptr)
                ((float*)a.h_t)[col] = h;
        }
    }
}

}  // namespace

hipError_t launch_stream_step(const StreamArgs& a, int dtype, hipStream_t stream)
{
    if (a.M <= 0)
        return hipSuccess;
    int64_t blocks = (a.M + kStreamThreads - 1) / kStreamThreads;
    if (blocks > 65536)
        blocks = 65536;  // the grid-stride loop covers the rest
    const dim3 grid((unsigned)blocks), block(kStreamThreads);
    switch (dtype) {
    case kF32: hipLaunchKernelGGL(stream_kernel<kF32>, grid, block, 0, stream, a); break;
    case kBF16: hipLaunchKernelGGL(stream_kernel<kBF16>, grid, block, 0, stream, a); break;
    case kQ88: hipLaunchKernelGGL(stream_kernel<kQ88>, grid, block, 0, stream, a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace mfpsn
