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
// The host passes the ring row of every tap (slot (t - m d) mod R, times the
// row length), so the kernel does no modular arithmetic.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>

#include "mfpsn.h"
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

// K is the order; FULL: every tap reaches back to time >= 0 (t >= (k-1)d),
// else the taps with m > m_max are left out of the sum (their ring slots are
// read like the others, in bounds, and not used: a fresh ring holds garbage
// there).  All loads of a step are issued before any is used.
template <int DT, int K, bool FULL>
__global__ __launch_bounds__(kStreamThreads) void stream_kernel(StreamArgs a)
{
    using ST = typename StreamIO<DT>::T;
    const ST* __restrict__ x_t = (const ST*)a.x_t;
    const ST* __restrict__ ring_in = (const ST*)a.ring;
    ST* __restrict__ ring = (ST*)a.ring;
    // M * 4 < 2^31 (checked on the host), so column indices are 32-bit
    const uint32_t M = (uint32_t)a.M;
    const uint32_t stride = gridDim.x * kStreamThreads;
    const int m_max = a.m_max;  // tap i = K-1-m looks back m*d steps
    for (uint32_t col = blockIdx.x * kStreamThreads + threadIdx.x; col < M; col += stride) {
        const int c = (int)((col / (uint32_t)a.S) % (uint32_t)a.C);
        ST v[K];
        int8_t tsg[K], tsh[K];
        v[0] = x_t[col];
#pragma unroll
        for (int m = 0; m < K; ++m) {
            tsg[m] = a.sign[c * K + (K - 1 - m)];
            tsh[m] = a.shift[c * K + (K - 1 - m)];
            if (m > 0)
                v[m] = ring_in[(size_t)a.rows[m] + col];
        }
        ring[(size_t)a.rows[0] + col] = v[0];
        // ascending tap order: m from K-1 down to 0
        if constexpr (DT == kQ88) {
            int32_t acc = ((const int32_t*)a.bias)[c];
#pragma unroll
            for (int m = K - 1; m >= 0; --m) {
                int s = tsh[m];
                s = s < a.shift_lo ? a.shift_lo : (s > a.shift_hi ? a.shift_hi : s);
                const int32_t y = StreamIO<DT>::value(v[m]) >> s;
                const int32_t term = tsg[m] < 0 ? -y : y;
                acc += (FULL || m <= m_max) ? term : 0;
            }
            a.spikes[col] = acc >= a.v_th_q ? 1 : 0;
            if (a.h_t != nullptr)
                ((int32_t*)a.h_t)[col] = acc;
        } else {
            float acc = 0.0f;
#pragma unroll
            for (int m = K - 1; m >= 0; --m) {
                int s = tsh[m];
                s = s < a.shift_lo ? a.shift_lo : (s > a.shift_hi ? a.shift_hi : s);
                float y = ldexpf(StreamIO<DT>::value(v[m]), -s);
                if (tsg[m] < 0)
                    y = -y;
                const float next = acc + y;
                acc = (FULL || m <= m_max) ? next : acc;
            }
            const float h = acc + ((const float*)a.bias)[c];
            a.spikes[col] = h >= a.v_th ? 1 : 0;
            if (a.h_t != nullptr)
                ((float*)a.h_t)[col] = h;
        }
    }
}

template <int DT, int K>
hipError_t launch_k(const StreamArgs& a, dim3 grid, hipStream_t stream)
{
    if (a.m_max == K - 1)
        hipLaunchKernelGGL((stream_kernel<DT, K, true>), grid, dim3(kStreamThreads), 0, stream, a);
    else
        hipLaunchKernelGGL((stream_kernel<DT, K, false>), grid, dim3(kStreamThreads), 0, stream, a);
    return hipGetLastError();
}

template <int DT, int... Ks>
hipError_t dispatch_k(const StreamArgs& a, dim3 grid, hipStream_t stream, std::integer_sequence<int, Ks...>)
{
    hipError_t e = hipErrorInvalidValue;
    (void)((a.k == Ks + 1 ? (e = launch_k<DT, Ks + 1>(a, grid, stream), true) : false) || ...);
    return e;
}

}  // namespace

hipError_t launch_stream_step(const StreamArgs& a, int dtype, hipStream_t stream)
{
    if (a.M <= 0)
        return hipSuccess;
    int64_t blocks = (a.M + kStreamThreads - 1) / kStreamThreads;
    if (blocks > 65536)
        blocks = 65536;  // the grid-stride loop covers the rest
    const dim3 grid((unsigned)blocks);
    using Orders = std::make_integer_sequence<int, MFPSN_MAX_K>;
    switch (dtype) {
    case kF32: return dispatch_k<kF32>(a, grid, stream, Orders{});
    case kBF16: return dispatch_k<kBF16>(a, grid, stream, Orders{});
    case kQ88: return dispatch_k<kQ88>(a, grid, stream, Orders{});
    default: return hipErrorInvalidValue;
    }
}

}  // namespace mfpsn
