// gfx950 kernel that makes one layer's spikes the next layer's input, for a
// stack of neuron layers with identity stateless layers in between (the
// sawtooth stack of Sec. 4.1 runs layers of dilation 1..P one after the
// other).  A spike is the value 1 in the next layer's storage type: float
// 1.0, bfloat16 0x3F80, Q8.8 256.  Elementwise and HBM-bound: 1 byte read and
// the storage type's size written per element.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfpsn.h"
#include "mfpsn_chain.h"

namespace mfpsn {
namespace {

constexpr int kChainThreads = 256;

template <typename T>
__device__ __forceinline__ T one_of();
template <>
__device__ __forceinline__ float one_of<float>() { return 1.0f; }
template <>
__device__ __forceinline__ uint16_t one_of<uint16_t>() { return 0x3F80; }  // bfloat16 1.0
template <>
__device__ __forceinline__ int16_t one_of<int16_t>() { return 256; }       // Q8.8 1.0

// VEC: groups of 4 elements, one 4-byte load and one 8- or 16-byte store per
// group, consecutive lanes on consecutive groups (every wave access one
// contiguous segment); 4 groups per lane and pass for loads in flight
template <typename T, bool VEC>
__global__ __launch_bounds__(kChainThreads) void spikes_to_input_kernel(const uint8_t* __restrict__ spikes,
                                                                        int64_t count, T* __restrict__ x)
{
    const T one = one_of<T>(), zero = T(0);
    const int64_t lane = (int64_t)blockIdx.x * kChainThreads + threadIdx.x, lanes = (int64_t)gridDim.x * kChainThreads;
    if constexpr (VEC) {
        const int64_t groups = count / 4;
        const uint32_t* __restrict__ s4 = reinterpret_cast<const uint32_t*>(spikes);
        for (int64_t j0 = lane; j0 < groups; j0 += 4 * lanes) {
            uint32_t b[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int64_t j = j0 + u * lanes;
                b[u] = j < groups ? s4[j] : 0u;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int64_t j = j0 + u * lanes;
                if (j >= groups)
                    break;
                uint32_t bits[4];  // the group's bit patterns
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const T v = ((b[u] >> (8 * e)) & 0xFFu) ? one : zero;
                    if constexpr (sizeof(T) == 4)
                        bits[e] = __builtin_bit_cast(uint32_t, v);
                    else
                        bits[e] = (uint32_t)__builtin_bit_cast(uint16_t, v);
                }
                if constexpr (sizeof(T) == 4)
                    reinterpret_cast<uint4*>(x)[j] = make_uint4(bits[0], bits[1], bits[2], bits[3]);
                else
                    reinterpret_cast<uint2*>(x)[j] = make_uint2(bits[0] | bits[1] << 16, bits[2] | bits[3] << 16);
            }
        }
        // the last count mod 4 elements, one per lane of the first block
        const int64_t rem = count - groups * 4;
        if (lane < rem)
            x[groups * 4 + lane] = spikes[groups * 4 + lane] ? one : zero;
    } else {
        for (int64_t j = lane; j < count; j += lanes)
            x[j] = spikes[j] ? one : zero;
    }
}

template <typename T>
void launch_typed(const uint8_t* spikes, int64_t count, void* x, hipStream_t st)
{
    const bool vec = ((uintptr_t)spikes % 4) == 0 && ((uintptr_t)x % (4 * sizeof(T))) == 0;
    const int64_t lanes = vec ? (count + 15) / 16 : count;
    int64_t blocks = (lanes + kChainThreads - 1) / kChainThreads;
    blocks = blocks < 1 ? 1 : (blocks > 65536 ? 65536 : blocks);
    if (vec)
        hipLaunchKernelGGL((spikes_to_input_kernel<T, true>), dim3((unsigned)blocks), dim3(kChainThreads), 0, st,
                           spikes, count, (T*)x);
    else
        hipLaunchKernelGGL((spikes_to_input_kernel<T, false>), dim3((unsigned)blocks), dim3(kChainThreads), 0, st,
                           spikes, count, (T*)x);
}

}  // namespace

hipError_t launch_spikes_to_input(const uint8_t* spikes, int64_t count, int32_t dtype, void* x, hipStream_t st)
{
    if (count <= 0)
        return hipSuccess;
    switch (dtype) {
    case MFPSN_F32: launch_typed<float>(spikes, count, x, st); break;
    case MFPSN_BF16: launch_typed<uint16_t>(spikes, count, x, st); break;
    default: launch_typed<int16_t>(spikes, count, x, st); break;
    }
    return hipGetLastError();
}

}  // namespace mfpsn
