// gfx950 kernel of the latent-weight gradient of the power-of-two quantizer
// (arXiv 2501.14490, Sec. 4.2).  The paper trains with the whole-quantizer
// straight-through estimator (dWq/dW = 1, so the latent gradient is the
// quantized weight's gradient unchanged); the variant it discusses first
// replaces only round()'s derivative by 1 (Eq. ste), which gives
// dWq/dW = 2^round(log2|W|) / |W| = |Wq| / |W| (Eq. ste_q).  Elementwise over
// the C*k weights: no multiply-free constraint applies (this is the gradient
// of a real-valued parameter, not a tap).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfpsn_qgrad.h"

namespace mfpsn {
namespace {

constexpr int kQgThreads = 256;

// mode 1: grad * (2^-shift / |w|): |Wq| = 2^-shift is exact, the quotient and
// the product are each rounded once; 0 where the factor is undefined or not
// finite (w = 0, w not finite, quotient overflow)
__global__ __launch_bounds__(kQgThreads) void qgrad_kernel(const float* __restrict__ w,
                                                           const int8_t* __restrict__ shift, int lo, int hi,
                                                           const float* __restrict__ g, int64_t count, int mode,
                                                           float* __restrict__ out)
{
    const int64_t stride = (int64_t)gridDim.x * kQgThreads;
    for (int64_t j = (int64_t)blockIdx.x * kQgThreads + threadIdx.x; j < count; j += stride) {
        if (mode == 0) {
            out[j] = g[j];
            continue;
        }
        const float a = __builtin_fabsf(w[j]);
        int s = shift[j];
        s = s < lo ? lo : (s > hi ? hi : s);
        const float q = ldexpf(1.0f, -s);
        const float f = q / a;
        const bool ok = a > 0.0f && a < __builtin_inff() && f < __builtin_inff();
        out[j] = ok ? g[j] * f : 0.0f;
    }
}

}  // namespace

hipError_t launch_quantizer_grad(const float* w, const int8_t* shift, int32_t lo, int32_t hi, const float* g,
                                 int64_t count, int32_t mode, float* out, hipStream_t stream)
{
    if (count <= 0)
        return hipSuccess;
    int64_t blocks = (count + kQgThreads - 1) / kQgThreads;
    if (blocks > 4096)
        blocks = 4096;
    hipLaunchKernelGGL(qgrad_kernel, dim3((unsigned)blocks), dim3(kQgThreads), 0, stream, w, shift, lo, hi, g,
                       count, mode, out);
    return hipGetLastError();
}

}  // namespace mfpsn
