// gfx950 kernels of the batch-normalized threshold with fused-weight
// quantization (arXiv 2501.14490, App. C, Eqs. weight fuse and bias fuse):
// the statistics of the latent-weight convolution, the fusion, and the
// backward of both.  The quantized charge, fire and surrogate backward in
// between are the library's own forward and backward kernels.
//
//   Tv[t,n,c,s] = sum_{i, tau >= 0} W[c,i] x[tau],  tau = t-(k-1-i)d     (latent weights)
//   mu_c, var_c = mean and biased variance of Tv over (t, n, s)
//   s_c = gamma_c / sqrt(var_c + eps),  W_f = s_c W,  b_f = beta_c - s_c mu_c
//
// Tv is evaluated in double: the product of two floats is exact there and the
// sum runs in ascending tap order, so every element of Tv (and of dTv below)
// is the same double on both sides of the parity tests.  The per-channel
// reductions use per-thread partial sums that a second kernel adds in a
// fixed order (so results do not depend on scheduling).  These kernels are
// simple and memory-bound: one thread per element or column, k loads per
// evaluation of Tv, with the reuse left to the caches.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mfpsn_bn.h"

namespace mfpsn {
namespace {

constexpr int kBnThreads = 256;

__device__ __forceinline__ double latent_conv(const float* __restrict__ x, size_t M, int64_t t, size_t col,
                                              const float* __restrict__ wc, int k, int d)
{
    double acc = 0.0;
    for (int i = 0; i < k; ++i) {
        const int64_t tau = t - (int64_t)(k - 1 - i) * d;
        if (tau >= 0)
            acc = acc + (double)wc[i] * (double)x[(size_t)tau * M + col];
    }
    return acc;
}

__device__ __forceinline__ int channel_of(size_t col, const BnGeom& g) { return (int)((col / g.S) % g.C); }

// partial sums of Tv and Tv^2 per (time chunk, column)
__global__ __launch_bounds__(kBnThreads) void bn_stats_partial(BnGeom g, const float* __restrict__ x,
                                                               const float* __restrict__ w,
                                                               double* __restrict__ part)
{
    const size_t total = (size_t)g.chunks * g.M;
    for (size_t q = (size_t)blockIdx.x * kBnThreads + threadIdx.x; q < total; q += (size_t)gridDim.x * kBnThreads) {
        const size_t col = q % g.M;
        const int ch = (int)(q / g.M);
        const int c = channel_of(col, g);
        const int t0 = ch * g.tc, t1 = min(g.T, t0 + g.tc);
        double s1 = 0.0, s2 = 0.0;
        for (int t = t0; t < t1; ++t) {
            const double v = latent_conv(x, g.M, t, col, w + (size_t)c * g.k, g.k, g.d);
            s1 += v;
            s2 += v * v;
        }
        part[2 * q + 0] = s1;
        part[2 * q + 1] = s2;
    }
}

// per channel: the sums in (chunk, n, s) order, the statistics and the fusion
__global__ __launch_bounds__(kBnThreads) void bn_fuse(BnGeom g, const double* __restrict__ part,
                                                      const float* __restrict__ w, const float* __restrict__ gamma,
                                                      const float* __restrict__ beta, float eps,
                                                      float* __restrict__ w_f, float* __restrict__ b_f,
                                                      double* __restrict__ aux, double* __restrict__ stats)
{
    for (int c = blockIdx.x * kBnThreads + threadIdx.x; c < g.C; c += gridDim.x * kBnThreads) {
        double s1 = 0.0, s2 = 0.0;
        for (int ch = 0; ch < g.chunks; ++ch)
            for (int n = 0; n < g.N; ++n)
                for (int s = 0; s < g.S; ++s) {
                    const size_t q = (size_t)ch * g.M + ((size_t)n * g.C + c) * g.S + s;
                    s1 += part[2 * q + 0];
                    s2 += part[2 * q + 1];
                }
        const double nc = (double)g.T * g.N * g.S;
        const double mu = s1 / nc;
        double var = s2 / nc - mu * mu;
        var = var > 0.0 ? var : 0.0;
        const double inv = 1.0 / sqrt(var + (double)eps);
        const double sc = (double)gamma[c] * inv;
        for (int i = 0; i < g.k; ++i)
            w_f[(size_t)c * g.k + i] = (float)(sc * (double)w[(size_t)c * g.k + i]);
        b_f[c] = (float)((double)beta[c] - sc * mu);
        aux[4 * (size_t)c + 0] = mu;
        aux[4 * (size_t)c + 1] = var;
        aux[4 * (size_t)c + 2] = sc;
        aux[4 * (size_t)c + 3] = inv;
        if (stats != nullptr) {
            stats[2 * (size_t)c + 0] = s1;
            stats[2 * (size_t)c + 1] = s2;
        }
    }
}

// per channel: gradients of gamma and beta, and dTv = a + b Tv
__global__ __launch_bounds__(kBnThreads) void bn_coef(BnGeom g, const float* __restrict__ w,
                                                      const double* __restrict__ aux, float eps,
                                                      const float* __restrict__ grad_wf,
                                                      const float* __restrict__ grad_bf, double* __restrict__ coef,
                                                      float* __restrict__ grad_gamma, float* __restrict__ grad_beta)
{
    for (int c = blockIdx.x * kBnThreads + threadIdx.x; c < g.C; c += gridDim.x * kBnThreads) {
        const double mu = aux[4 * (size_t)c + 0], var = aux[4 * (size_t)c + 1];
        const double sc = aux[4 * (size_t)c + 2], inv = aux[4 * (size_t)c + 3];
        const double gbf = (double)grad_bf[c];
        double dsc = 0.0;
        for (int i = 0; i < g.k; ++i)
            dsc += (double)grad_wf[(size_t)c * g.k + i] * (double)w[(size_t)c * g.k + i];
        dsc -= gbf * mu;
        grad_gamma[c] = (float)(dsc * inv);
        grad_beta[c] = (float)gbf;
        const double dvar = -dsc * sc / (2.0 * (var + (double)eps));
        const double dmu = -sc * gbf;
        const double nc = (double)g.T * g.N * g.S;
        const double b = 2.0 * dvar / nc;
        const double a = dmu / nc - b * mu;
        coef[2 * (size_t)c + 0] = a;
        coef[2 * (size_t)c + 1] = b;
    }
}

// dTv of every element (kept in the workspace)
__global__ __launch_bounds__(kBnThreads) void bn_dtv(BnGeom g, const float* __restrict__ x,
                                                     const float* __restrict__ w, const double* __restrict__ coef,
                                                     double* __restrict__ dtv)
{
    const size_t total = (size_t)g.T * g.M;
    for (size_t e = (size_t)blockIdx.x * kBnThreads + threadIdx.x; e < total; e += (size_t)gridDim.x * kBnThreads) {
        const size_t col = e % g.M;
        const int64_t t = (int64_t)(e / g.M);
        const int c = channel_of(col, g);
        const double v = latent_conv(x, g.M, t, col, w + (size_t)c * g.k, g.k, g.d);
        dtv[e] = coef[2 * c + 0] + coef[2 * c + 1] * v;
    }
}

// grad_x += sum_i W[c,i] dTv[t + (k-1-i)d]  (ascending i, terms past T left out)
__global__ __launch_bounds__(kBnThreads) void bn_gx(BnGeom g, const float* __restrict__ w,
                                                    const double* __restrict__ dtv, float* __restrict__ grad_x)
{
    const size_t total = (size_t)g.T * g.M;
    for (size_t e = (size_t)blockIdx.x * kBnThreads + threadIdx.x; e < total; e += (size_t)gridDim.x * kBnThreads) {
        const size_t col = e % g.M;
        const int64_t t = (int64_t)(e / g.M);
        const int c = channel_of(col, g);
        double acc = 0.0;
        for (int i = 0; i < g.k; ++i) {
            const int64_t to = t + (int64_t)(g.k - 1 - i) * g.d;
            if (to < g.T)
                acc = acc + (double)w[(size_t)c * g.k + i] * dtv[(size_t)to * g.M + col];
        }
        grad_x[e] = (float)((double)grad_x[e] + acc);
    }
}

// per (column, tap): sum_t dTv[t] x[t-(k-1-i)d]
__global__ __launch_bounds__(kBnThreads) void bn_gw_partial(BnGeom g, const float* __restrict__ x,
                                                            const double* __restrict__ dtv,
                                                            double* __restrict__ part)
{
    const size_t total = (size_t)g.M * g.k;
    for (size_t q = (size_t)blockIdx.x * kBnThreads + threadIdx.x; q < total; q += (size_t)gridDim.x * kBnThreads) {
        const size_t col = q % g.M;
        const int i = (int)(q / g.M);
        const int64_t off = (int64_t)(g.k - 1 - i) * g.d;
        double acc = 0.0;
        for (int64_t t = off; t < g.T; ++t)
            acc += dtv[(size_t)t * g.M + col] * (double)x[(size_t)(t - off) * g.M + col];
        part[q] = acc;
    }
}

// per (channel, tap): grad_w = s grad_wf + the partials in (n, s) order
__global__ __launch_bounds__(kBnThreads) void bn_gw_final(BnGeom g, const double* __restrict__ part,
                                                          const double* __restrict__ aux,
                                                          const float* __restrict__ grad_wf,
                                                          float* __restrict__ grad_w)
{
    const size_t total = (size_t)g.C * g.k;
    for (size_t e = (size_t)blockIdx.x * kBnThreads + threadIdx.x; e < total; e += (size_t)gridDim.x * kBnThreads) {
        const int c = (int)(e / g.k), i = (int)(e - (size_t)c * g.k);
        double acc = 0.0;
        for (int n = 0; n < g.N; ++n)
            for (int s = 0; s < g.S; ++s)
                acc += part[(size_t)i * g.M + ((size_t)n * g.C + c) * g.S + s];
        const double direct = aux[4 * (size_t)c + 2] * (double)grad_wf[e];
        grad_w[e] = (float)(direct + acc);
    }
}

unsigned grid_for(size_t items)
{
    size_t b = (items + kBnThreads - 1) / kBnThreads;
    return (unsigned)(b < 1 ? 1 : (b > 65536 ? 65536 : b));
}

}  // namespace

size_t bn_workspace_bytes(const BnGeom& g)
{
    const size_t fwd = (size_t)g.chunks * g.M * 2 * sizeof(double);
    const size_t bwd = ((size_t)g.C * 2 + (size_t)g.T * g.M + (size_t)g.M * g.k) * sizeof(double);
    return fwd > bwd ? fwd : bwd;
}

hipError_t launch_bn_forward_stats(const BnGeom& g, const float* x, const float* w, const float* gamma,
                                   const float* beta, float eps, float* w_f, float* b_f, double* aux,
                                   double* stats, void* workspace, hipStream_t st)
{
    double* part = (double*)workspace;
    hipLaunchKernelGGL(bn_stats_partial, dim3(grid_for((size_t)g.chunks * g.M)), dim3(kBnThreads), 0, st, g, x, w,
                       part);
    hipLaunchKernelGGL(bn_fuse, dim3(grid_for(g.C)), dim3(kBnThreads), 0, st, g, part, w, gamma, beta, eps, w_f, b_f,
                       aux, stats);
    return hipGetLastError();
}

hipError_t launch_bn_backward(const BnGeom& g, const float* x, const float* w, const double* aux, float eps,
                              const float* grad_wf, const float* grad_bf, float* grad_x, float* grad_w,
                              float* grad_gamma, float* grad_beta, void* workspace, hipStream_t st)
{
    double* coef = (double*)workspace;
    double* dtv = coef + 2 * (size_t)g.C;
    double* part = dtv + (size_t)g.T * g.M;
    hipLaunchKernelGGL(bn_coef, dim3(grid_for(g.C)), dim3(kBnThreads), 0, st, g, w, aux, eps, grad_wf, grad_bf, coef,
                       grad_gamma, grad_beta);
    hipLaunchKernelGGL(bn_dtv, dim3(grid_for((size_t)g.T * g.M)), dim3(kBnThreads), 0, st, g, x, w, coef, dtv);
    hipLaunchKernelGGL(bn_gx, dim3(grid_for((size_t)g.T * g.M)), dim3(kBnThreads), 0, st, g, w, dtv, grad_x);
    hipLaunchKernelGGL(bn_gw_partial, dim3(grid_for((size_t)g.M * g.k)), dim3(kBnThreads), 0, st, g, x, dtv, part);
    hipLaunchKernelGGL(bn_gw_final, dim3(grid_for((size_t)g.C * g.k)), dim3(kBnThreads), 0, st, g, part, aux, grad_wf,
                       grad_w);
    return hipGetLastError();
}

}  // namespace mfpsn
