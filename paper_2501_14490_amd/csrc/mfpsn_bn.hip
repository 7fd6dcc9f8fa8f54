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
// is the same double on both sides of the parity tests.  Each pass walks the
// residue classes of the dilation in chunks, one thread per (chunk, class,
// column), with the last k inputs in registers (every input loaded once per
// pass).  The per-channel reductions are deterministic: each thread sums over
// its own items (all in one channel), and two further levels add those
// partials in a fixed order.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>

#include "mfpsn.h"
#include "mfpsn_bn.h"

namespace mfpsn {
namespace {

__device__ __forceinline__ int channel_of(size_t col, const BnGeom& g) { return (int)((col / g.S) % g.C); }

// Fixed-order sum of a block's per-thread values (a binary tree in LDS):
// the result does not depend on scheduling
__device__ __forceinline__ double block_sum(double v, double* red)
{
    red[threadIdx.x] = v;
    __syncthreads();
    for (int h = kBnThreads / 2; h > 0; h >>= 1) {
        if ((int)threadIdx.x < h)
            red[threadIdx.x] = red[threadIdx.x] + red[threadIdx.x + h];
        __syncthreads();
    }
    const double r = red[0];
    __syncthreads();
    return r;
}

// Walk items: (chunk ch, residue class r, column col), col fastest:
// q = (ch * d + r) * M + col.  A thread walks the class steps j of class r
// (time r + j d) over its chunk [j0, j1) and keeps the last K inputs of the
// class in a register ring, so every input is loaded once per pass.  The
// step loop runs in blocks of K steps, unrolled, so the ring slot of every
// step is fixed at compile time (no register moves), and each block issues
// the loads of the next one (K steps of latency to hide).
struct WalkItem {
    size_t col;
    int r, j0, j1, Lr, c;
};
__device__ __forceinline__ WalkItem walk_item(const BnGeom& g, size_t q)
{
    WalkItem it;
    it.col = q % g.M;
    const size_t cr = q / g.M;
    it.r = (int)(cr % g.d);
    const int ch = (int)(cr / g.d);
    it.Lr = g.tq + (it.r < g.tr ? 1 : 0);
    it.j0 = ch * g.lc;
    it.j1 = min(it.Lr, it.j0 + g.lc);
    it.c = channel_of(it.col, g);
    return it;
}
// element offset of class step j of the item's column (j >= 0)
__device__ __forceinline__ size_t row_of(const BnGeom& g, const WalkItem& it, int j)
{
    return ((size_t)it.r + (size_t)j * g.d) * g.M + it.col;
}

template <int K>
__device__ __forceinline__ void load_weights(const float* __restrict__ wc, double (&wd)[K])
{
#pragma unroll
    for (int i = 0; i < K; ++i)
        wd[i] = (double)wc[i];
}

// Tv from the ring, taps in ascending order from +0.  slot(i) is the ring
// slot of the input tap i reads.  A product of two floats is exact in double,
// so the fused multiply-add rounds exactly as a product and a sum do; an
// input before time 0 sits in the ring as 0 and adds a zero, which leaves the
// sum as it is (the sum is never -0), as leaving the tap out does.
template <int K, typename Slot>
__device__ __forceinline__ double ring_conv(const double (&ring)[K], const double (&wd)[K], Slot slot)
{
    double acc = 0.0;
#pragma unroll
    for (int i = 0; i < K; ++i)
        acc = __builtin_fma(wd[i], ring[slot(i)], acc);
    return acc;
}

// A forward walk over the item's steps [j0, j1) (j1 > j0).  Ring slot of
// class step t: (t - j0) mod K, so step j0 + bK + u reads tap i from slot
// (u + i + 1) mod K and stores its own input in slot u.  step(v, u) gets Tv
// of the step and u; the ring is visible to it through the reference.
template <int K, typename Step>
__device__ __forceinline__ void forward_walk(const BnGeom& g, const WalkItem& it, const float* __restrict__ x,
                                             const double (&wd)[K], double (&ring)[K], Step&& step)
{
    const ptrdiff_t drow = (ptrdiff_t)g.d * (ptrdiff_t)g.M;
    const size_t last = row_of(g, it, it.j1 - 1);
    ring[0] = 0.0;
#pragma unroll
    for (int m = 1; m < K; ++m) {  // steps j0-K+1 .. j0-1, 0 before time 0
        const int jj = it.j0 - K + m;
        const float v = x[row_of(g, it, jj > 0 ? jj : 0)];
        ring[m] = jj >= 0 ? (double)v : 0.0;
    }
    // stage[u]: x of the step that takes slot u next; the next load's offset
    // runs one class row per step, clamped to the last step of the item
    float stage[K];
    size_t nxt = row_of(g, it, it.j0);
#pragma unroll
    for (int u = 0; u < K; ++u, nxt += drow)
        stage[u] = x[nxt < last ? nxt : last];
    const int n = it.j1 - it.j0, nfull = n / K, rem = n - nfull * K;
    for (int b = 0; b < nfull; ++b) {
#pragma unroll
        for (int u = 0; u < K; ++u, nxt += drow) {
            ring[u] = (double)stage[u];
            stage[u] = x[nxt < last ? nxt : last];
            step(ring_conv<K>(ring, wd, [u](int i) { return (u + i + 1) % K; }), u);
        }
    }
#pragma unroll
    for (int u = 0; u < K; ++u)
        if (u < rem) {
            ring[u] = (double)stage[u];
            step(ring_conv<K>(ring, wd, [u](int i) { return (u + i + 1) % K; }), u);
        }
}

// The shift of channel c's statistics: Tv of the channel's last time step at
// its first column (n = 0, s = 0), taps in ascending order.  Every element of
// the channel is summed as Tv - pivot, so the variance comes from sums of
// deviations from a value near the mean instead of the difference of two
// large sums (which would cancel when |mean| >> standard deviation).
__device__ __forceinline__ double pivot_tv(const BnGeom& g, const float* __restrict__ x,
                                           const float* __restrict__ w, int c)
{
    const int t = g.T - 1;
    const size_t col = (size_t)c * g.S;
    double acc = 0.0;
    for (int i = 0; i < g.k; ++i) {
        const int64_t tau = (int64_t)t - (int64_t)(g.k - 1 - i) * g.d;
        if (tau >= 0)
            acc = __builtin_fma((double)w[(size_t)c * g.k + i], (double)x[(size_t)tau * g.M + col], acc);
    }
    return acc;
}

// statistics partials: thread t's sums of Tv - pivot and (Tv - pivot)^2 over
// the steps of all its items (one channel), written to part[t] and
// part[G + t]
template <int K>
__global__ __launch_bounds__(kBnThreads) void bn_stats_walk(BnGeom g, const float* __restrict__ x,
                                                            const float* __restrict__ w, double* __restrict__ part)
{
    const size_t t = (size_t)blockIdx.x * kBnThreads + threadIdx.x;
    double s1 = 0.0, s2 = 0.0;
    for (size_t q = t; q < g.items; q += g.G) {
        const WalkItem it = walk_item(g, q);
        if (it.j1 > it.j0) {
            double wd[K], ring[K];
            load_weights<K>(w + (size_t)it.c * K, wd);
            const double p = pivot_tv(g, x, w, it.c);
            forward_walk<K>(g, it, x, wd, ring, [&](double v, int) {
                const double e = v - p;
                s1 = s1 + e;
                s2 = __builtin_fma(e, e, s2);
            });
        }
    }
    part[t] = s1;
    part[g.G + t] = s2;
}

// First level of the per-channel sums: for each value v < nval and column
// j < S*C, the partials of threads row*S*C + j summed over the rows of one
// group of kBnRowGroup rows, in row order, to inter[(v * NG + group) * SC + j]
__global__ __launch_bounds__(kBnThreads) void bn_rows(BnGeom g, int nval, const double* __restrict__ part,
                                                      double* __restrict__ inter)
{
    const size_t SC = (size_t)g.S * g.C, per_v = (size_t)g.NG * SC, total = (size_t)nval * per_v;
    for (size_t e = (size_t)blockIdx.x * kBnThreads + threadIdx.x; e < total; e += (size_t)gridDim.x * kBnThreads) {
        const size_t v = e / per_v, rest = e - v * per_v, grp = rest / SC, j = rest - grp * SC;
        const size_t r0 = grp * kBnRowGroup, r1 = min((size_t)g.R, r0 + kBnRowGroup);
        double acc = 0.0;
        for (size_t r = r0; r < r1; ++r) {
            const size_t tt = r * SC + j;
            if (tt < g.G)
                acc += part[v * g.G + tt];
        }
        inter[e] = acc;
    }
}

// second level: channel c's entries of value v, (group, s) for s < S, as a
// list that thread j of a block reads at j, j+256, ... (then the tree)
__device__ __forceinline__ double channel_sum(const BnGeom& g, const double* __restrict__ inter, int v, int c,
                                              double* red)
{
    const size_t SC = (size_t)g.S * g.C, n = (size_t)g.NG * g.S;
    double a = 0.0;
    for (size_t e = threadIdx.x; e < n; e += kBnThreads) {
        const size_t grp = e / g.S, sp = e - grp * g.S;
        a += inter[((size_t)v * g.NG + grp) * SC + (size_t)c * g.S + sp];
    }
    return block_sum(a, red);
}

// one block per channel: the sums, the statistics and the fusion
__global__ __launch_bounds__(kBnThreads) void bn_fuse(BnGeom g, const double* __restrict__ inter,
                                                      const float* __restrict__ x,
                                                      const float* __restrict__ w, const float* __restrict__ gamma,
                                                      const float* __restrict__ beta, float eps,
                                                      float* __restrict__ w_f, float* __restrict__ b_f,
                                                      double* __restrict__ aux, double* __restrict__ stats)
{
    __shared__ double red[kBnThreads];
    for (int c = blockIdx.x; c < g.C; c += gridDim.x) {
        const double s1 = channel_sum(g, inter, 0, c, red);  // sum of Tv - pivot
        const double s2 = channel_sum(g, inter, 1, c, red);  // sum of (Tv - pivot)^2
        if (threadIdx.x == 0) {
            const double nc = (double)g.T * g.N * g.S;
            const double p = nc > 0 ? pivot_tv(g, x, w, c) : 0.0;
            const double dm = nc > 0 ? s1 / nc : 0.0;  // mean - pivot
            const double mu = p + dm;
            double var = nc > 0 ? s2 / nc - dm * dm : 0.0;
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
                // sum Tv and sum Tv^2 from the shifted sums
                stats[2 * (size_t)c + 0] = nc * p + s1;
                stats[2 * (size_t)c + 1] = s2 + 2.0 * p * s1 + nc * p * p;
            }
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
#pragma unroll 8
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

// The backward of the statistics path in one reverse walk per item, steps
// jtop down to j0 (jtop: up to K-1 steps above the chunk, which only feed
// outputs of the chunk).  Step j gives dTv[j] = a + b Tv[j] and
//  - its terms W[i] dTv[j] for the input gradients j-(K-1-i): each output
//    collects its terms in a register, from i = 0 to K-1 (ascending taps, as
//    the steps descend), and is complete after its own step, when grad_x[j]
//    gets it;
//  - for a step of the chunk, its terms dTv[j] x[j-(K-1-i)] of the weight
//    gradient, summed per thread over all its items (one channel) and
//    written to part[i * G + t].
// Slot of class step t, in the ring and among the outputs: (jtop - t) mod K.
template <int K>
__global__ __launch_bounds__(kBnThreads) void bn_bwd_walk(BnGeom g, const float* __restrict__ x,
                                                         const float* __restrict__ w, const double* __restrict__ coef,
                                                         float* __restrict__ grad_x, double* __restrict__ part)
{
    const size_t t = (size_t)blockIdx.x * kBnThreads + threadIdx.x;
    double gw[K];
#pragma unroll
    for (int i = 0; i < K; ++i)
        gw[i] = 0.0;
    const ptrdiff_t drow = (ptrdiff_t)g.d * (ptrdiff_t)g.M;
    for (size_t q = t; q < g.items; q += g.G) {
        const WalkItem it = walk_item(g, q);
        if (it.j0 >= it.j1)
            continue;
        // the coefficients and weights are loaded first, so that the first
        // step waits for the oldest loads only (the compiler's wait
        // placement, common to every pass through the step loop, then leaves
        // the ring's loads in flight)
        const double ca = coef[2 * it.c + 0], cb = coef[2 * it.c + 1];
        double wd[K];
        load_weights<K>(w + (size_t)it.c * K, wd);
        __builtin_amdgcn_sched_barrier(0);
        const int jtop = min(it.j1 + K - 1, it.Lr) - 1;
        const size_t first = row_of(g, it, 0);
        double ring[K], A[K];
#pragma unroll
        for (int m = 0; m < K; ++m) {  // steps jtop .. jtop-K+1, 0 before time 0
            const int jj = jtop - m;
            const float v = x[row_of(g, it, jj > 0 ? jj : 0)];
            ring[m] = jj >= 0 ? (double)v : 0.0;
            A[m] = 0.0;
        }
        // stage[u]: x of step jtop-K-u (entering slot u), gstage[u]: grad_x
        // of step jtop-u (leaving slot u); offsets run down one class row per
        // step, clamped to step 0, and an input before time 0 enters as 0
        float stage[K], gstage[K];
        ptrdiff_t xo = (ptrdiff_t)row_of(g, it, jtop) - (ptrdiff_t)K * drow;
        ptrdiff_t go = (ptrdiff_t)row_of(g, it, jtop);
#pragma unroll
        for (int u = 0; u < K; ++u, xo -= drow, go -= drow) {
            stage[u] = x[xo > (ptrdiff_t)first ? xo : (ptrdiff_t)first];
            gstage[u] = grad_x[go > (ptrdiff_t)first ? go : (ptrdiff_t)first];
        }
        const int n = jtop - it.j0 + 1, nfull = n / K, rem = n - nfull * K;
        ptrdiff_t so = (ptrdiff_t)row_of(g, it, jtop);  // grad_x element of the current step
        auto step = [&](int u, int j) {
            const double v = ring_conv<K>(ring, wd, [u](int i) { return (u + K - 1 - i) % K; });
            const double dtv = ca + cb * v;
#pragma unroll
            for (int i = 0; i < K; ++i) {
                const int o = (u + K - 1 - i) % K;
                A[o] = A[o] + wd[i] * dtv;
            }
            if (j < it.j1) {
                grad_x[so] = (float)((double)gstage[u] + A[u]);
#pragma unroll
                for (int i = 0; i < K; ++i)
                    gw[i] = __builtin_fma(dtv, ring[(u + K - 1 - i) % K], gw[i]);
            }
            A[u] = 0.0;
            ring[u] = j - K >= 0 ? (double)stage[u] : 0.0;
        };
        int j = jtop;
        for (int b = 0; b < nfull; ++b) {
#pragma unroll
            for (int u = 0; u < K; ++u, --j, xo -= drow, go -= drow, so -= drow) {
                step(u, j);
                stage[u] = x[xo > (ptrdiff_t)first ? xo : (ptrdiff_t)first];
                gstage[u] = grad_x[go > (ptrdiff_t)first ? go : (ptrdiff_t)first];
            }
        }
#pragma unroll
        for (int u = 0; u < K; ++u, --j, so -= drow)
            if (u < rem)
                step(u, j);
    }
#pragma unroll
    for (int i = 0; i < K; ++i)
        part[(size_t)i * g.G + t] = gw[i];
}

// one block per (channel, tap): grad_w = s grad_wf + the channel's sum
__global__ __launch_bounds__(kBnThreads) void bn_gw_final(BnGeom g, const double* __restrict__ inter,
                                                          const double* __restrict__ aux,
                                                          const float* __restrict__ grad_wf,
                                                          float* __restrict__ grad_w)
{
    __shared__ double red[kBnThreads];
    const size_t total = (size_t)g.C * g.k;
    for (size_t e = blockIdx.x; e < total; e += gridDim.x) {
        const int c = (int)(e / g.k), i = (int)(e - (size_t)c * g.k);
        const double acc = channel_sum(g, inter, i, c, red);
        if (threadIdx.x == 0)
            grad_w[e] = (float)(aux[4 * (size_t)c + 2] * (double)grad_wf[e] + acc);
    }
}

unsigned blocks_for(size_t outputs) { return (unsigned)(outputs < 1 ? 1 : (outputs > 65536 ? 65536 : outputs)); }
unsigned grid_for(size_t threads) { return blocks_for((threads + kBnThreads - 1) / kBnThreads); }
// the walks: exactly G threads (the partial layout depends on it)
dim3 walk_grid(const BnGeom& g) { return dim3((unsigned)(g.G / kBnThreads)); }

template <int K>
void launch_stats_k(const BnGeom& g, const float* x, const float* w, double* part, hipStream_t st)
{
    hipLaunchKernelGGL(bn_stats_walk<K>, walk_grid(g), dim3(kBnThreads), 0, st, g, x, w, part);
}
template <int K>
void launch_bwd_k(const BnGeom& g, const float* x, const float* w, const double* coef, float* grad_x, double* part,
                  hipStream_t st)
{
    hipLaunchKernelGGL(bn_bwd_walk<K>, walk_grid(g), dim3(kBnThreads), 0, st, g, x, w, coef, grad_x, part);
}
template <int... Ks>
void stats_dispatch(const BnGeom& g, const float* x, const float* w, double* part, hipStream_t st,
                    std::integer_sequence<int, Ks...>)
{
    (void)((g.k == Ks + 1 ? (launch_stats_k<Ks + 1>(g, x, w, part, st), true) : false) || ...);
}
template <int... Ks>
void bwd_dispatch(const BnGeom& g, const float* x, const float* w, const double* coef, float* grad_x, double* part,
                  hipStream_t st, std::integer_sequence<int, Ks...>)
{
    (void)((g.k == Ks + 1 ? (launch_bwd_k<Ks + 1>(g, x, w, coef, grad_x, part, st), true) : false) || ...);
}
using BnOrders = std::make_integer_sequence<int, MFPSN_MAX_K>;

}  // namespace

// workspace: [coef: 2C][part: G * max(k, 2)][inter: max(k, 2) * NG * S*C] doubles
size_t bn_workspace_bytes(const BnGeom& g)
{
    const size_t nval = g.k > 2 ? (size_t)g.k : 2;
    return ((size_t)2 * g.C + g.G * nval + nval * g.NG * (size_t)g.S * g.C) * sizeof(double);
}
namespace {
struct BnWork {
    double *coef, *part, *inter;
};
BnWork carve(const BnGeom& g, void* workspace)
{
    const size_t nval = g.k > 2 ? (size_t)g.k : 2;
    BnWork w;
    w.coef = (double*)workspace;
    w.part = w.coef + 2 * (size_t)g.C;
    w.inter = w.part + g.G * nval;
    return w;
}
}  // namespace

hipError_t launch_bn_forward_stats(const BnGeom& g, const float* x, const float* w, const float* gamma,
                                   const float* beta, float eps, float* w_f, float* b_f, double* aux,
                                   double* stats, void* workspace, hipStream_t st)
{
    const BnWork ws = carve(g, workspace);
    stats_dispatch(g, x, w, ws.part, st, BnOrders{});
    hipLaunchKernelGGL(bn_rows, dim3(grid_for((size_t)2 * g.NG * g.S * g.C)), dim3(kBnThreads), 0, st, g, 2, ws.part,
                       ws.inter);
    hipLaunchKernelGGL(bn_fuse, dim3(blocks_for(g.C)), dim3(kBnThreads), 0, st, g, ws.inter, x, w, gamma, beta, eps,
                       w_f, b_f, aux, stats);
    return hipGetLastError();
}

hipError_t launch_bn_backward(const BnGeom& g, const float* x, const float* w, const double* aux, float eps,
                              const float* grad_wf, const float* grad_bf, float* grad_x, float* grad_w,
                              float* grad_gamma, float* grad_beta, void* workspace, hipStream_t st)
{
    const BnWork ws = carve(g, workspace);
    hipLaunchKernelGGL(bn_coef, dim3(grid_for(g.C)), dim3(kBnThreads), 0, st, g, w, aux, eps, grad_wf, grad_bf,
                       ws.coef, grad_gamma, grad_beta);
    bwd_dispatch(g, x, w, ws.coef, grad_x, ws.part, st, BnOrders{});
    hipLaunchKernelGGL(bn_rows, dim3(grid_for((size_t)g.k * g.NG * g.S * g.C)), dim3(kBnThreads), 0, st, g, g.k,
                       ws.part, ws.inter);
    hipLaunchKernelGGL(bn_gw_final, dim3(blocks_for((size_t)g.C * g.k)), dim3(kBnThreads), 0, st, g, ws.inter, aux,
                       grad_wf, grad_w);
    return hipGetLastError();
}

}  // namespace mfpsn
