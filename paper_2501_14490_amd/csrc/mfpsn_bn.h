// Internal interface of the batch-normalization kernels (mfpsn_bn.hip) for
// the C-ABI layer.  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace mfpsn {

struct BnGeom {
    int32_t T, N, C, S, k, d;
    size_t M;        // N*C*S
    int32_t tq, tr;  // T = tq * d + tr: class r has tq + (r < tr) steps
    int32_t lc;      // class steps per walk chunk
    int32_t nch;     // chunks per class, ceil(ceil(T/d) / lc)
    size_t items;    // walk items, nch * d * M
    size_t G;        // walk threads: thread t takes items t, t + G, ...; all of
                     // them in channel ((t mod S*C) / S) (G is a multiple of
                     // S*C and of the block size, or no thread has two items)
    int32_t R;       // partial rows, ceil(G / (S*C)): thread t = row * S*C + j
    int32_t NG;      // row groups of the first reduction level, ceil(R / kBnRowGroup)
};
constexpr int kBnThreads = 256;
constexpr int kBnRowGroup = 16;

size_t bn_workspace_bytes(const BnGeom& g);
hipError_t launch_bn_forward_stats(const BnGeom& g, const float* x, const float* w, const float* gamma,
                                   const float* beta, float eps, float* w_f, float* b_f, double* aux,
                                   double* stats, void* workspace, hipStream_t stream);
hipError_t launch_bn_backward(const BnGeom& g, const float* x, const float* w, const double* aux, float eps,
                              const float* grad_wf, const float* grad_bf, float* grad_x, float* grad_w,
                              float* grad_gamma, float* grad_beta, void* workspace, hipStream_t stream);

}  // namespace mfpsn
