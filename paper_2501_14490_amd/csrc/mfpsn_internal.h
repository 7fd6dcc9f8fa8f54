// Internal interface between the C-ABI layer (mfpsn_api.cpp) and the gfx950
// kernels (mfpsn_kernels.hip).  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace mfpsn {

enum Dtype : int32_t { kF32 = 0, kBF16 = 1, kQ88 = 2 };

// How the 64 lanes of a wave map onto the columns (n, c, s) of x[T][N][C][S].
//   kLaneChannel (S == 1, C >= 64): lane l is channel 64*g + l of one sample n;
//       a wave's loads are 64 consecutive channels (coalesced) and every lane
//       owns a different channel, so grad_w needs no cross-lane reduction.
//   kPlane (S >= 2, or C < 64): every lane of a block shares one channel c
//       (taps are wave-uniform); a wave covers 64 consecutive positions
//       n*S + s of the channel's (n, s) plane.
//   kFlat (forward, S a multiple of nv): a wave covers 64*nv consecutive
//       columns of the flattened row of M = N*C*S columns, 16 (or 8) bytes
//       per lane; every lane loads the taps of its own channel (S % nv == 0
//       keeps a lane's nv columns in one channel).
enum Mode : int32_t { kLaneChannel = 0, kPlane = 1, kFlat = 2 };

// Launch geometry, computed on the host by plan() and passed by value.
struct Geom {
    int32_t T, N, C, S;
    int32_t k, d;
    int32_t mode;
    int32_t nv;        // adjacent columns per lane: 1, or 2 (plane mode, S even), or
                       // 2, 4, 8 (flat mode)
    int32_t tiles;     // tiles per group: lane-channel N; plane ceil(N*S/(64*nv)),
                       // or N * row_tiles with line-aligned rows; flat ceil(M/(64*nv))
    int32_t row_tiles; // plane tiles per (n, c) row when tiles follow 128-byte lines
                       // within each row (0: tiles run over the flattened (n, s) plane)
    int32_t line_elems;// elements per 128-byte line (128 / esize)
    int32_t tq, tr;    // T = tq * d + tr
    int32_t ncls;      // residue classes with a step: min(d, T) (at least 1)
    int32_t nchunks;   // time chunks per residue class
    int32_t chunk;     // class steps per chunk
    int32_t cap;       // longest run of class steps one walk may span (a multiple
                       // of k: its rows keep every 32-bit buffer offset in range)
    int32_t run_max;   // consecutive chunks of one class that one walk takes
    int32_t groups;    // gridDim.y: channel groups (lane-channel), channels (plane) or 1 (flat)
    int32_t blocks;    // gridDim.x: blocks per group (set by the launcher; the
                       // planner's value is the upper bound the workspace is sized for)
    int64_t items;     // items per group = tiles * d * nchunks (< 2^31)
    int32_t strided;   // 1: wave w takes items w, w + nw, ... (nw waves per group);
                       // 0: a contiguous range of items
    uint32_t M;        // N*C*S, columns per time step
    int32_t esize;     // bytes per stored element of x / grad_spikes
    int32_t shift_lo, shift_hi;
    int32_t sg;        // surrogate kind
    float alpha, v_th;
    int32_t v_th_q;
    // A float tap's product x * (sign 2^-shift) is exact for every shift in
    // [shift_lo, shift_hi] when x is zero or fast_lo <= |x| < fast_hi; such
    // inputs add their terms with one fused multiply-add, the others (tiny,
    // huge, infinite, NaN) round the product first, then add.
    float fast_lo, fast_hi;
    // 1: every stored input has exact tap products, so the inputs are not
    // checked (bf16 storage with shifts in [0, 16]: an input is m 2^e with
    // |m| < 2^8 and e >= -133, so m 2^(e - s) is a float for s <= 16 and
    // never grows for s >= 0; infinities and NaN give the same result either
    // way)
    int32_t x_exact;
};

// Columns per lane of the flat forward: 16 bytes of x per lane up to order
// 8, 8 bytes up to order 16 (the ring holds k*nv values per lane); 0: none
// (higher orders).
constexpr int flat_nv(int k, int dtype)
{
    const int es = dtype == kF32 ? 4 : 2;
    return k <= 8 ? 16 / es : (k <= 16 ? 8 / es : 0);
}

constexpr int kWaves = 4;          // waves per block
constexpr int kPairMaxK = 16;      // highest order with two-column (nv = 2) kernels
constexpr int kThreads = 64 * kWaves;
constexpr int64_t kMaxGroupItems = ((int64_t)1 << 31) - 1;  // items of one group

// Chunks of the residue classes for the backward's `waves` resident waves per
// group (host).  A wave's items are a contiguous range, and the consecutive
// chunks of one class in it are walked as one (up to run_max of them), so a
// chunk costs no halo of its own: the chunk length only decides how evenly
// the ranges can be cut.  Candidates are the whole class (at most cap steps)
// and its halvings down to k steps; the estimate of the longest range is
// ceil(items / waves) chunks of the mean chunk length, plus one halo of k - 1
// steps when a class is cut.  Ties keep the longer chunk.
inline void balance_chunks(Geom& g, int64_t waves)
{
    const int64_t K = g.k;
    const int64_t L = g.T > 0 ? ((int64_t)g.T + g.d - 1) / g.d : 0;  // the longest class
    if (L == 0 || waves < 1 || g.cap < K)
        return;
    const int64_t base = (int64_t)g.tiles * g.ncls;
    const double halo = (double)(K - 1);
    int64_t c = (L + K - 1) / K * K;
    if (c > g.cap)
        c = g.cap;
    int64_t best_c = 0;
    double best = 0.0;
    for (;;) {
        const int64_t n = (L + c - 1) / c;
        const int64_t items = base * n;
        if (items <= kMaxGroupItems) {
            const double cost =
                (double)((items + waves - 1) / waves) * ((double)L / (double)n) + (n > 1 ? halo : 0.0);
            if (best_c == 0 || cost < best) {
                best = cost;
                best_c = c;
            }
        }
        const int64_t h = (c / 2 + K - 1) / K * K;
        if (h < K || h >= c)
            break;
        c = h;
    }
    if (best_c == 0)
        return;
    g.chunk = (int32_t)best_c;
    g.nchunks = (int32_t)((L + best_c - 1) / best_c);
    g.items = base * g.nchunks;
    g.run_max = (int32_t)(g.cap / best_c > 0 ? g.cap / best_c : 1);
}
// Upper bound of blocks resident on one GPU at once (8 blocks of 4 waves per
// CU is 8 waves per SIMD; 320 CUs covers every CDNA part): the persistent grid
// never exceeds it, so it also bounds the backward's partial rows.
constexpr int kMaxResidentBlocks = 8 * 320;

struct FwdArgs {
    Geom g;
    const void* x;
    const int8_t* sign;
    const int8_t* shift;
    const void* bias;
    const void* v_th_c;  // nullable: per-channel thresholds, float or int32 [C]
    uint8_t* spikes;
    void* h_out;       // nullable: potentials H
    void* sg_out;      // nullable: surrogate factor of H
};

struct BwdArgs {
    Geom g;
    const void* x;
    const void* gs;
    const void* h;     // potentials H saved by the forward (nullable)
    const void* sg;    // surrogate factor saved by the forward (nullable; used if set)
    const int8_t* sign;
    const int8_t* shift;
    const void* bias;
    const void* v_th_c;  // nullable: per-channel thresholds, float or int32 [C]
    void* grad_x;
    double* partial;   // [blocks][k+1][C]
};

struct FinArgs {
    int32_t C, k, blocks, dtype;
    const double* partial;
    void* grad_w;
    void* grad_b;
    void* grad_vth;    // nullable: -grad_b
};

// The launchers size the persistent grid from the kernel's occupancy and
// store the blocks per group they launched in a.g.blocks.
template <int K, int DT> hipError_t fwd_k(FwdArgs& a, hipStream_t stream);
template <int K, int DT> hipError_t bwd_k(BwdArgs& a, hipStream_t stream);

hipError_t launch_forward(FwdArgs& a, int dtype, hipStream_t stream);
hipError_t launch_backward(BwdArgs& a, int dtype, hipStream_t stream);
hipError_t launch_finalize(const FinArgs& a, hipStream_t stream);
hipError_t launch_quantize(const float* w, int64_t count, int32_t lo, int32_t hi, int8_t* sign,
                           int8_t* shift, hipStream_t stream);

}  // namespace mfpsn
