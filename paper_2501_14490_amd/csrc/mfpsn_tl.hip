// gfx950 kernels of the mul-free channel-wise neuron (arXiv 2501.14490,
// Eqs. mfdpsn_charge, mfdpsn_fire; App. A.3 Eqs. backward_X, backward_W,
// backward_b) for the time-last layout [N][C][S][T] (time innermost, the
// paper's second layout).
//
// Short columns (T <= 64): one wave per group of 64 columns, lane = column,
// the group transposed through LDS (tl_cols_kernel, tl_cols_bwd_kernel).
// Long columns: a wave per segment of consecutive time steps of one column,
// lane = time step, so the channel and its k taps are the same on every lane;
// the segment's inputs and the history its taps read are staged in the
// wave's LDS window with coalesced loads (tl_seg_fwd_kernel,
// tl_seg_bwd_kernel; tl_fwd_kernel for histories above 1024 steps, with the
// next segment's loads in flight while it computes and the taps read from
// global memory past 2048 steps).
//
// The arithmetic is the definition's, as in the time-first kernels: taps in
// ascending order starting from the first one whose input exists (time >= 0),
// bias last, every add rounded; a float tap is x * 2^-shift with the sign
// applied after the scaling, as an integer add to the bit pattern when every
// staged input of the wave lies in the range where that is exact, else as
// v_ldexp_f32 and a sign flip; a Q8.8 tap is an arithmetic right shift and a
// negation after it (integer sums: any order gives the same value).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "mfpsn.h"
#include "mfpsn_surrogate.h"
#include "mfpsn_tl.h"

namespace mfpsn {
namespace {

template <int DT> struct TlIO;
template <> struct TlIO<MFPSN_F32> {
    using V = float;
    static __device__ __forceinline__ V ld(const void* p, int64_t e) { return ((const float*)p)[e]; }
};
template <> struct TlIO<MFPSN_BF16> {
    using V = float;
    static __device__ __forceinline__ V ld(const void* p, int64_t e)
    {
        return __builtin_bit_cast(float, (uint32_t)((const uint16_t*)p)[e] << 16);
    }
};
template <> struct TlIO<MFPSN_Q8_8> {
    using V = int32_t;
    static __device__ __forceinline__ V ld(const void* p, int64_t e) { return (int32_t)((const int16_t*)p)[e]; }
};

__device__ __forceinline__ int uniform_i(int v) { return __builtin_amdgcn_readfirstlane(v); }

// LDS writes of every lane of the wave before any lane reads (a wave's LDS
// operations run in order; this keeps the compiler from moving them)
__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One segment: steps [t0, t0 + 64 NS) of one column; its window of staged
// inputs [ws, we) is the segment and the (K-1) d steps before it
struct TlUnit {
    int64_t cbase;  // flat offset of the column's time 0
    int t0, ws, we, c;
};

// Forward for histories above kTlBwdMaxSpan steps (and T > kTlColsMaxT).
// Persistent waves: wave w takes segments w, w + W, ... (W waves in the
// grid) of 64 NS consecutive time steps of one column, lane l taking steps
// t0 + l + 64 v; the taps are wave-uniform and sit in scalar registers.
// LDS: the segment and the (k-1) d steps before it in the wave's window
// (every tap then reads its input at t - (k-1-i) d: consecutive lanes,
// consecutive addresses), the first NS+2 loads of the next segment's window
// in flight while the current one computes; without LDS (histories above
// kTlMaxHalo) the taps read global memory.
template <int DT, int K, int NS, bool LDS>
__global__ __launch_bounds__(kTlWaves * 64) void tl_fwd_kernel(TlArgs a)
{
    using V = typename TlIO<DT>::V;
    constexpr bool kF = DT != MFPSN_Q8_8;
    constexpr int kW = 64 * NS, kStage = NS + 2;
    extern __shared__ uint32_t tl_lds[];
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6), lane = (int)threadIdx.x & 63;
    const int64_t units = a.M * a.nseg, stride = (int64_t)gridDim.x * kTlWaves;
    const int span = (K - 1) * a.d;
    V* win = reinterpret_cast<V*>(tl_lds) + (size_t)wave * (kW + a.halo);
    auto unit_of = [&](int64_t u) {
        TlUnit q;
        const int64_t col = u / a.nseg;
        q.t0 = (int)(u - col * a.nseg) * kW;
        q.c = (int)((col / a.S) % a.C);
        q.cbase = col * (int64_t)a.T;
        q.ws = q.t0 - span > 0 ? q.t0 - span : 0;
        q.we = q.t0 + kW < a.T ? q.t0 + kW : a.T;
        return q;
    };
    V buf[kStage];
    auto issue = [&](const TlUnit& q) {
#pragma unroll
        for (int j = 0; j < kStage; ++j) {
            const int t = q.ws + lane + 64 * j;
            buf[j] = TlIO<DT>::ld(a.x, q.cbase + (t < q.we ? t : q.we - 1));
        }
    };
    int64_t u = (int64_t)blockIdx.x * kTlWaves + wave;  // wave-uniform
    if (u >= units)
        return;  // no block-wide barrier in this kernel
    TlUnit cur = unit_of(u);
    if constexpr (LDS)
        issue(cur);
    for (; u < units; u += stride) {
        // taps of the segment's channel (wave-uniform): float bit-pattern
        // addend of x * 2^-s with the sign, or the Q8.8 shift and negation
        int sh[K], neg[K];
        uint32_t kc[K];
#pragma unroll
        for (int i = 0; i < K; ++i) {
            int sv = a.shift[cur.c * K + i];
            sv = sv < a.shift_lo ? a.shift_lo : (sv > a.shift_hi ? a.shift_hi : sv);
            const bool n = a.sign[cur.c * K + i] < 0;
            sh[i] = uniform_i(sv);
            neg[i] = uniform_i(n ? -1 : 0);
            kc[i] = (uint32_t)uniform_i((int)(((uint32_t)(-sv) << 23) ^ (n ? 0x80000000u : 0u)));
        }
        V bias;
        if constexpr (kF)
            bias = ((const float*)a.bias)[cur.c];
        else
            bias = ((const int32_t*)a.bias)[cur.c];

        bool slow = !LDS;  // the global-memory variant always takes the exact taps
        TlUnit nxt = cur;
        if constexpr (LDS) {
            bool out = false;
#pragma unroll
            for (int j = 0; j < kStage; ++j) {
                const int t = cur.ws + lane + 64 * j;
                if (t < cur.we) {
                    win[t - cur.ws] = buf[j];
                    if constexpr (kF) {
                        const float m = __builtin_fabsf(buf[j]);
                        out = out || !(m >= a.fast_lo && m < a.fast_hi);
                    }
                }
            }
            for (int t = cur.ws + lane + 64 * kStage; t < cur.we; t += 64) {  // longer histories
                const V v = TlIO<DT>::ld(a.x, cur.cbase + t);
                win[t - cur.ws] = v;
                if constexpr (kF) {
                    const float m = __builtin_fabsf(v);
                    out = out || !(m >= a.fast_lo && m < a.fast_hi);
                }
            }
            slow = __builtin_amdgcn_ballot_w64(out) != 0;
            wave_lds_sync();
            if (u + stride < units) {  // the next segment's loads, in flight during this one
                nxt = unit_of(u + stride);
                issue(nxt);
            }
        }

        // the tap input of output t: time t - (K-1-i) d; EXACT: v_ldexp_f32
        // and a sign flip, else the bit-pattern add (float); Q8.8 shift and
        // negation
        auto tap = [&](V in, int i, auto exact) -> V {
            if constexpr (kF) {
                if constexpr (decltype(exact)::value) {
                    const float y = ldexpf(in, -sh[i]);
                    return neg[i] ? -y : y;
                } else {
                    return __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, in) + kc[i]);
                }
            } else {
                const int32_t y = in >> sh[i];
                return (y ^ neg[i]) - neg[i];
            }
        };
        auto input = [&](int tt) -> V {
            if constexpr (LDS)
                return win[tt - cur.ws];
            else
                return TlIO<DT>::ld(a.x, cur.cbase + tt);
        };
        auto outputs = [&](auto exact) {
#pragma unroll
            for (int v = 0; v < NS; ++v) {
                const int t = cur.t0 + lane + 64 * v;
                if (cur.t0 + 64 * v >= a.T)
                    break;
                // lanes past the column's end compute on its last time step
                // (every address stays inside the window and the column) and
                // store nothing
                const int tc = t < a.T ? t : a.T - 1;
                V in[K];  // all inputs first: the reads issue back to back
#pragma unroll
                for (int i = 0; i < K; ++i) {
                    const int tt = tc - (K - 1 - i) * a.d;
                    in[i] = input(tt > 0 ? tt : 0);
                }
                V acc;
                if (cur.t0 + 64 * v >= span) {
                    // every tap of every lane reads a time >= 0 (wave-uniform)
                    acc = tap(in[0], 0, exact);
#pragma unroll
                    for (int i = 1; i < K; ++i)
                        acc = acc + tap(in[i], i, exact);
                } else {
                    // from the first tap whose input exists
                    const int back = tc / a.d;
                    const int imin = K - 1 - back > 0 ? K - 1 - back : 0;
                    acc = V(0);
#pragma unroll
                    for (int i = 0; i < K; ++i) {
                        const V term = tap(in[i], i, exact);
                        if constexpr (kF)
                            acc = i < imin ? acc : (i == imin ? term : acc + term);
                        else
                            acc = i < imin ? acc : acc + term;
                    }
                }
                if (t >= a.T)
                    continue;
                const V h = acc + bias;
                const int64_t e = cur.cbase + t;
                bool fire;
                if constexpr (kF)
                    fire = h >= a.v_th;
                else
                    fire = h >= a.v_th_q;
                a.spikes[e] = fire ? 1 : 0;
                if (a.h_out != nullptr)
                    reinterpret_cast<V*>(a.h_out)[e] = h;
            }
        };
        if (kF && slow)
            outputs(std::true_type{});
        else
            outputs(std::false_type{});
        if constexpr (LDS) {
            wave_lds_sync();  // every read of the window before the next segment's writes
            cur = nxt;
        } else if (u + stride < units) {
            cur = unit_of(u + stride);
        }
    }
}

typedef uint32_t U32x4 __attribute__((ext_vector_type(4)));

// Four consecutive stored elements (one vector load)
template <int DT> struct TlVec4;
template <> struct TlVec4<MFPSN_F32> {
    static __device__ __forceinline__ void ld(const void* p, int64_t e, float (&v)[4])
    {
        const float4 w = *reinterpret_cast<const float4*>((const float*)p + e);
        v[0] = w.x, v[1] = w.y, v[2] = w.z, v[3] = w.w;
    }
};
template <> struct TlVec4<MFPSN_BF16> {
    static __device__ __forceinline__ void ld(const void* p, int64_t e, float (&v)[4])
    {
        const uint2 w = *reinterpret_cast<const uint2*>((const uint16_t*)p + e);
        v[0] = __builtin_bit_cast(float, w.x << 16), v[1] = __builtin_bit_cast(float, w.x & 0xffff0000u);
        v[2] = __builtin_bit_cast(float, w.y << 16), v[3] = __builtin_bit_cast(float, w.y & 0xffff0000u);
    }
};
template <> struct TlVec4<MFPSN_Q8_8> {
    static __device__ __forceinline__ void ld(const void* p, int64_t e, int32_t (&v)[4])
    {
        const uint2 w = *reinterpret_cast<const uint2*>((const int16_t*)p + e);
        v[0] = (int32_t)(w.x << 16) >> 16, v[1] = (int32_t)w.x >> 16;
        v[2] = (int32_t)(w.y << 16) >> 16, v[3] = (int32_t)w.y >> 16;
    }
};

// The k taps of one lane's channel: for float data the bit-pattern addend
// kc = (-s) 2^23 + sign 2^31 (mod 2^32) of x * 2^-s with the sign (the
// exact path takes -s from bits 23..30 and the sign from what remains once
// (-s) 2^23 is taken away), for Q8.8 the shift and the negation mask.
template <int DT, int K> struct TlLaneTaps {
    static constexpr bool kF = DT != MFPSN_Q8_8;
    using V = typename TlIO<DT>::V;
    uint32_t kc[kF ? K : 1];
    int sh[kF ? 1 : K], neg[kF ? 1 : K];
    int nneg;  // Q8.8: number of negative taps
    __device__ __forceinline__ void load(const int8_t* sign, const int8_t* shift, int c, int lo, int hi)
    {
        nneg = 0;
#pragma unroll
        for (int i = 0; i < K; ++i) {
            int sv = shift[c * K + i];
            sv = sv < lo ? lo : (sv > hi ? hi : sv);
            const bool n = sign[c * K + i] < 0;
            if constexpr (kF) {
                kc[i] = ((uint32_t)(-sv) << 23) ^ (n ? 0x80000000u : 0u);
            } else {
                sh[i] = sv, neg[i] = n ? -1 : 0;
                nneg += n ? 1 : 0;
            }
        }
    }
    // A sum over all k taps (every input exists) as start() followed by
    // accumulate() per tap in ascending order.  Float: +0 and one rounded add
    // per term, as apply().  Q8.8: ((v >> s) ^ m) is +(v >> s) or -(v >> s) - 1,
    // so the sum starts at the number of negative taps and adds it unchanged
    // (integers: the same value).
    __device__ __forceinline__ V start() const
    {
        if constexpr (kF)
            return V(0);
        else
            return nneg;
    }
    template <bool EXACT> __device__ __forceinline__ V accumulate(V acc, V in, int i) const
    {
        if constexpr (kF)
            return acc + apply<EXACT>(in, i);
        else
            return ((in >> sh[i]) ^ neg[i]) + acc;
    }
    // sign * in * 2^-s: EXACT by v_ldexp_f32 and a sign flip, else by the
    // bit-pattern add (exact for |in| in the fast range); Q8.8 floor shift
    // and negation
    template <bool EXACT> __device__ __forceinline__ V apply(V in, int i) const
    {
        if constexpr (kF) {
            if constexpr (EXACT) {
                const int e = (int32_t)(kc[i] << 1) >> 24;
                const uint32_t sb = (kc[i] - ((uint32_t)e << 23)) & 0x80000000u;
                return __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, ldexpf(in, e)) ^ sb);
            } else {
                return __builtin_bit_cast(float, __builtin_bit_cast(uint32_t, in) + kc[i]);
            }
        } else {
            return ((in >> sh[i]) ^ neg[i]) - neg[i];
        }
    }
};

constexpr int kTlRow = 65;                             // words per time row of a transposed tile
constexpr int kTlMaxChunks = 16 * kTlColsMaxT / 64;     // 4-element chunks per lane and group

// Column of the e-th element of a group of columns of length T (e < 64 T)
__device__ __forceinline__ int tl_col_of(int e, int T, uint32_t tdiv)
{
    return T == 1 ? e : (int)__umulhi((uint32_t)e, tdiv);
}

// Stages a group's ncols * T contiguous elements of src (from element gbase)
// into the transposed tile tile[tau * kTlRow + col], with 4-element vector
// loads for a whole group when vec is set.  Returns (wave-uniform) whether
// some staged float lies outside [lo, hi); always false for Q8.8.
template <int DT>
__device__ __forceinline__ bool tl_stage(const void* src, int64_t gbase, int ncols, int T, uint32_t tdiv, bool vec,
                                         typename TlIO<DT>::V* tile, float lo, float hi)
{
    using V = typename TlIO<DT>::V;
    constexpr bool kF = DT != MFPSN_Q8_8;
    const int lane = (int)threadIdx.x & 63;
    bool out = false;
    auto put = [&](int e, V v) {
        const int c = tl_col_of(e, T, tdiv);
        tile[(e - c * T) * kTlRow + c] = v;
        if constexpr (kF) {
            const float m = __builtin_fabsf(v);
            out = out || !(m >= lo && m < hi);
        }
    };
    if (ncols == 64 && vec) {
        const int nch = 16 * T;  // 4-element chunks of the group
        V v[kTlMaxChunks][4];
#pragma unroll
        for (int j = 0; j < kTlMaxChunks; ++j)
            if (lane + 64 * j < nch)
                TlVec4<DT>::ld(src, gbase + 4 * (lane + 64 * j), v[j]);
#pragma unroll
        for (int j = 0; j < kTlMaxChunks; ++j)
            if (lane + 64 * j < nch) {
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    put(4 * (lane + 64 * j) + q, v[j][q]);
            }
    } else {
        for (int e = lane; e < ncols * T; e += 64)
            put(e, TlIO<DT>::ld(src, gbase + e));
    }
    return kF && __builtin_amdgcn_ballot_w64(out) != 0;
}

// Short columns (T <= kTlColsMaxT): one wave per group of 64 columns,
// lane = column.  The group's inputs, 64 T contiguous elements, are read with
// coalesced loads and written transposed into LDS, one row of 64 columns per
// time step (row stride 65 words: a row read by the 64 lanes touches every
// bank once).  Each lane then walks its column in time with the taps of its
// own channel in registers, reading the k inputs of an output from its LDS
// column, and puts its spikes into a [column][time] byte tile that is
// written back with 16-byte stores.
template <int DT, int K>
__global__ __launch_bounds__(64) void tl_cols_kernel(TlArgs a)
{
    using V = typename TlIO<DT>::V;
    constexpr bool kF = DT != MFPSN_Q8_8;
    constexpr int kRow = kTlRow;
    extern __shared__ uint32_t tl_lds[];
    const int lane = (int)threadIdx.x;
    const int T = a.T;
    const int64_t col0 = (int64_t)blockIdx.x * 64;
    const int ncols = a.M - col0 < 64 ? (int)(a.M - col0) : 64;
    const int64_t gbase = col0 * T;
    V* xt = reinterpret_cast<V*>(tl_lds);
    uint8_t* st = reinterpret_cast<uint8_t*>(tl_lds) + ((T * kRow * 4 + 15) & ~15);
    const bool slow = tl_stage<DT>(a.x, gbase, ncols, T, a.tdiv, a.vec_x, xt, a.fast_lo, a.fast_hi);

    const int64_t col = col0 + (lane < ncols ? lane : 0);
    const int c = (int)((col / a.S) % a.C);
    TlLaneTaps<DT, K> taps;
    taps.load(a.sign, a.shift, c, a.shift_lo, a.shift_hi);
    V bias;
    if constexpr (kF)
        bias = ((const float*)a.bias)[c];
    else
        bias = ((const int32_t*)a.bias)[c];
    wave_lds_sync();

    auto tap = [&](V in, int i, auto exact) -> V { return taps.template apply<decltype(exact)::value>(in, i); };
    const int span = (K - 1) * a.d;
    const bool pack = (T & 3) == 0;
    // NO outputs per pass, so that their NO * K LDS reads are in flight together
    constexpr int NO = K <= 16 ? 4 : 2;
    auto walk = [&](auto exact) {
        for (int t0 = 0; t0 < T; t0 += NO) {
            V acc[NO];
#pragma unroll
            for (int j = 0; j < NO; ++j)
                acc[j] = V(0);
            if (t0 >= span) {
                // every tap input exists; outputs past the column's end read
                // its last step (in the tile) and are not stored
#pragma unroll
                for (int j = 0; j < NO; ++j) {
                    const int t = t0 + j < T ? t0 + j : T - 1;
                    V in[K];
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        in[i] = xt[(t - (K - 1 - i) * a.d) * kRow + lane];
                    acc[j] = taps.start();
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        acc[j] = taps.template accumulate<decltype(exact)::value>(acc[j], in[i], i);
                }
            } else {
                // from the first tap whose input exists (time >= 0): the
                // others read time 0 and are not added
#pragma unroll
                for (int j = 0; j < NO; ++j) {
                    const int t = t0 + j < T ? t0 + j : T - 1;
                    V in[K];
#pragma unroll
                    for (int i = 0; i < K; ++i) {
                        const int tau = t - (K - 1 - i) * a.d;
                        in[i] = xt[(tau > 0 ? tau : 0) * kRow + lane];
                    }
#pragma unroll
                    for (int i = 0; i < K; ++i) {
                        const V sum = acc[j] + tap(in[i], i, exact);
                        acc[j] = t - (K - 1 - i) * a.d >= 0 ? sum : acc[j];
                    }
                }
            }
            uint32_t s4 = 0;
#pragma unroll
            for (int j = 0; j < NO; ++j) {
                const int t = t0 + j;
                const V h = acc[j] + bias;
                bool fire;
                if constexpr (kF)
                    fire = h >= a.v_th;
                else
                    fire = h >= a.v_th_q;
                s4 |= (fire ? 1u : 0u) << (8 * j);
                if (t < T) {
                    if (!pack)
                        st[lane * T + t] = fire ? 1 : 0;
                    if (a.h_out != nullptr && lane < ncols)
                        reinterpret_cast<V*>(a.h_out)[gbase + (int64_t)lane * T + t] = h;
                }
            }
            if (pack) {  // T and t0 multiples of 4
                if constexpr (NO == 4) {
                    *reinterpret_cast<uint32_t*>(st + lane * T + t0) = s4;
                } else {
                    *reinterpret_cast<uint16_t*>(st + lane * T + t0) = (uint16_t)s4;
                }
            }
        }
    };
    if (slow)
        walk(std::true_type{});
    else
        walk(std::false_type{});
    wave_lds_sync();

    if (ncols == 64 && a.vec_s) {
        for (int q = lane; q < 4 * T; q += 64)
            __builtin_nontemporal_store(reinterpret_cast<const U32x4*>(st)[q],
                                        reinterpret_cast<U32x4*>(a.spikes + gbase) + q);
    } else {
        for (int e = lane; e < ncols * T; e += 64)
            a.spikes[gbase + e] = st[e];
    }
}

// 64-bit values across lanes (two 32-bit shuffles)
__device__ __forceinline__ double tl_shfl_up(double v, int off)
{
    return __shfl_up(v, (unsigned)off, 64);
}
__device__ __forceinline__ int64_t tl_shfl_up(int64_t v, int off)
{
    const int lo = __shfl_up((int)(uint32_t)v, (unsigned)off, 64);
    const int hi = __shfl_up((int)(uint32_t)((uint64_t)v >> 32), (unsigned)off, 64);
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// bfloat16 bits of a float, round to nearest even (NaN stays NaN)
__device__ __forceinline__ uint16_t tl_bf16_rne(float v)
{
    const uint32_t b = __builtin_bit_cast(uint32_t, v);
    if ((b & 0x7fffffffu) > 0x7f800000u)
        return (uint16_t)((b >> 16) | 0x40u);
    return (uint16_t)((b + 0x7fffu + ((b >> 16) & 1u)) >> 16);
}

// Backward (App. A.3: Eqs. backward_X, backward_W, backward_b, generalized
// to dilation d) for short columns in the time-last layout, lane = column
// as in tl_cols_kernel.  The group's x and grad_spikes are staged transposed
// in LDS.  A forward walk recomputes H (the definition's sum), takes
// dH = grad_spikes * sigma'(H - V_th), writes dH over grad_spikes in the
// tile and adds the exact products x[t - (k-1-i) d] dH[t] and dH[t] of the
// lane's column to its grad_w / grad_b sums (double, or int64 for Q8.8).  A
// second walk forms grad_x[t] = sum over taps i ascending, with
// t + (k-1-i) d < T, of sign_i dH[t + (k-1-i) d] 2^-s_i into the x tile,
// which is stored with coalesced writes.  The 64 lanes' sums are reduced per
// (n, c) row (lanes of one row are consecutive) and stored to the row's slot
// of this block, part[block + n C + c][k+1].
template <int DT, int K>
__global__ __launch_bounds__(64) void tl_cols_bwd_kernel(TlBwdArgs a)
{
    using V = typename TlIO<DT>::V;
    constexpr bool kF = DT != MFPSN_Q8_8;
    using W = std::conditional_t<kF, double, int64_t>;
    constexpr int kRow = kTlRow;
    extern __shared__ uint32_t tl_lds[];
    const int lane = (int)threadIdx.x;
    const int T = a.T;
    const int64_t col0 = (int64_t)blockIdx.x * 64;
    const int ncols = a.M - col0 < 64 ? (int)(a.M - col0) : 64;
    const int64_t gbase = col0 * T;
    V* xt = reinterpret_cast<V*>(tl_lds);  // x, then grad_x; row T zeros
    V* gt = xt + (T + 1) * kRow;           // grad_spikes, then dH; row T zeros
    const bool slow_x = tl_stage<DT>(a.x, gbase, ncols, T, a.tdiv, a.vec_x, xt, a.fast_lo, a.fast_hi);
    (void)tl_stage<DT>(a.g, gbase, ncols, T, a.tdiv, a.vec_x, gt, 0.0f, 0.0f);

    const int64_t col = col0 + (lane < ncols ? lane : 0);
    const int c = (int)((col / a.S) % a.C);
    TlLaneTaps<DT, K> taps;
    taps.load(a.sign, a.shift, c, a.shift_lo, a.shift_hi);
    V bias;
    if constexpr (kF)
        bias = ((const float*)a.bias)[c];
    else
        bias = ((const int32_t*)a.bias)[c];
    Surrogate sg;
    sg.init(a.sg, a.alpha);
    wave_lds_sync();

    // Taps whose input lies outside the sequence read row T of a tile, which
    // holds zeros: their grad_w products are zeros, and with the ldexp taps
    // their terms are zeros too, which leave a sum that starts at +0 as it
    // is; the exponent-add taps of such inputs are not zeros and are
    // selected away.
    xt[T * kRow + lane] = V(0);
    gt[T * kRow + lane] = V(0);
    const int span = (K - 1) * a.d;

    // walk 1: H, dH (over grad_spikes in the tile), grad_w and grad_b sums.
    // Steps go in pairs whose LDS reads all issue before either step's
    // write, so that two independent chains are in flight; steps whose taps
    // reach before time 0 (t < span) run apart, with the selects they need.
    W gw[K], gb = W(0);
#pragma unroll
    for (int i = 0; i < K; ++i)
        gw[i] = W(0);
    bool out_dh = false;
    auto walk1 = [&](auto exact) {
        constexpr bool EX = decltype(exact)::value;
        auto steps = [&](int t, auto npair, auto edge_c) {
            constexpr int NP = decltype(npair)::value;
            constexpr bool NEAR = decltype(edge_c)::value;  // some tap before time 0
            constexpr bool EDGE = NEAR && !EX;              // ... whose term must be selected away
            V in[NP][K], gv[NP], dh[NP];
#pragma unroll
            for (int p = 0; p < NP; ++p) {
#pragma unroll
                for (int i = 0; i < K; ++i) {
                    const int tau = t + p - (K - 1 - i) * a.d;
                    in[p][i] = xt[(NEAR && tau < 0 ? T : tau) * kRow + lane];
                }
                gv[p] = gt[(t + p) * kRow + lane];
            }
#pragma unroll
            for (int p = 0; p < NP; ++p) {
                V acc;
                if constexpr (EDGE) {
                    acc = V(0);
#pragma unroll
                    for (int i = 0; i < K; ++i) {
                        const V sum = acc + taps.template apply<EX>(in[p][i], i);
                        acc = t + p - (K - 1 - i) * a.d >= 0 ? sum : acc;
                    }
                } else {
                    // every term counts (the zero rows' terms are zeros)
                    acc = taps.start();
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        acc = taps.template accumulate<EX>(acc, in[p][i], i);
                }
                const V h = acc + bias;
                dh[p] = delta_h(gv[p], sg_factor(sg, h, a.v_th, a.v_th_q));
            }
#pragma unroll
            for (int p = 0; p < NP; ++p) {
                gt[(t + p) * kRow + lane] = dh[p];
                gb += (W)dh[p];
#pragma unroll
                for (int i = 0; i < K; ++i) {
                    if constexpr (kF)
                        gw[i] = __builtin_fma((double)in[p][i], (double)dh[p], gw[i]);  // exact product, one rounding
                    else
                        gw[i] += (int64_t)in[p][i] * (int64_t)dh[p];
                }
                if constexpr (kF) {
                    const float m = __builtin_fabsf(dh[p]);
                    out_dh = out_dh || !(m >= a.fast_lo && m < a.fast_hi);
                }
            }
        };
        const int te = span < T ? span : T;
        int t = 0;
        for (; t + 1 < te; t += 2)
            steps(t, std::integral_constant<int, 2>{}, std::true_type{});
        if (t < te)
            steps(t++, std::integral_constant<int, 1>{}, std::true_type{});
        for (; t + 1 < T; t += 2)
            steps(t, std::integral_constant<int, 2>{}, std::false_type{});
        if (t < T)
            steps(t, std::integral_constant<int, 1>{}, std::false_type{});
    };
    if (slow_x)
        walk1(std::true_type{});
    else
        walk1(std::false_type{});
    const bool slow_dh = kF && __builtin_amdgcn_ballot_w64(out_dh) != 0;
    wave_lds_sync();

    // walk 2: grad_x into the x tile, in pairs as walk 1; steps whose taps
    // reach past T-1 (t >= T - span) run apart with their selects
    auto walk2 = [&](auto exact) {
        constexpr bool EX = decltype(exact)::value;
        auto steps = [&](int t, auto npair, auto edge_c) {
            constexpr int NP = decltype(npair)::value;
            constexpr bool NEAR = decltype(edge_c)::value;  // some tap past T-1
            constexpr bool EDGE = NEAR && !EX;
            V in[NP][K];
#pragma unroll
            for (int p = 0; p < NP; ++p) {
#pragma unroll
                for (int i = 0; i < K; ++i) {
                    const int tau = t + p + (K - 1 - i) * a.d;
                    in[p][i] = gt[(NEAR && tau >= T ? T : tau) * kRow + lane];
                }
            }
            V acc[NP];
#pragma unroll
            for (int p = 0; p < NP; ++p) {
                if constexpr (EDGE) {
                    acc[p] = V(0);
#pragma unroll
                    for (int i = 0; i < K; ++i) {
                        const V sum = acc[p] + taps.template apply<EX>(in[p][i], i);
                        acc[p] = t + p + (K - 1 - i) * a.d < T ? sum : acc[p];
                    }
                } else {
                    acc[p] = taps.start();
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        acc[p] = taps.template accumulate<EX>(acc[p], in[p][i], i);
                }
            }
#pragma unroll
            for (int p = 0; p < NP; ++p)
                xt[(t + p) * kRow + lane] = acc[p];
        };
        const int tb = T - span > 0 ? T - span : 0;  // first step with a tap past T-1
        int t = 0;
        for (; t + 1 < tb; t += 2)
            steps(t, std::integral_constant<int, 2>{}, std::false_type{});
        if (t < tb)
            steps(t++, std::integral_constant<int, 1>{}, std::false_type{});
        for (; t + 1 < T; t += 2)
            steps(t, std::integral_constant<int, 2>{}, std::true_type{});
        if (t < T)
            steps(t, std::integral_constant<int, 1>{}, std::true_type{});
    };
    if (slow_dh)
        walk2(std::true_type{});
    else
        walk2(std::false_type{});
    wave_lds_sync();

    for (int e = lane; e < ncols * T; e += 64) {
        const int cc = tl_col_of(e, T, a.tdiv);
        const V v = xt[(e - cc * T) * kRow + cc];
        if constexpr (DT == MFPSN_BF16)
            reinterpret_cast<uint16_t*>(a.grad_x)[gbase + e] = tl_bf16_rne(v);
        else
            reinterpret_cast<V*>(a.grad_x)[gbase + e] = v;
    }

    // per-channel sums: segments of consecutive lanes with one channel
    // (lanes past the last column form their own and add nothing)
    const int cl = lane < ncols ? c : -1;
    const int cprev = __shfl_up(cl, 1u, 64);
    const uint64_t heads = __builtin_amdgcn_ballot_w64(lane == 0 || cprev != cl);
    const int seg = __popcll(heads & (lane == 63 ? ~0ull : ((2ull << lane) - 1))) - 1;
    const int seg_next = __shfl_down(seg, 1u, 64);
    const bool last = cl >= 0 && (lane == 63 || seg_next != seg);
    // same[j]: the lane 2^j below is in this lane's segment.  The shuffle
    // runs on every lane: a lane that sat out of it would hand 0 to the
    // lane reading it.
    bool same[6];
#pragma unroll
    for (int j = 0; j < 6; ++j) {
        const int below = __shfl_up(seg, (unsigned)(1 << j), 64);
        same[j] = (lane >= (1 << j)) & (below == seg);
    }
    auto seg_sum = [&](W v) {
#pragma unroll
        for (int j = 0; j < 6; ++j) {
            const W u = tl_shfl_up(v, 1 << j);
            v = same[j] ? v + u : v;
        }
        return v;
    };
    W* slot = reinterpret_cast<W*>(a.part) + ((int64_t)blockIdx.x + col / a.S) * (K + 1);
#pragma unroll
    for (int i = 0; i < K; ++i) {
        const W v = seg_sum(gw[i]);
        if (last)
            slot[i] = v;
    }
    const W v = seg_sum(gb);
    if (last)
        slot[K] = v;
}

// dst[j] = src[cbase + t_first + j] for j in [0, n), 0 where the time
// t_first + j lies outside [0, T); the loads go in batches of eight per lane,
// all issued before their LDS writes.  With CHECK, returns (wave-uniform)
// whether some staged float lies outside [lo, hi).
template <int DT, bool CHECK>
__device__ __forceinline__ bool tl_stage_window(const void* src, int64_t cbase, int t_first, int n, int T,
                                                typename TlIO<DT>::V* dst, float lo, float hi)
{
    using V = typename TlIO<DT>::V;
    constexpr int B = 8;
    const int lane = (int)threadIdx.x & 63;
    bool out = false;
    for (int base = 0; base < n; base += 64 * B) {
        V v[B];
#pragma unroll
        for (int q = 0; q < B; ++q) {
            const int j = base + lane + 64 * q;
            const int t = t_first + j;
            v[q] = j < n && t >= 0 && t < T ? TlIO<DT>::ld(src, cbase + t) : V(0);
        }
#pragma unroll
        for (int q = 0; q < B; ++q) {
            const int j = base + lane + 64 * q;
            if (j < n) {
                dst[j] = v[q];
                if constexpr (CHECK && DT != MFPSN_Q8_8) {
                    const int t = t_first + j;
                    const float m = __builtin_fabsf(v[q]);
                    out = out || (t >= 0 && t < T && !(m >= lo && m < hi));
                }
            }
        }
    }
    return CHECK && DT != MFPSN_Q8_8 && __builtin_amdgcn_ballot_w64(out) != 0;
}

// Sum over the 64 lanes, every lane gets it
template <typename W> __device__ __forceinline__ W tl_wave_sum(W v)
{
#pragma unroll
    for (int j = 1; j < 64; j <<= 1) {
        if constexpr (std::is_same_v<W, double>) {
            v += __shfl_xor(v, j, 64);
        } else {
            const int lo = __shfl_xor((int)(uint32_t)v, j, 64);
            const int hi = __shfl_xor((int)(uint32_t)((uint64_t)v >> 32), j, 64);
            v += (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
        }
    }
    return v;
}

// Backward for long columns (T > kTlColsMaxT) in the time-last layout:
// persistent waves over segments of L = a.seg time steps of one column, lane
// = time step, so the taps are the same on every lane.  With P = (k-1) d,
// a segment [t0, t0 + L) stages x over [t0 - P, t0 + L + P) and grad_spikes
// over [t0, t0 + L + P) in the wave's LDS windows (zeros outside [0, T)),
// recomputes H and dH over [t0, t0 + L + P) (the dH its grad_x needs), adds
// the exact products and dH of its own steps to grad_w / grad_b sums, forms
// grad_x over its own steps from the dH window.  A wave takes a contiguous
// run of a.chunk segments in channel-major order and stores its sums to
// its slot of the channel, part[wave + c][k+1], when the channel changes
// and at the end.  The dH of the P steps after a segment is recomputed by
// the next one.
template <int DT, int K>
__global__ __launch_bounds__(kTlWaves * 64) void tl_seg_bwd_kernel(TlBwdArgs a)
{
    using V = typename TlIO<DT>::V;
    constexpr bool kF = DT != MFPSN_Q8_8;
    using W = std::conditional_t<kF, double, int64_t>;
    extern __shared__ uint32_t tl_lds[];
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6), lane = (int)threadIdx.x & 63;
    const int T = a.T, d = a.d, span = (K - 1) * d, L = a.seg;
    const int xw = L + 2 * span, dw = L + span;
    V* xs = reinterpret_cast<V*>(tl_lds) + (size_t)wave * (xw + dw);
    V* ds = xs + xw;
    // units in channel-major order (c, n, s, segment); wave w takes the
    // contiguous run [w chunk, (w+1) chunk), so its sums stay in registers
    // while the channel stays the same
    const int64_t units = a.M * a.nseg, per_c = units / a.C;
    const int64_t chunk = a.chunk;
    const int64_t wg = (int64_t)blockIdx.x * kTlWaves + wave;
    const int64_t v0 = wg * chunk;
    const int64_t v1 = v0 + chunk < units ? v0 + chunk : units;
    Surrogate sg;
    sg.init(a.sg, a.alpha);
    W* part = reinterpret_cast<W*>(a.part);
    W gw[K], gb = W(0);
#pragma unroll
    for (int i = 0; i < K; ++i)
        gw[i] = W(0);
    TlLaneTaps<DT, K> taps;
    V bias = V(0);
    int cur = -1;  // channel of the sums (wave-uniform)
    auto flush = [&]() {
        if (cur < 0)
            return;
        W* slot = part + (wg + cur) * (K + 1);
#pragma unroll
        for (int i = 0; i < K; ++i) {
            const W v = tl_wave_sum(gw[i]);
            gw[i] = W(0);
            if (lane == 0)
                slot[i] = v;
        }
        const W v = tl_wave_sum(gb);
        gb = W(0);
        if (lane == 0)
            slot[K] = v;
    };
    for (int64_t u = v0; u < v1; ++u) {
        const int c = (int)(u / per_c);
        const int64_t r = u - (int64_t)c * per_c;
        const int64_t ns = r / a.nseg;  // n S + s
        const int t0 = (int)(r - ns * a.nseg) * L;
        const int64_t n = ns / a.S;
        const int64_t col = (n * a.C + c) * a.S + (ns - n * a.S);
        const int64_t cbase = col * (int64_t)T;
        if (c != cur) {
            flush();
            cur = c;
            taps.load(a.sign, a.shift, c, a.shift_lo, a.shift_hi);
            if constexpr (kF)
                bias = ((const float*)a.bias)[c];
            else
                bias = ((const int32_t*)a.bias)[c];
        }
        const bool slow_x = tl_stage_window<DT, true>(a.x, cbase, t0 - span, xw, T, xs, a.fast_lo, a.fast_hi);
        (void)tl_stage_window<DT, false>(a.g, cbase, t0, dw, T, ds, 0.0f, 0.0f);
        wave_lds_sync();

        // H and dH over [t0, t0 + L + P); x of time t - (k-1-i) d is xs[j + i d]
        bool out_dh = false;
        const bool head = t0 < span;  // some tap input before time 0 (zeros in the window)
        auto walk1 = [&](auto exact) {
            constexpr bool EX = decltype(exact)::value;
            for (int j = lane; j < dw; j += 64) {
                const int t = t0 + j;
                if (t >= T)
                    break;
                V acc = V(0);
                if (!EX && head) {
#pragma unroll
                    for (int i = 0; i < K; ++i) {
                        const V sum = acc + taps.template apply<EX>(xs[j + i * d], i);
                        acc = t - (K - 1 - i) * d >= 0 ? sum : acc;
                    }
                } else {
                    acc = taps.start();
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        acc = taps.template accumulate<EX>(acc, xs[j + i * d], i);
                }
                const V h = acc + bias;
                const V dh = delta_h(ds[j], sg_factor(sg, h, a.v_th, a.v_th_q));
                ds[j] = dh;
                if constexpr (kF) {
                    const float m = __builtin_fabsf(dh);
                    out_dh = out_dh || !(m >= a.fast_lo && m < a.fast_hi);
                }
                if (j < L) {  // this segment's own step
                    gb += (W)dh;
#pragma unroll
                    for (int i = 0; i < K; ++i) {
                        if constexpr (kF)
                            gw[i] = __builtin_fma((double)xs[j + i * d], (double)dh, gw[i]);
                        else
                            gw[i] += (int64_t)xs[j + i * d] * (int64_t)dh;
                    }
                }
            }
        };
        if (slow_x)
            walk1(std::true_type{});
        else
            walk1(std::false_type{});
        const bool slow_dh = kF && __builtin_amdgcn_ballot_w64(out_dh) != 0;
        wave_lds_sync();

        // grad_x over [t0, t0 + L): dH of time t + (k-1-i) d is ds[j + (k-1-i) d]
        const bool tail = t0 + L + span > T;  // some tap input past the end (zeros)
        auto walk2 = [&](auto exact) {
            constexpr bool EX = decltype(exact)::value;
            for (int j = lane; j < L; j += 64) {
                const int t = t0 + j;
                if (t >= T)
                    break;
                V acc = V(0);
                if (!EX && tail) {
#pragma unroll
                    for (int i = 0; i < K; ++i) {
                        const V sum = acc + taps.template apply<EX>(ds[j + (K - 1 - i) * d], i);
                        acc = t + (K - 1 - i) * d < T ? sum : acc;
                    }
                } else {
                    acc = taps.start();
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        acc = taps.template accumulate<EX>(acc, ds[j + (K - 1 - i) * d], i);
                }
                if constexpr (DT == MFPSN_BF16)
                    reinterpret_cast<uint16_t*>(a.grad_x)[cbase + t] = tl_bf16_rne(acc);
                else
                    reinterpret_cast<V*>(a.grad_x)[cbase + t] = acc;
            }
        };
        if (slow_dh)
            walk2(std::true_type{});
        else
            walk2(std::false_type{});
        wave_lds_sync();  // every read of the windows before the next segment's writes
    }
    flush();
}

__global__ void tl_zero_kernel(uint64_t* p, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0;
}

// acc[i][c] = the sum of channel c's slots of sum i, in a fixed order.  The
// channel's groups are g = n C + c, n < ng, each of z consecutive units of
// a sequence cut into pieces of b units (blocks or waves); group g meets
// the pieces first = g z / b .. last = (g z + z - 1) / b, whose slots are
// piece + g.  One wave per (c, i): lane l adds the (n, piece) pairs
// l + 64 j in four interleaved sums, which are added pairwise, then across
// the lanes in a fixed tree.
template <typename W>
__global__ __launch_bounds__(64) void tl_bwd_reduce_kernel(const W* part, W* acc, int32_t C, int32_t k1, int64_t ng,
                                                           int64_t z, int64_t b)
{
    const int c = blockIdx.x, i = blockIdx.y, lane = threadIdx.x;
    const int64_t span = (z + b - 1) / b + 1;  // pieces one group can meet, at most
    const int64_t total = ng * span;
    auto term = [&](int64_t q) -> W {
        if (q >= total)
            return W(0);
        const int64_t n = q / span, j = q - n * span;
        const int64_t g = n * C + c;
        const int64_t first = g * z / b, last = (g * z + z - 1) / b;
        return first + j <= last ? part[(first + j + g) * k1 + i] : W(0);
    };
    W s[4] = {W(0), W(0), W(0), W(0)};
    for (int64_t q = lane; q < total; q += 256) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
            s[u] += term(q + 64 * u);
    }
    const W v = tl_wave_sum((s[0] + s[1]) + (s[2] + s[3]));
    if (lane == 0)
        acc[(int64_t)i * C + c] = v;
}

// Forward for long columns (T > kTlColsMaxT) with histories P = (k-1) d of
// at most kTlBwdMaxSpan steps: persistent waves over segments [t0, t0 + L)
// of one column (L = a.seg), lane = time step, in channel-major runs as in
// tl_seg_bwd_kernel (the taps are loaded again only when the channel
// changes).  A segment stages x over [t0 - P, t0 + L) in the wave's LDS
// window (zeros before time 0), so the input of tap i for step t0 + j is
// xs[j + i d]; only the first segment of a column, whose taps reach before
// time 0, selects the exponent-add terms of those zeros away.
template <int DT, int K>
__global__ __launch_bounds__(kTlWaves * 64) void tl_seg_fwd_kernel(TlArgs a)
{
    using V = typename TlIO<DT>::V;
    constexpr bool kF = DT != MFPSN_Q8_8;
    extern __shared__ uint32_t tl_lds[];
    const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6), lane = (int)threadIdx.x & 63;
    const int T = a.T, d = a.d, span = (K - 1) * d, L = a.seg;
    const int xw = L + span;
    V* xs = reinterpret_cast<V*>(tl_lds) + (size_t)wave * xw;
    const int64_t units = a.M * a.nseg, per_c = units / a.C;
    const int64_t nwaves = (int64_t)gridDim.x * kTlWaves;
    const int64_t chunk = (units + nwaves - 1) / nwaves;
    const int64_t v0 = ((int64_t)blockIdx.x * kTlWaves + wave) * chunk;
    const int64_t v1 = v0 + chunk < units ? v0 + chunk : units;
    TlLaneTaps<DT, K> taps;
    V bias = V(0);
    int cur = -1;
    for (int64_t u = v0; u < v1; ++u) {
        const int c = (int)(u / per_c);
        const int64_t r = u - (int64_t)c * per_c;
        const int64_t ns = r / a.nseg;  // n S + s
        const int t0 = (int)(r - ns * a.nseg) * L;
        const int64_t n = ns / a.S;
        const int64_t cbase = ((n * a.C + c) * a.S + (ns - n * a.S)) * (int64_t)T;
        if (c != cur) {
            cur = c;
            taps.load(a.sign, a.shift, c, a.shift_lo, a.shift_hi);
            if constexpr (kF)
                bias = ((const float*)a.bias)[c];
            else
                bias = ((const int32_t*)a.bias)[c];
        }
        const bool slow = tl_stage_window<DT, true>(a.x, cbase, t0 - span, xw, T, xs, a.fast_lo, a.fast_hi);
        wave_lds_sync();
        const bool head = t0 < span;
        auto walk = [&](auto exact) {
            constexpr bool EX = decltype(exact)::value;
            for (int j = lane; j < L; j += 64) {
                const int t = t0 + j;
                if (t >= T)
                    break;
                V acc = V(0);
                if (!EX && head) {
#pragma unroll
                    for (int i = 0; i < K; ++i) {
                        const V sum = acc + taps.template apply<EX>(xs[j + i * d], i);
                        acc = t - (K - 1 - i) * d >= 0 ? sum : acc;
                    }
                } else {
                    acc = taps.start();
#pragma unroll
                    for (int i = 0; i < K; ++i)
                        acc = taps.template accumulate<EX>(acc, xs[j + i * d], i);
                }
                const V h = acc + bias;
                bool fire;
                if constexpr (kF)
                    fire = h >= a.v_th;
                else
                    fire = h >= a.v_th_q;
                a.spikes[cbase + t] = fire ? 1 : 0;
                if (a.h_out != nullptr)
                    reinterpret_cast<V*>(a.h_out)[cbase + t] = h;
            }
        };
        if (slow)
            walk(std::true_type{});
        else
            walk(std::false_type{});
        wave_lds_sync();  // every read of the window before the next segment's writes
    }
}

template <int DT, int K, int NS, bool LDS>
void launch_variant(const TlArgs& a, hipStream_t st)
{
    constexpr int kW = 64 * NS;
    auto kern = tl_fwd_kernel<DT, K, NS, LDS>;
    const size_t lds = LDS ? (size_t)kTlWaves * (kW + a.halo) * 4 : 0;
    // persistent grid: every resident block slot of the device, at most one
    // segment per wave
    static int resident = 0, cus = 0;
    static size_t resident_lds = (size_t)-1;
    if (resident == 0 || resident_lds != lds) {
        int dev = 0, nb = 0;
        (void)hipGetDevice(&dev);
        (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kern, kTlWaves * 64, lds);
        resident = nb > 0 ? nb : 1;
        resident_lds = lds;
    }
    const int64_t units = a.M * a.nseg;
    int64_t blocks = (units + kTlWaves - 1) / kTlWaves;
    const int64_t cap = (int64_t)resident * (cus > 0 ? cus : 1);
    blocks = blocks < cap ? blocks : cap;
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kTlWaves * 64), lds, st, a);
}

template <int DT, int K>
void launch_k(const TlArgs& a, hipStream_t st)
{
    if (a.T <= kTlColsMaxT) {
        const size_t lds = ((size_t)a.T * 65 * 4 + 15) / 16 * 16 + (size_t)64 * a.T;
        const int64_t blocks = (a.M + 63) / 64;
        auto kern = tl_cols_kernel<DT, K>;
        hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(64), lds, st, a);
        return;
    }
    if (a.seg > 0) {  // histories of at most kTlBwdMaxSpan steps
        const size_t lds = (size_t)kTlWaves * ((size_t)a.seg + (size_t)(K - 1) * a.d) * 4;
        auto kern = tl_seg_fwd_kernel<DT, K>;
        int dev = 0, nb = 0, cus = 0;
        (void)hipGetDevice(&dev);
        (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kern, kTlWaves * 64, lds);
        const int64_t units = a.M * a.nseg;
        int64_t blocks = (units + kTlWaves - 1) / kTlWaves;
        const int64_t cap = (int64_t)(nb > 0 ? nb : 1) * (cus > 0 ? cus : 1);
        blocks = blocks < cap ? blocks : cap;
        hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kTlWaves * 64), lds, st, a);
        return;
    }
    const bool lds = a.halo > 0 || (K - 1) * a.d == 0;
    const bool short_steps = a.steps_per_lane == 1;
    if (lds)
        short_steps ? launch_variant<DT, K, 1, true>(a, st) : launch_variant<DT, K, 4, true>(a, st);
    else
        short_steps ? launch_variant<DT, K, 1, false>(a, st) : launch_variant<DT, K, 4, false>(a, st);
}
template <int DT, int... Ks>
void dispatch_k(const TlArgs& a, hipStream_t st, std::integer_sequence<int, Ks...>)
{
    (void)((a.k == Ks + 1 ? (launch_k<DT, Ks + 1>(a, st), true) : false) || ...);
}

template <int DT, int K>
int64_t launch_bwd_k(const TlBwdArgs& a, hipStream_t st)
{
    if (a.T <= kTlColsMaxT) {
        const size_t lds = (size_t)2 * (a.T + 1) * kTlRow * 4;
        const int64_t blocks = (a.M + 63) / 64;
        auto kern = tl_cols_bwd_kernel<DT, K>;
        hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(64), lds, st, a);
        return 64;
    }
    // persistent grid: every resident block slot (at most kTlSegMaxBlocks,
    // which bounds the slots), at most one segment per wave
    const int span = (K - 1) * a.d;
    const size_t lds = (size_t)kTlWaves * (2 * (size_t)a.seg + 3 * (size_t)span) * 4;
    auto kern = tl_seg_bwd_kernel<DT, K>;
    int dev = 0, nb = 0, cus = 0;
    (void)hipGetDevice(&dev);
    (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    (void)hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kern, kTlWaves * 64, lds);
    const int64_t units = a.M * a.nseg;
    int64_t blocks = (units + kTlWaves - 1) / kTlWaves;
    const int64_t cap = (int64_t)(nb > 0 ? nb : 1) * (cus > 0 ? cus : 1);
    blocks = blocks < cap ? blocks : cap;
    blocks = blocks < kTlSegMaxBlocks ? blocks : kTlSegMaxBlocks;
    TlBwdArgs b = a;
    const int64_t nwaves = blocks * kTlWaves;
    b.chunk = (units + nwaves - 1) / nwaves;
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(kTlWaves * 64), lds, st, b);
    return b.chunk;
}
template <int DT, int... Ks>
int64_t dispatch_bwd_k(const TlBwdArgs& a, hipStream_t st, std::integer_sequence<int, Ks...>)
{
    int64_t piece = 0;
    (void)((a.k == Ks + 1 ? (piece = launch_bwd_k<DT, Ks + 1>(a, st), true) : false) || ...);
    return piece;
}

}  // namespace

// Every storage type's kernels are compiled in a translation unit of their
// own (MFPSN_TL_DTYPE = 0, 1, 2); the unit without it holds the dispatch.
#if defined(MFPSN_TL_DTYPE)
using TlKs = std::make_integer_sequence<int, MFPSN_MAX_K>;
#if MFPSN_TL_DTYPE == 0
void tl_forward_f32(const TlArgs& a, hipStream_t st) { dispatch_k<MFPSN_F32>(a, st, TlKs{}); }
int64_t tl_backward_f32(const TlBwdArgs& a, hipStream_t st) { return dispatch_bwd_k<MFPSN_F32>(a, st, TlKs{}); }
#elif MFPSN_TL_DTYPE == 1
void tl_forward_bf16(const TlArgs& a, hipStream_t st) { dispatch_k<MFPSN_BF16>(a, st, TlKs{}); }
int64_t tl_backward_bf16(const TlBwdArgs& a, hipStream_t st) { return dispatch_bwd_k<MFPSN_BF16>(a, st, TlKs{}); }
#else
void tl_forward_q88(const TlArgs& a, hipStream_t st) { dispatch_k<MFPSN_Q8_8>(a, st, TlKs{}); }
int64_t tl_backward_q88(const TlBwdArgs& a, hipStream_t st) { return dispatch_bwd_k<MFPSN_Q8_8>(a, st, TlKs{}); }
#endif
#else
hipError_t launch_forward_time_last(const TlArgs& a, int dtype, hipStream_t st)
{
    if (a.M == 0 || a.T == 0)
        return hipSuccess;
    switch (dtype) {
    case MFPSN_F32: tl_forward_f32(a, st); break;
    case MFPSN_BF16: tl_forward_bf16(a, st); break;
    default: tl_forward_q88(a, st); break;
    }
    return hipGetLastError();
}

hipError_t launch_backward_time_last(const TlBwdArgs& a, int dtype, hipStream_t st)
{
    const int64_t n = (int64_t)(a.k + 1) * a.C;
    if (n == 0)
        return hipSuccess;
    if (a.M == 0 || a.T == 0) {
        const int64_t blocks = (n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024;
        hipLaunchKernelGGL(tl_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, st, (uint64_t*)a.acc, n);
        return hipGetLastError();
    }
    int64_t piece = 0;
    switch (dtype) {
    case MFPSN_F32: piece = tl_backward_f32(a, st); break;
    case MFPSN_BF16: piece = tl_backward_bf16(a, st); break;
    default: piece = tl_backward_q88(a, st); break;
    }
    // groups: the (n, c) rows of S columns, or the channels' runs of segments
    const bool cols = a.T <= kTlColsMaxT;
    const int64_t ng = cols ? a.M / ((int64_t)a.C * a.S) : 1;
    const int64_t z = cols ? (int64_t)a.S : a.M / a.C * a.nseg;
    const dim3 grid((unsigned)a.C, (unsigned)(a.k + 1));
    if (dtype == MFPSN_Q8_8)
        hipLaunchKernelGGL(tl_bwd_reduce_kernel<int64_t>, grid, dim3(64), 0, st, (const int64_t*)a.part,
                           (int64_t*)a.acc, a.C, a.k + 1, ng, z, piece);
    else
        hipLaunchKernelGGL(tl_bwd_reduce_kernel<double>, grid, dim3(64), 0, st, (const double*)a.part,
                           (double*)a.acc, a.C, a.k + 1, ng, z, piece);
    return hipGetLastError();
}
#endif

}  // namespace mfpsn
