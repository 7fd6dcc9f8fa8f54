// gfx950 forward of the mul-free channel-wise neuron (arXiv 2501.14490,
// Eqs. mfdpsn_charge, mfdpsn_fire) for the time-last layout [N][C][S][T]
// (time innermost, the paper's second layout).
//
// A wave takes segments of 64 or 256 consecutive time steps of one column
// (lane l: steps t0 + l + 64 v), so its channel, and with it the k taps, are
// the same on every lane and sit in scalar registers.  The wave stages the
// inputs its taps read, x[t0 - (k-1)d .. t0 + 64 NS - 1] of its column, in
// its own LDS window with coalesced loads; every tap then reads its input
// from LDS at t - (k-1-i) d (consecutive lanes, consecutive addresses).
// Waves are persistent, and the loads of a wave's next segment are in flight
// while it computes the current one.  A history longer than the LDS slots
// reads the taps from global memory instead.
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

#include <utility>

#include "mfpsn.h"
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

// Persistent waves: wave w takes segments w, w + W, ... (W waves in the
// grid); NS time steps per lane and segment (64 NS per segment); LDS: the
// window in LDS, the first NS+2 loads of the next segment's window in
// flight while the current one computes.
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

}  // namespace

hipError_t launch_forward_time_last(const TlArgs& a, int dtype, hipStream_t st)
{
    if (a.M == 0 || a.T == 0)
        return hipSuccess;
    using Ks = std::make_integer_sequence<int, MFPSN_MAX_K>;
    switch (dtype) {
    case MFPSN_F32: dispatch_k<MFPSN_F32>(a, st, Ks{}); break;
    case MFPSN_BF16: dispatch_k<MFPSN_BF16>(a, st, Ks{}); break;
    default: dispatch_k<MFPSN_Q8_8>(a, st, Ks{}); break;
    }
    return hipGetLastError();
}

}  // namespace mfpsn
