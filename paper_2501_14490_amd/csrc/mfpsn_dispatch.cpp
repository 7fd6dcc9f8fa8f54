// Dispatch of the forward / backward launchers over the order k and the
// storage type; the instantiations live in the per-range translation units
// built from mfpsn_kernels.hip.
#include <utility>

#include "mfpsn.h"
#include "mfpsn_internal.h"

namespace mfpsn {
namespace {

template <int DT, int... Ks>
hipError_t fwd_dispatch(int k, FwdArgs& a, hipStream_t st, std::integer_sequence<int, Ks...>)
{
    hipError_t e = hipErrorInvalidValue;
    (void)((k == Ks + 1 ? (e = fwd_k<Ks + 1, DT>(a, st), true) : false) || ...);
    return e;
}

template <int DT, int... Ks>
hipError_t bwd_dispatch(int k, BwdArgs& a, hipStream_t st, std::integer_sequence<int, Ks...>)
{
    hipError_t e = hipErrorInvalidValue;
    (void)((k == Ks + 1 ? (e = bwd_k<Ks + 1, DT>(a, st), true) : false) || ...);
    return e;
}

using Orders = std::make_integer_sequence<int, MFPSN_MAX_K>;

}  // namespace

hipError_t launch_forward(FwdArgs& a, int dtype, hipStream_t st)
{
    switch (dtype) {
    case kF32: return fwd_dispatch<kF32>(a.g.k, a, st, Orders{});
    case kBF16: return fwd_dispatch<kBF16>(a.g.k, a, st, Orders{});
    case kQ88: return fwd_dispatch<kQ88>(a.g.k, a, st, Orders{});
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_backward(BwdArgs& a, int dtype, hipStream_t st)
{
    switch (dtype) {
    case kF32: return bwd_dispatch<kF32>(a.g.k, a, st, Orders{});
    case kBF16: return bwd_dispatch<kBF16>(a.g.k, a, st, Orders{});
    case kQ88: return bwd_dispatch<kQ88>(a.g.k, a, st, Orders{});
    default: return hipErrorInvalidValue;
    }
}

}  // namespace mfpsn
