// Host-only stand-ins for the GPU launchers of libmfpsn.so, for a sanitized
// CPU build of the C-ABI layer (mfpsn_api.cpp, mfpsn_api_ext.cpp): each one
// counts the launch it was asked for and launches nothing, so a driver can
// check that every rejected call returns before it would touch the GPU.
// Test infrastructure only.
#include "mfpsn_bn.h"
#include "mfpsn_chain.h"
#include "mfpsn_internal.h"
#include "mfpsn_qgrad.h"
#include "mfpsn_stream.h"
#include "mfpsn_tl.h"

extern "C" {
long stub_launches = 0;
}

namespace mfpsn {

hipError_t launch_forward(FwdArgs&, int, hipStream_t) { ++stub_launches; return hipSuccess; }
hipError_t launch_backward(BwdArgs&, int, hipStream_t) { ++stub_launches; return hipSuccess; }
hipError_t launch_finalize(const FinArgs&, hipStream_t) { ++stub_launches; return hipSuccess; }
hipError_t launch_quantize(const float*, int64_t, int32_t, int32_t, int8_t*, int8_t*, hipStream_t)
{
    ++stub_launches;
    return hipSuccess;
}
hipError_t launch_stream_step(const StreamArgs&, int, hipStream_t) { ++stub_launches; return hipSuccess; }
hipError_t launch_quantizer_grad(const float*, const int8_t*, int32_t, int32_t, const float*, int64_t, int32_t,
                                 float*, hipStream_t)
{
    ++stub_launches;
    return hipSuccess;
}
hipError_t launch_spikes_to_input(const uint8_t*, int64_t, int32_t, void*, hipStream_t)
{
    ++stub_launches;
    return hipSuccess;
}
hipError_t launch_forward_time_last(const TlArgs&, int, hipStream_t) { ++stub_launches; return hipSuccess; }
hipError_t launch_backward_time_last(const TlBwdArgs&, int, hipStream_t) { ++stub_launches; return hipSuccess; }
size_t bn_workspace_bytes(const BnGeom& g) { return ((size_t)2 * g.C + 64) * sizeof(double); }
hipError_t launch_bn_forward_stats(const BnGeom&, const float*, const float*, const float*, const float*, float,
                                   float*, float*, double*, double*, void*, hipStream_t)
{
    ++stub_launches;
    return hipSuccess;
}
hipError_t launch_bn_backward(const BnGeom&, const float*, const float*, const double*, float, const float*,
                              const float*, float*, float*, float*, float*, void*, hipStream_t)
{
    ++stub_launches;
    return hipSuccess;
}

}  // namespace mfpsn
