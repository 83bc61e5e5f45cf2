// Stand-ins for the GPU launchers of libspice_moe, for the host-only sanitizer build of the
// library's C++ (no device code is compiled there).  Each reports that there is no device,
// so a host path that reaches a launch returns SPICE_ERR_HIP instead of running a kernel.
#include "spice_internal.h"

namespace spice {
bool expert_gemm_applies(const FfnArgs&) { return false; }
hipError_t launch_expert_gemm(const FfnArgs&, bool, bool, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_route_bucket(const RouteArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_layer_decode(const RouteArgs&, const FfnArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_expert_ffn(const FfnArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_expert_ffn_mx(const FfnArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_shared_gate(const void*, const void*, int32_t, int32_t, int32_t, float*, hipStream_t) {
    return hipErrorNoDevice;
}
hipError_t launch_expert_ffn_fetched(const FfnArgs&, const FetchArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_combine(const CombineArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_spec_update(const SpecArgs&, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_fit_setup(int32_t, int32_t*, int32_t*, int32_t*, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_fit_residual(size_t, float*, const float*, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_fit_gram(int32_t, int32_t, int, const void*, double*, hipStream_t) { return hipErrorNoDevice; }
hipError_t launch_fit_project(int32_t, int32_t, int32_t, int, const void*, const double*, float*, bool, hipStream_t) {
    return hipErrorNoDevice;
}
hipError_t launch_fill_u32(uint32_t*, size_t, uint32_t, hipStream_t) { return hipErrorNoDevice; }
}  // namespace spice
