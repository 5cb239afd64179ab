// host_sanitize_stubs.cpp -- stand-ins for the kernel launchers (defined in
// the library's .hip sources) so that the C ABI layer links into the
// sanitized host-only driver.  Host-only paths never reach them; each
// returns an error if one is called.
#include "disco_internal.h"

namespace disco {

hipError_t launch_fused(const ExecArgs&, const PackedDev&, float*) { return hipErrorNotSupported; }
hipError_t launch_sweep(const ExecArgs&, float*) { return hipErrorNotSupported; }
bool gather_z_split(const ExecArgs&) { return false; }
hipError_t launch_stencil(const ExecArgs&, const PackedDev&, float*) { return hipErrorNotSupported; }
hipError_t launch_spectral(const ExecArgs&, float*, int) { return hipErrorNotSupported; }
hipError_t launch_zero_fill(void*, size_t, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_weight_grad(const void*, const void*, void*, float*, int, int, int, int, int, int64_t, bool,
                              hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_gather_z_all(const ExecArgs&, float*, float*) { return hipErrorNotSupported; }
size_t weight_grad_ws_bytes(int, int, int, int64_t) { return 0; }
hipError_t launch_weight_grad_dw(const void*, const void*, void*, float*, int, int, int, int, int64_t, hipStream_t) {
    return hipErrorNotSupported;
}
size_t workspace_bytes_fused(const ExecArgs&, const PackedDev&) { return 0; }
size_t workspace_bytes_mfma(const ExecArgs&) { return 0; }
hipError_t launch_mfma(const ExecArgs&, void*) { return hipErrorNotSupported; }
size_t workspace_bytes_sweep(const ExecArgs&) { return 0; }
hipError_t launch_stencil_blocked(const ExecArgs&, const StencilDev&, float*) { return hipErrorNotSupported; }
size_t weight_grad_ws_bytes_dw(int, int, int, int64_t) { return 0; }
size_t workspace_bytes_spectral(const ExecArgs&) { return 0; }
hipError_t launch_contract_then_gather(const ExecArgs&, float*) { return hipErrorNotSupported; }
hipError_t launch_gather_then_contract(const ExecArgs&, float*) { return hipErrorNotSupported; }
size_t workspace_bytes_gather_z_all(const ExecArgs&) { return 0; }
size_t workspace_bytes_contract_then_gather(const ExecArgs&) { return 0; }
size_t workspace_bytes_gather_then_contract(const ExecArgs&) { return 0; }
size_t spectral_dyhat_bytes(const ExecArgs&, int) { return 0; }
size_t weight_grad_split_ws_bytes(int, int, int, int64_t, int, int64_t) { return 0; }
hipError_t launch_gather_z_light(const ExecArgs&, float*, float*, float2**) { return hipErrorNotSupported; }
hipError_t launch_spectral_dyhat(const ExecArgs&, const float*, int, float2*) { return hipErrorNotSupported; }
hipError_t launch_weight_grad_split(const float*, const float*, int, int64_t, int64_t, const float*, const float*, int,
                                    int64_t, float*, float*, int, int, int, bool, hipStream_t) {
    return hipErrorNotSupported;
}

}  // namespace disco
