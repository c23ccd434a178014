// Test-only stand-ins for the kernel launchers of libspecfp8, so that the
// host side of the C ABI (api.cpp, validate.cpp, plan.cpp) links into a
// library without device code, built with AddressSanitizer and
// UndefinedBehaviorSanitizer.  Argument-validation calls return before any
// launch; a call that reached one of these would report SPEC_ERR_HIP.
#include "../../paper_2606_18502_amd/csrc/kernels.hpp"

namespace specfp8 {

hipError_t launch_quantize(const uint16_t*, int64_t, int64_t, int64_t, int, int, float*, uint8_t*, int64_t,
                           hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_silu_mul(const uint16_t*, int64_t, int64_t, int64_t, uint16_t*, int64_t, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_clip_count(const uint16_t*, int64_t, int64_t, int64_t, const float*, unsigned long long*,
                             hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_kv_cache_write(const uint16_t*, int64_t, const uint16_t*, int64_t, const int64_t*, int64_t,
                                 int64_t, int64_t, int64_t, int, float*, float*, uint8_t*, uint8_t*, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_gemm(const GemmPlan&, const uint8_t*, int64_t, const float*, int, const uint8_t*, int64_t,
                       const float*, int, int64_t, int64_t, int64_t, void*, int64_t, int, void*, hipStream_t, int,
                       float, float2*, int64_t, int64_t) {
    return hipErrorNotSupported;
}
hipError_t launch_accept(const AcceptPlan&, const uint16_t*, const uint16_t*, const int32_t*, const float*, int64_t,
                         int64_t, int64_t, float, int32_t*, int32_t*, void*, hipStream_t, const float2*, int64_t,
                         int64_t) {
    return hipErrorNotSupported;
}
hipError_t accept_scratch(void**) { return hipErrorNotSupported; }
hipError_t launch_accept_tree(const AcceptPlan&, const uint16_t*, const int32_t*, const int32_t*, const float*,
                              int64_t, int64_t, int64_t, float, int32_t*, int32_t*, int32_t*, void*, hipStream_t) {
    return hipErrorNotSupported;
}
hipError_t launch_tree_mask(const int32_t*, int64_t, int64_t, uint64_t*, int32_t*, hipStream_t) {
    return hipErrorNotSupported;
}

}  // namespace specfp8
