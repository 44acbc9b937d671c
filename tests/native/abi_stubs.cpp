// Launcher stand-ins for a host-only build of the C ABI (api.hip) under
// AddressSanitizer and UndefinedBehaviorSanitizer: every launch_* returns
// success without touching device memory, so the ABI's argument checks,
// workspace planning and pointer arithmetic run to the end on the CPU.
// The three sizing helpers return values of the same shape as the real
// ones (their values do not matter for memory safety of the host code).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "kernels.hpp"

namespace gmb {

hipError_t launch_state_init(uint32_t*, uint32_t*, int64_t, hipStream_t) { return hipSuccess; }
hipError_t launch_seed_scan(const SeedArgs&, int, const CsrArgs&, hipStream_t) { return hipSuccess; }
hipError_t launch_sample_table(const CsrArgs&, const int32_t*, const HopArgs&, uint32_t*, uint32_t*, uint32_t,
                               uint32_t, int, const DeferredArgs&, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_assign(const AssignArgs&, int, const CsrArgs&, int64_t, int, int32_t*, uint32_t*, uint32_t*,
                         hipStream_t) {
  return hipSuccess;
}
hipError_t launch_sample(const CsrArgs&, const int32_t*, const HopArgs&, uint32_t*, uint32_t, uint32_t, int,
                         const DeferredArgs&, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_route(const RouteArgs&, hipStream_t) { return hipSuccess; }
hipError_t launch_sample_route(const CsrArgs&, const SampleArgs&, const RouteArgs&, hipStream_t) { return hipSuccess; }
hipError_t launch_owner(const OwnerArgs&, hipStream_t) { return hipSuccess; }
hipError_t launch_rank(const RankArgs&, int, const CsrArgs&, int, int, int32_t*, uint32_t*, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_validate(const ValidateArgs&, int64_t, uint32_t*, hipStream_t) { return hipSuccess; }
hipError_t launch_fix(const DeferredArgs&, const int32_t*, const int32_t*, int64_t, uint32_t*, int64_t, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_gather(const int32_t*, const int32_t*, int64_t, const void*, int64_t, int64_t, void*, uint32_t*,
                         hipStream_t) {
  return hipSuccess;
}
hipError_t launch_mean_aggregate(const int32_t*, const int32_t*, const int32_t*, const void*, int, int, void*, int64_t,
                                 int, int64_t, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_sage_linear(const int32_t*, const void*, const void*, const void*, const void*, const float*, int,
                              int, int, int, int, void*, int64_t, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_xent(const float*, const int32_t*, int, int, int, float*, float*, int32_t*, int64_t, hipStream_t) {
  return hipSuccess;
}
int wgrad_ldp(int d_out) { return (d_out + 3) / 4 * 4; }
int wgrad_parts(int64_t cap_rows, int, int) { return static_cast<int>(std::min<int64_t>(8, std::max<int64_t>(1, cap_rows / 64))); }
hipError_t launch_wgrad(const int32_t*, const float*, const float*, int, const float*, int, int, int64_t, float*,
                        float*, float*, float*, const float*, int, float*, WgradArgs*, ReduceArgs*, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_dgrad(const int32_t*, const float*, int, int, const float*, const float*, int, float*, float*,
                        int64_t, const int32_t*, const int32_t*, int64_t, int32_t, int32_t*, hipStream_t) {
  return hipSuccess;
}
int64_t csc_scan_tiles(int64_t cap_src) { return std::max<int64_t>(1, (cap_src + 1023) / 1024); }
hipError_t launch_mean_backward(const int32_t*, const int32_t*, const int32_t*, int64_t, int32_t, const float*,
                                const float*, int, float*, int64_t, int64_t, int32_t*, int32_t*, int32_t*, uint32_t*,
                                int2*, int32_t*, float*, const int32_t*, int64_t, float, const WgradArgs*,
                                const ReduceArgs*, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_sgd(const SgdArgs&, float, hipStream_t) { return hipSuccess; }
hipError_t launch_widen(const WidenArgs&, hipStream_t) { return hipSuccess; }
hipError_t launch_zero(const SgdArgs&, float*, hipStream_t) { return hipSuccess; }

}  // namespace gmb
