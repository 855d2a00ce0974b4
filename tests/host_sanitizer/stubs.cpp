// Stand-ins for the kernel launchers and the two HIP runtime calls the C-ABI layer makes, so the
// ABI's validation, workspace and dispatch code builds as plain host C++ under AddressSanitizer
// and UndefinedBehaviorSanitizer.  Every launch "fails" (hipErrorNotSupported) after being
// counted, so a valid call exercises the whole host-side setup and returns MOE_ERR_HIP; no
// device pointer is ever dereferenced.
#include <hip/hip_runtime_api.h>

#include "../../paper_2607_18631_amd/csrc/kernels.hpp"

int g_launches = 0;
int g_events = 0;

extern "C" hipError_t hipEventRecord(hipEvent_t, hipStream_t) {
  ++g_events;
  return hipSuccess;
}
extern "C" const char* hipGetErrorString(hipError_t) { return "stub launch"; }

namespace moe {
static hipError_t launched() {
  ++g_launches;
  return hipErrorNotSupported;
}
hipError_t launch_grouped_gemm(const GemmProblem&, hipStream_t) { return launched(); }
hipError_t launch_gemm_bwd(const GemmBwdProblem&, hipStream_t) { return launched(); }
hipError_t launch_gate(const GateProblem&, hipStream_t) { return launched(); }
hipError_t launch_permute(const PermuteProblem&, hipStream_t, int (*)()) { return launched(); }
hipError_t launch_combine(const CombineProblem&, hipStream_t) { return launched(); }
hipError_t launch_gather(const PermuteProblem&, hipStream_t) { return launched(); }
hipError_t launch_combine_bwd(const CombineBwdProblem&, hipStream_t) { return launched(); }
hipError_t launch_gate_bwd(const GateBwdProblem&, hipStream_t) { return launched(); }
hipError_t launch_unpermute_sum(const UnpermuteSumProblem&, hipStream_t) { return launched(); }
hipError_t launch_sum_partials(const float*, int, int64_t, bf16_t*, hipStream_t) { return launched(); }
hipError_t launch_zero_f32(float*, int64_t, hipStream_t) { return launched(); }
hipError_t launch_round_bf16(const float*, bf16_t*, int64_t, hipStream_t) { return launched(); }
hipError_t permute_scratch(void** ptr) {
  *ptr = nullptr;
  return launched();
}
}  // namespace moe
