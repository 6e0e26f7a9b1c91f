// Host-only stand-ins for the kernel launchers (csrc/launch.h), so that the
// C-ABI validation layer (csrc/api.cpp) can be built for the CPU with
// AddressSanitizer and UndefinedBehaviorSanitizer and exercised without a
// GPU.  No launcher is reached in such a run: without a device, every call
// that passes validation stops at the device check.  Each stand-in reports
// hipErrorNoDevice.
#include "launch.h"

namespace nvfp4 {

hipError_t launch_act_quant(const void*, int64_t, int64_t, int64_t, uint8_t*, uint8_t*, float*, bool, float*,
                            hipStream_t) {
  return hipErrorNoDevice;
}
hipError_t act_scratch(float**) { return hipErrorNoDevice; }
hipError_t launch_act_amax(const void*, int64_t, int64_t, int64_t, float*, int*, hipStream_t) {
  return hipErrorNoDevice;
}
hipError_t launch_rmsnorm_quant(const void*, int64_t, int64_t, int64_t, const void*, float, const float*, uint8_t*,
                                uint8_t*, void*, int64_t, hipStream_t) {
  return hipErrorNoDevice;
}
hipError_t launch_pack_weight(const void*, int64_t, int64_t, int64_t, const int64_t*, int, float*, bool, void*,
                              float*, hipStream_t) {
  return hipErrorNoDevice;
}
hipError_t launch_unpack_weight(const void*, int64_t, int64_t, uint8_t*, uint8_t*, hipStream_t) {
  return hipErrorNoDevice;
}
hipError_t launch_harmonize_weight(void*, int64_t, int64_t, const int64_t*, int, const float*, float*, hipStream_t) {
  return hipErrorNoDevice;
}
hipError_t launch_gemm(const uint8_t*, const uint8_t*, const float*, int64_t, int64_t, const void*, int64_t,
                       const int64_t*, int, const float*, void*, int64_t, bool, void*, size_t, hipStream_t) {
  return hipErrorNoDevice;
}
size_t gemm_workspace_bytes(int64_t, int64_t, int64_t) { return 0; }
const char* gemm_kernel_for(int64_t, int64_t, int64_t, int, bool) { return nullptr; }
hipError_t launch_gemm_gdn_gates(const uint8_t*, const uint8_t*, const float*, int64_t, int64_t, const void*, int64_t,
                                 const float*, const float*, const float*, void*, int64_t, bool, hipStream_t) {
  return hipErrorNoDevice;
}
bool quant_gemm_uses_decode_path(int64_t M, int64_t N) { return M >= 1 && M <= 32 && N > 128; }
size_t quant_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  return 4096 + (quant_gemm_uses_decode_path(M, N) ? (size_t)(M * K) : 0);
}
hipError_t launch_quant_gemm(const void*, int64_t, int64_t, int64_t, float*, bool, void*, const void*, int64_t,
                             const int64_t*, int, const float*, uint8_t*, uint8_t*, void*, int64_t, bool,
                             hipStream_t) {
  return hipErrorNoDevice;
}

}  // namespace nvfp4
