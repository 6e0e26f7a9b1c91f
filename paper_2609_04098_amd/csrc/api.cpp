// C ABI of the NVFP4 W4A4 linear layer (include/nvfp4.h): synchronous
// argument validation, the gfx950 device check, workspace sizing and
// dispatch to the kernel launchers.  No exception or C++ type crosses the
// ABI; errors are status codes, and the HIP error of the last NVFP4_EHIP is
// kept per host thread.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <math.h>
#include <string.h>

#include <mutex>

#include "launch.h"
#include "nvfp4.h"
#include "packed_layout.h"

static_assert(NVFP4_SEG_TABLE == NVFP4_MAX_SEGMENTS + 1, "segment table size");

namespace {

thread_local int g_last_hip_error = 0;

constexpr int kMaxDevices = 64;
std::once_flag g_dev_once[kMaxDevices];
int g_dev_ok[kMaxDevices];   // 1: gfx950, 0: other

int fail_hip(hipError_t e) {
  g_last_hip_error = (int)e;
  return NVFP4_EHIP;
}

// NVFP4_OK if the current device is gfx950.
int check_device() {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail_hip(e);
  if (dev < 0 || dev >= kMaxDevices) return NVFP4_EUNSUPPORTED;
  std::call_once(g_dev_once[dev], [dev]() {
    hipDeviceProp_t prop;
    g_dev_ok[dev] = 0;
    if (hipGetDeviceProperties(&prop, dev) == hipSuccess)
      g_dev_ok[dev] = strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 0;
  });
  return g_dev_ok[dev] ? NVFP4_OK : NVFP4_EUNSUPPORTED;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int64_t kI32Lim = (int64_t)1 << 31;

// Segment table: n_seg in [1, NVFP4_MAX_SEGMENTS], offsets strictly
// increasing from 0 to N.
bool valid_segments(const int64_t* offs, int n_seg, int64_t n) {
  if (offs == nullptr || n_seg < 1 || n_seg > NVFP4_MAX_SEGMENTS) return false;
  if (offs[0] != 0 || offs[n_seg] != n) return false;
  for (int i = 0; i < n_seg; ++i)
    if (offs[i + 1] <= offs[i]) return false;
  return true;
}

}  // namespace

extern "C" {

const char* nvfp4_status_str(int status) {
  switch (status) {
    case NVFP4_OK: return "NVFP4_OK";
    case NVFP4_EINVAL: return "NVFP4_EINVAL: invalid argument";
    case NVFP4_EUNSUPPORTED: return "NVFP4_EUNSUPPORTED: device is not gfx950, or the shape is not supported";
    case NVFP4_EWORKSPACE: return "NVFP4_EWORKSPACE: workspace or buffer too small";
    case NVFP4_EHIP: return "NVFP4_EHIP: HIP runtime error";
    default: return "NVFP4: unknown status";
  }
}

int nvfp4_last_hip_error(void) { return g_last_hip_error; }

size_t nvfp4_quantize_act_workspace(int64_t M, int64_t K) {
  (void)M;
  (void)K;
  return (size_t)nvfp4::kActPartials * sizeof(float);
}

// Arguments of nvfp4_quantize_act other than the workspace.
static int check_act_args(const void* x, int64_t M, int64_t K, int64_t ldx, const uint8_t* codes,
                          const uint8_t* scales, const float* g_enc, int mode) {
  if (mode != NVFP4_DYNAMIC && mode != NVFP4_STATIC) return NVFP4_EINVAL;
  if (M < 0 || K < 0 || K % NVFP4_BLOCK != 0) return NVFP4_EINVAL;
  if (g_enc == nullptr || (reinterpret_cast<uintptr_t>(g_enc) & 3u)) return NVFP4_EINVAL;
  if (M != 0 && K != 0) {
    if (ldx < K || ldx % 8 != 0) return NVFP4_EINVAL;
    if (M * ldx >= kI32Lim || M * K >= kI32Lim) return NVFP4_EINVAL;
    if (x == nullptr || codes == nullptr || scales == nullptr) return NVFP4_EINVAL;
    if (!aligned16(x) || !aligned16(codes) || !aligned16(scales)) return NVFP4_EINVAL;
  }
  return NVFP4_OK;
}

int nvfp4_quantize_act(const void* x, int64_t M, int64_t K, int64_t ldx, uint8_t* codes,
                       uint8_t* scales, float* g_enc, int mode, void* workspace,
                       size_t workspace_bytes, void* stream) {
  int st = check_act_args(x, M, K, ldx, codes, scales, g_enc, mode);
  if (st != NVFP4_OK) return st;
  const bool empty = (M == 0 || K == 0);
  const bool dynamic = mode == NVFP4_DYNAMIC;
  if (dynamic && !empty) {
    if (workspace == nullptr || !aligned16(workspace)) return NVFP4_EINVAL;
    if (workspace_bytes < nvfp4_quantize_act_workspace(M, K)) return NVFP4_EWORKSPACE;
  }
  st = check_device();
  if (st != NVFP4_OK) return st;
  if (empty && !dynamic) return NVFP4_OK;
  hipError_t e = nvfp4::launch_act_quant(x, M, K, ldx, codes, scales, g_enc, dynamic,
                                         static_cast<float*>(workspace),
                                         static_cast<hipStream_t>(stream));
  return e == hipSuccess ? NVFP4_OK : fail_hip(e);
}

int nvfp4_quantize_act_noalloc(const void* x, int64_t M, int64_t K, int64_t ldx, uint8_t* codes,
                               uint8_t* scales, float* g_enc, int mode, void* stream) {
  int st = check_act_args(x, M, K, ldx, codes, scales, g_enc, mode);
  if (st != NVFP4_OK) return st;
  const bool empty = (M == 0 || K == 0);
  const bool dynamic = mode == NVFP4_DYNAMIC;
  if (dynamic && nvfp4_quantize_act_workspace(M, K) > nvfp4::kActScratchBytes) return NVFP4_EWORKSPACE;
  st = check_device();
  if (st != NVFP4_OK) return st;
  if (empty && !dynamic) return NVFP4_OK;
  float* ws = nullptr;
  if (dynamic && !empty) {
    hipError_t e = nvfp4::act_scratch(&ws);
    if (e != hipSuccess) return fail_hip(e);
  }
  hipError_t e = nvfp4::launch_act_quant(x, M, K, ldx, codes, scales, g_enc, dynamic, ws,
                                         static_cast<hipStream_t>(stream));
  return e == hipSuccess ? NVFP4_OK : fail_hip(e);
}

int nvfp4_rmsnorm_quantize_act(const void* x, int64_t M, int64_t K, int64_t ldx, const void* gamma,
                               float eps, uint8_t* codes, uint8_t* scales, const float* g_enc, void* y,
                               int64_t ldy, void* stream) {
  if (M < 0 || K < NVFP4_BLOCK || K % NVFP4_BLOCK != 0) return NVFP4_EINVAL;
  if (!(eps >= 0.0f) || !isfinite(eps)) return NVFP4_EINVAL;
  if (g_enc == nullptr || (reinterpret_cast<uintptr_t>(g_enc) & 3u)) return NVFP4_EINVAL;
  if (gamma == nullptr || !aligned16(gamma)) return NVFP4_EINVAL;
  if (M > 0) {
    if (ldx < K || ldx % 8 != 0 || M * ldx >= kI32Lim || M * K >= kI32Lim) return NVFP4_EINVAL;
    if (x == nullptr || codes == nullptr || scales == nullptr) return NVFP4_EINVAL;
    if (!aligned16(x) || !aligned16(codes) || !aligned16(scales)) return NVFP4_EINVAL;
    if (y != nullptr && (ldy < K || ldy % 8 != 0 || M * ldy >= kI32Lim || !aligned16(y))) return NVFP4_EINVAL;
  }
  int st = check_device();
  if (st != NVFP4_OK) return st;
  hipError_t e = nvfp4::launch_rmsnorm_quant(x, M, K, ldx, gamma, eps, g_enc, codes, scales, y, ldy,
                                             static_cast<hipStream_t>(stream));
  return e == hipSuccess ? NVFP4_OK : fail_hip(e);
}

size_t nvfp4_packed_weight_bytes(int64_t N, int64_t K) {
  if (N <= 0 || K <= 0) return 0;
  return (size_t)nvfp4::packed_dims(N, K).bytes;
}

size_t nvfp4_pack_weight_workspace_bytes(int64_t N, int64_t K, int n_seg) {
  (void)N;
  (void)K;
  if (n_seg < 1) n_seg = 1;
  if (n_seg > NVFP4_MAX_SEGMENTS) n_seg = NVFP4_MAX_SEGMENTS;
  return (size_t)n_seg * nvfp4::kWeightPartials * sizeof(float);
}

int nvfp4_pack_weight(const void* w, int64_t N, int64_t K, int64_t ldw, const int64_t* seg_offsets,
                      int n_seg, float* g_enc_seg, int mode, void* packed, size_t packed_bytes,
                      void* workspace, size_t workspace_bytes, void* stream) {
  if (mode != NVFP4_DYNAMIC && mode != NVFP4_STATIC) return NVFP4_EINVAL;
  if (N < 1 || K < NVFP4_BLOCK || K % NVFP4_BLOCK != 0) return NVFP4_EINVAL;
  if (ldw < K || ldw % 8 != 0 || N * ldw >= kI32Lim) return NVFP4_EINVAL;
  if (w == nullptr || packed == nullptr || g_enc_seg == nullptr) return NVFP4_EINVAL;
  if (!aligned16(w) || !aligned16(packed) || (reinterpret_cast<uintptr_t>(g_enc_seg) & 3u))
    return NVFP4_EINVAL;
  if (!valid_segments(seg_offsets, n_seg, N)) return NVFP4_EINVAL;
  const nvfp4::PackedDims d = nvfp4::packed_dims(N, K);
  if (d.bytes >= kI32Lim) return NVFP4_EINVAL;
  if (packed_bytes < (size_t)d.bytes) return NVFP4_EWORKSPACE;
  const bool dynamic = mode == NVFP4_DYNAMIC;
  if (dynamic) {
    if (workspace == nullptr || !aligned16(workspace)) return NVFP4_EINVAL;
    if (workspace_bytes < nvfp4_pack_weight_workspace_bytes(N, K, n_seg)) return NVFP4_EWORKSPACE;
  }
  int st = check_device();
  if (st != NVFP4_OK) return st;
  hipError_t e = nvfp4::launch_pack_weight(w, N, K, ldw, seg_offsets, n_seg, g_enc_seg, dynamic,
                                           packed, static_cast<float*>(workspace),
                                           static_cast<hipStream_t>(stream));
  return e == hipSuccess ? NVFP4_OK : fail_hip(e);
}

int nvfp4_unpack_weight(const void* packed, int64_t N, int64_t K, uint8_t* codes, uint8_t* scales,
                        void* stream) {
  if (N < 1 || K < NVFP4_BLOCK || K % NVFP4_BLOCK != 0) return NVFP4_EINVAL;
  if (nvfp4::packed_dims(N, K).bytes >= kI32Lim) return NVFP4_EINVAL;
  if (packed == nullptr || codes == nullptr || scales == nullptr) return NVFP4_EINVAL;
  if (!aligned16(packed) || !aligned16(codes) || !aligned16(scales)) return NVFP4_EINVAL;
  int st = check_device();
  if (st != NVFP4_OK) return st;
  hipError_t e = nvfp4::launch_unpack_weight(packed, N, K, codes, scales,
                                             static_cast<hipStream_t>(stream));
  return e == hipSuccess ? NVFP4_OK : fail_hip(e);
}

int nvfp4_harmonize_weight(void* packed, int64_t N, int64_t K, const int64_t* seg_offsets, int n_seg,
                           const float* g_enc_seg, float* g_shared, void* stream) {
  if (N < 1 || K < NVFP4_BLOCK || K % NVFP4_BLOCK != 0) return NVFP4_EINVAL;
  if (nvfp4::packed_dims(N, K).bytes >= kI32Lim) return NVFP4_EINVAL;
  if (!valid_segments(seg_offsets, n_seg, N)) return NVFP4_EINVAL;
  if (packed == nullptr || g_enc_seg == nullptr || g_shared == nullptr) return NVFP4_EINVAL;
  if (!aligned16(packed) || (reinterpret_cast<uintptr_t>(g_enc_seg) & 3u) ||
      (reinterpret_cast<uintptr_t>(g_shared) & 3u))
    return NVFP4_EINVAL;
  if (g_shared >= g_enc_seg && g_shared < g_enc_seg + n_seg) return NVFP4_EINVAL;
  int st = check_device();
  if (st != NVFP4_OK) return st;
  hipError_t e = nvfp4::launch_harmonize_weight(packed, N, K, seg_offsets, n_seg, g_enc_seg, g_shared,
                                                static_cast<hipStream_t>(stream));
  return e == hipSuccess ? NVFP4_OK : fail_hip(e);
}

// Argument checks shared by nvfp4_gemm and nvfp4_gemm_with_workspace.
static int check_gemm_args(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_g_enc, int64_t M,
                           int64_t K, const void* w_packed, int64_t N, const int64_t* seg_offsets, int n_seg,
                           const float* w_g_enc_seg, void* y, int64_t ldy, int y_dtype) {
  if (y_dtype != NVFP4_BF16 && y_dtype != NVFP4_F32) return NVFP4_EINVAL;
  if (M < 0 || N < 1 || K < NVFP4_BLOCK || K % NVFP4_BLOCK != 0) return NVFP4_EINVAL;
  if (ldy < N) return NVFP4_EINVAL;
  if (M * K >= kI32Lim || N * K >= kI32Lim || M * ldy >= kI32Lim) return NVFP4_EINVAL;
  if (nvfp4::packed_dims(N, K).bytes >= kI32Lim) return NVFP4_EINVAL;
  if (!valid_segments(seg_offsets, n_seg, N)) return NVFP4_EINVAL;
  if (a_g_enc == nullptr || w_g_enc_seg == nullptr || w_packed == nullptr) return NVFP4_EINVAL;
  if ((reinterpret_cast<uintptr_t>(a_g_enc) & 3u) || (reinterpret_cast<uintptr_t>(w_g_enc_seg) & 3u))
    return NVFP4_EINVAL;
  if (!aligned16(w_packed)) return NVFP4_EINVAL;
  if (M > 0) {
    if (a_codes == nullptr || a_scales == nullptr || y == nullptr) return NVFP4_EINVAL;
    if (!aligned16(a_codes) || !aligned16(a_scales)) return NVFP4_EINVAL;
    const uintptr_t elem = y_dtype == NVFP4_F32 ? 4u : 2u;
    if (reinterpret_cast<uintptr_t>(y) % elem) return NVFP4_EINVAL;
  }
  return NVFP4_OK;
}

int nvfp4_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_g_enc, int64_t M,
               int64_t K, const void* w_packed, int64_t N, const int64_t* seg_offsets, int n_seg,
               const float* w_g_enc_seg, void* y, int64_t ldy, int y_dtype, void* stream) {
  int st = check_gemm_args(a_codes, a_scales, a_g_enc, M, K, w_packed, N, seg_offsets, n_seg, w_g_enc_seg, y, ldy,
                           y_dtype);
  if (st != NVFP4_OK) return st;
  st = check_device();
  if (st != NVFP4_OK) return st;
  hipError_t e = nvfp4::launch_gemm(a_codes, a_scales, a_g_enc, M, K, w_packed, N, seg_offsets, n_seg,
                                    w_g_enc_seg, y, ldy, y_dtype == NVFP4_F32, nullptr, 0,
                                    static_cast<hipStream_t>(stream));
  return e == hipSuccess ? NVFP4_OK : fail_hip(e);
}

size_t nvfp4_gemm_workspace(int64_t M, int64_t N, int64_t K) {
  if (M < 0 || N < 1 || K < NVFP4_BLOCK || K % NVFP4_BLOCK != 0) return 0;
  if (M * K >= kI32Lim || N * K >= kI32Lim) return 0;
  if (check_device() != NVFP4_OK) return 0;
  return nvfp4::gemm_workspace_bytes(M, N, K);
}

int nvfp4_gemm_with_workspace(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_g_enc, int64_t M,
                              int64_t K, const void* w_packed, int64_t N, const int64_t* seg_offsets, int n_seg,
                              const float* w_g_enc_seg, void* y, int64_t ldy, int y_dtype, void* workspace,
                              size_t workspace_bytes, void* stream) {
  int st = check_gemm_args(a_codes, a_scales, a_g_enc, M, K, w_packed, N, seg_offsets, n_seg, w_g_enc_seg, y, ldy,
                           y_dtype);
  if (st != NVFP4_OK) return st;
  if (workspace != nullptr && !aligned16(workspace)) return NVFP4_EINVAL;
  st = check_device();
  if (st != NVFP4_OK) return st;
  const size_t need = M > 0 ? nvfp4::gemm_workspace_bytes(M, N, K) : 0;
  if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return NVFP4_EWORKSPACE;
  hipError_t e = nvfp4::launch_gemm(a_codes, a_scales, a_g_enc, M, K, w_packed, N, seg_offsets, n_seg,
                                    w_g_enc_seg, y, ldy, y_dtype == NVFP4_F32, need > 0 ? workspace : nullptr,
                                    workspace_bytes, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? NVFP4_OK : fail_hip(e);
}

const char* nvfp4_gemm_kernel(int64_t M, int64_t N, int64_t K, int part, int with_workspace) {
  if (M < 0 || N < 1 || K < NVFP4_BLOCK || K % NVFP4_BLOCK != 0 || (part != 0 && part != 1)) return nullptr;
  if (with_workspace != 0 && with_workspace != 1) return nullptr;
  if (check_device() != NVFP4_OK) return nullptr;
  return nvfp4::gemm_kernel_for(M, N, K, part, with_workspace == 1);
}

int nvfp4_gemm_gdn_gates(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_g_enc, int64_t M,
                         int64_t K, const void* w_packed, int64_t H, const float* w_g_enc_seg,
                         const float* a_log, const float* dt_bias, void* y, int64_t ldy, int y_dtype,
                         void* stream) {
  if (y_dtype != NVFP4_BF16 && y_dtype != NVFP4_F32) return NVFP4_EINVAL;
  if (M < 0 || H < 1 || K < NVFP4_BLOCK || K % NVFP4_BLOCK != 0) return NVFP4_EINVAL;
  const int64_t N = 2 * H;
  if (ldy < N) return NVFP4_EINVAL;
  if (M * K >= kI32Lim || N * K >= kI32Lim || M * ldy >= kI32Lim) return NVFP4_EINVAL;
  if (nvfp4::packed_dims(N, K).bytes >= kI32Lim) return NVFP4_EINVAL;
  if (a_g_enc == nullptr || w_g_enc_seg == nullptr || w_packed == nullptr || a_log == nullptr ||
      dt_bias == nullptr)
    return NVFP4_EINVAL;
  if ((reinterpret_cast<uintptr_t>(a_g_enc) & 3u) || (reinterpret_cast<uintptr_t>(w_g_enc_seg) & 3u) ||
      (reinterpret_cast<uintptr_t>(a_log) & 3u) || (reinterpret_cast<uintptr_t>(dt_bias) & 3u))
    return NVFP4_EINVAL;
  if (!aligned16(w_packed)) return NVFP4_EINVAL;
  if (M > 0) {
    if (a_codes == nullptr || a_scales == nullptr || y == nullptr) return NVFP4_EINVAL;
    if (!aligned16(a_codes) || !aligned16(a_scales)) return NVFP4_EINVAL;
    const uintptr_t elem = y_dtype == NVFP4_F32 ? 4u : 2u;
    if (reinterpret_cast<uintptr_t>(y) % elem) return NVFP4_EINVAL;
  }
  if (K % 64 != 0) return NVFP4_EUNSUPPORTED;
  int st = check_device();
  if (st != NVFP4_OK) return st;
  hipError_t e = nvfp4::launch_gemm_gdn_gates(a_codes, a_scales, a_g_enc, M, K, w_packed, H, w_g_enc_seg, a_log,
                                              dt_bias, y, ldy, y_dtype == NVFP4_F32,
                                              static_cast<hipStream_t>(stream));
  return e == hipSuccess ? NVFP4_OK : fail_hip(e);
}

size_t nvfp4_quantize_gemm_workspace(int64_t M, int64_t N, int64_t K) {
  if (M < 0 || N < 1 || K < 0) return 0;
  return nvfp4::quant_gemm_workspace_bytes(M, N, K);
}

int nvfp4_quantize_gemm(const void* x, int64_t M, int64_t K, int64_t ldx, float* a_g_enc, int mode,
                        void* workspace, size_t workspace_bytes, const void* w_packed, int64_t N,
                        const int64_t* seg_offsets, int n_seg, const float* w_g_enc_seg, uint8_t* a_codes,
                        uint8_t* a_scales, void* y, int64_t ldy, int y_dtype, void* stream) {
  if (mode != NVFP4_DYNAMIC && mode != NVFP4_STATIC) return NVFP4_EINVAL;
  if (y_dtype != NVFP4_BF16 && y_dtype != NVFP4_F32) return NVFP4_EINVAL;
  if (M < 0 || N < 1 || K < NVFP4_BLOCK || K % NVFP4_BLOCK != 0) return NVFP4_EINVAL;
  if (ldy < N) return NVFP4_EINVAL;
  if (M * K >= kI32Lim || N * K >= kI32Lim || M * ldy >= kI32Lim) return NVFP4_EINVAL;
  if (nvfp4::packed_dims(N, K).bytes >= kI32Lim) return NVFP4_EINVAL;
  if (!valid_segments(seg_offsets, n_seg, N)) return NVFP4_EINVAL;
  if (a_g_enc == nullptr || w_g_enc_seg == nullptr || w_packed == nullptr) return NVFP4_EINVAL;
  if ((reinterpret_cast<uintptr_t>(a_g_enc) & 3u) || (reinterpret_cast<uintptr_t>(w_g_enc_seg) & 3u))
    return NVFP4_EINVAL;
  if (!aligned16(w_packed)) return NVFP4_EINVAL;
  if ((a_codes == nullptr) != (a_scales == nullptr)) return NVFP4_EINVAL;
  const bool dynamic = mode == NVFP4_DYNAMIC;
  if (M > 0) {
    if (ldx < K || ldx % 8 != 0 || M * ldx >= kI32Lim) return NVFP4_EINVAL;
    if (x == nullptr || y == nullptr || !aligned16(x)) return NVFP4_EINVAL;
    if (a_codes != nullptr && (!aligned16(a_codes) || !aligned16(a_scales))) return NVFP4_EINVAL;
    const uintptr_t elem = y_dtype == NVFP4_F32 ? 4u : 2u;
    if (reinterpret_cast<uintptr_t>(y) % elem) return NVFP4_EINVAL;
  }
  if (dynamic || nvfp4::quant_gemm_uses_decode_path(M, N)) {
    if (workspace == nullptr || !aligned16(workspace)) return NVFP4_EINVAL;
    if (workspace_bytes < nvfp4_quantize_gemm_workspace(M, N, K)) return NVFP4_EWORKSPACE;
  }
  if ((N > 128 && M > 32) || K % 64 != 0) return NVFP4_EUNSUPPORTED;
  int st = check_device();
  if (st != NVFP4_OK) return st;
  hipError_t e = nvfp4::launch_quant_gemm(x, M, K, ldx, a_g_enc, dynamic, workspace, w_packed, N, seg_offsets,
                                          n_seg, w_g_enc_seg, a_codes, a_scales, y, ldy, y_dtype == NVFP4_F32,
                                          static_cast<hipStream_t>(stream));
  return e == hipSuccess ? NVFP4_OK : fail_hip(e);
}

}  // extern "C"
