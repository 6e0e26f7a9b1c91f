// Host dispatch of the NVFP4 GEMM (nvfp4_gemm, nvfp4_gemm_gdn_gates): picks
// the kernel family for a shape.  The kernels and the numerics are described
// in gemm_common.h.
#include <mutex>

#include "gemm_common.h"

namespace nvfp4 {

namespace {
constexpr int kMaxDevices = 64;
std::once_flag g_cu_once[kMaxDevices];
int g_cu_count[kMaxDevices];
}  // namespace

// Compute units of the current device (cached per device, thread-safe).
static uint32_t cu_count() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 0;
  std::call_once(g_cu_once[dev], [dev]() {
    int n = 0;
    g_cu_count[dev] = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess ? n : 0;
  });
  return (uint32_t)g_cu_count[dev];
}

// The kernels one nvfp4_gemm call launches for a shape (n_cu: compute units
// of the device).
GemmPlan plan_gemm(int64_t M, int64_t N, int64_t K, uint32_t n_cu, bool with_ws) {
  GemmPlan g{};
  g.n_split = (uint32_t)N;
  const bool aligned = (K % 64) == 0;
  if (M == 0) {
    g.first = GemmPlan::kNone;
  } else if (aligned && N <= 96) {
    g.first = GemmPlan::kSplitkNarrow;
  } else if (aligned && M <= 32) {
    g.first = M <= 8 ? GemmPlan::kSplitkDecodeFew : GemmPlan::kSplitkDecode;
  } else if (aligned) {
    // Square tiles fill whole rounds of one workgroup per CU.  When the last
    // round would be at most half full and its tiles make whole tile
    // columns, those columns run as a second launch: with a workspace and
    // K % 512 == 0, the same square tiles as two K halves on twice the CUs
    // (FP32 partial sums, then a summing pass: about 0.55 of a round plus
    // the pass); otherwise as 256 x 128 tiles (two per CU), about 0.7 of a
    // round.  Scale super-stages need K % 256 == 0 (whole groups of 4
    // chunks).
    g.first = (K % 256) == 0 ? GemmPlan::kLdsSuper : GemmPlan::kLdsSquare;
    const uint32_t tiles_m = (uint32_t)((M + kSquareTile - 1) / kSquareTile);
    const uint32_t tiles_n = (uint32_t)((N + kSquareTile - 1) / kSquareTile);
    const uint32_t rem = n_cu ? (tiles_m * tiles_n) % n_cu : 0;
    if (rem != 0 && rem <= n_cu / 2 && rem % tiles_m == 0 && rem / tiles_m < tiles_n) {
      g.n_split = (tiles_n - rem / tiles_m) * kSquareTile;
      g.second = (with_ws && K % 512 == 0) ? GemmPlan::kLdsSuperHalves : GemmPlan::kLdsTall;
    }
  } else {
    g.first = GemmPlan::kReg;
  }
  return g;
}

size_t plan_workspace_bytes(const GemmPlan& g, int64_t M, int64_t N) {
  if (g.second != GemmPlan::kLdsSuperHalves) return 0;
  return (size_t)2 * (size_t)M * (size_t)halves_row((uint32_t)N - g.n_split) * sizeof(float);
}

const char* gemm_kernel_name(int kind) {
  switch (kind) {
    case GemmPlan::kLdsSquare: return "gemm_lds_kernel<LdsSquare> (256x256 tiles)";
    case GemmPlan::kLdsSuper: return "gemm_lds_kernel<LdsSquareSuper> (256x256 tiles, scale super-stages)";
    case GemmPlan::kLdsTall: return "gemm_lds_kernel<LdsTall> (256x128 tiles)";
    case GemmPlan::kLdsSuperHalves:
      return "gemm_lds_kernel<LdsSquareSuper> (256x256 tiles, two K halves, FP32 partials) + sum_halves_kernel";
    case GemmPlan::kSplitkNarrow: return "gemm_splitk_kernel<4,2,3,3> (64x96 tiles, split-K)";
    case GemmPlan::kSplitkDecode: return "gemm_splitk_kernel<4,1,2,3> (32x64 tiles, split-K, shared activation ring)";
    case GemmPlan::kSplitkDecodeFew: return "gemm_splitk_kernel<4,1,1,3> (32x32 tiles, split-K, per-wave rings)";
    case GemmPlan::kReg: return "gemm_reg_kernel<2,2,4,4> (256x256 tiles, register path)";
    default: return "none";
  }
}

const char* gemm_kernel_for(int64_t M, int64_t N, int64_t K, int part, bool with_ws) {
  const uint32_t n_cu = cu_count();
  if (n_cu == 0) return nullptr;
  const GemmPlan g = plan_gemm(M, N, K, n_cu, with_ws);
  const int kind = part == 0 ? g.first : g.second;
  return kind == GemmPlan::kNone ? nullptr : gemm_kernel_name(kind);
}

static hipError_t run_one(int kind, const GemmOperands& o, const GemmParams& p, uint32_t n_begin, uint32_t n_end,
                          bool out_f32, bool aligned, hipStream_t stream) {
  switch (kind) {
    case GemmPlan::kLdsSquare: return launch_lds_square(o, p, n_begin, n_end, out_f32, stream);
    case GemmPlan::kLdsSuper:
      return out_f32 ? launch_lds_super_f32(o, p, n_begin, n_end, stream)
                     : launch_lds_super_bf16(o, p, n_begin, n_end, stream);
    case GemmPlan::kLdsTall: return launch_lds_tall(o, p, n_begin, n_end, out_f32, stream);
    case GemmPlan::kSplitkNarrow: return launch_splitk_narrow(o, p, out_f32, false, stream);
    case GemmPlan::kSplitkDecode:
    case GemmPlan::kSplitkDecodeFew: return launch_splitk_decode(o, p, out_f32, stream);
    case GemmPlan::kReg: return launch_reg_square(o, p, out_f32, aligned, stream);
    default: return hipSuccess;
  }
}

size_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  const uint32_t n_cu = cu_count();
  if (n_cu == 0 || M == 0) return 0;
  return plan_workspace_bytes(plan_gemm(M, N, K, n_cu, true), M, N);
}

hipError_t launch_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_g,
                       int64_t M, int64_t K, const void* w_packed, int64_t N,
                       const int64_t* seg_offsets, int n_seg, const float* w_g, void* y,
                       int64_t ldy, bool out_f32, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  GemmParams p = gemm_params(M, K, N, seg_offsets, n_seg, ldy);
  p.y_pairs = (ldy % 2 == 0) && (reinterpret_cast<uintptr_t>(y) % 4 == 0) ? 1u : 0u;
  p.y_stream = !out_f32 && (uint64_t)M * (uint64_t)N * 2u >= kMallBytes ? 1u : 0u;
  const GemmOperands o{a_codes, a_scales, a_g, static_cast<const uint8_t*>(w_packed), w_g, y};
  GemmPlan g = plan_gemm(M, N, K, cu_count(), workspace != nullptr);
  if (g.second == GemmPlan::kLdsSuperHalves && workspace_bytes < plan_workspace_bytes(g, M, N))
    g = plan_gemm(M, N, K, cu_count(), false);
  const bool aligned = (K % 64) == 0;
  hipError_t e = run_one(g.first, o, p, 0, g.n_split, out_f32, aligned, stream);
  if (e != hipSuccess || g.second == GemmPlan::kNone) return e;
  if (g.second == GemmPlan::kLdsSuperHalves) {
    float* parts = static_cast<float*>(workspace);
    e = launch_lds_super_halves(o, p, g.n_split, (uint32_t)N, parts, stream);
    if (e != hipSuccess) return e;
    return launch_sum_halves(parts, (uint32_t)M, (uint32_t)N - g.n_split, y, (uint32_t)ldy, g.n_split, out_f32, stream);
  }
  return run_one(g.second, o, p, g.n_split, (uint32_t)N, out_f32, aligned, stream);
}

hipError_t launch_gemm_gdn_gates(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_g,
                                 int64_t M, int64_t K, const void* w_packed, int64_t H, const float* w_g,
                                 const float* a_log, const float* dt_bias, void* y, int64_t ldy,
                                 bool out_f32, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  const int64_t offs[3] = {0, H, 2 * H};
  GemmParams p = gemm_params(M, K, 2 * H, offs, 2, ldy);
  p.gate_a_log = a_log;
  p.gate_dt_bias = dt_bias;
  p.gate_h = (uint32_t)H;
  const GemmOperands o{a_codes, a_scales, a_g, static_cast<const uint8_t*>(w_packed), w_g, y};
  return launch_splitk_narrow(o, p, out_f32, true, stream);
}

}  // namespace nvfp4
