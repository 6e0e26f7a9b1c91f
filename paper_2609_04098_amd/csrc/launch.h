// Host-side launchers of the NVFP4 kernels (called by api.cpp after argument
// validation) and the constants that size their workspaces.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

// Entries of the segment-offset table passed to kernels (max segments + 1).
#define NVFP4_SEG_TABLE 9

namespace nvfp4 {

// Partial maxima written by the activation amax pass (one per workgroup).
constexpr int kActPartials = 1024;
// Bytes of the per-device scratch array of the allocation-free quantizer
// (the partial maxima).
constexpr size_t kActScratchBytes = kActPartials * sizeof(float);
// Upper bound on quantize workgroups (grid-strided beyond that): 8 per CU
// of a 256-CU device, 8 waves per SIMD.  In dynamic mode every workgroup
// first reduces the amax pass's partial maxima, so fewer, longer-lived
// workgroups spend less on that preamble.
constexpr int kActQuantGridCap = 2048;
// Partial maxima per weight segment.
constexpr int kWeightPartials = 256;

hipError_t launch_act_quant(const void* x, int64_t M, int64_t K, int64_t ldx, uint8_t* codes,
                            uint8_t* scales, float* g_enc, bool dynamic, float* partial,
                            hipStream_t stream);

// Device address of the current device's scratch array (kActScratchBytes),
// taken once per device with hipGetSymbolAddress.
hipError_t act_scratch(float** ptr);

// Pass 1 of the dynamic quantizer: partial maxima of |x| into `partial`
// (n_partial <= kActPartials values).
hipError_t launch_act_amax(const void* x, int64_t M, int64_t K, int64_t ldx, float* partial, int* n_partial,
                           hipStream_t stream);

hipError_t launch_rmsnorm_quant(const void* x, int64_t M, int64_t K, int64_t ldx, const void* gamma,
                                float eps, const float* g_enc, uint8_t* codes, uint8_t* scales, void* y,
                                int64_t ldy, hipStream_t stream);

hipError_t launch_pack_weight(const void* w, int64_t N, int64_t K, int64_t ldw,
                              const int64_t* seg_offsets, int n_seg, float* g_enc_seg,
                              bool dynamic, void* packed, float* partial, hipStream_t stream);

hipError_t launch_unpack_weight(const void* packed, int64_t N, int64_t K, uint8_t* codes,
                                uint8_t* scales, hipStream_t stream);

hipError_t launch_harmonize_weight(void* packed, int64_t N, int64_t K, const int64_t* seg_offsets,
                                   int n_seg, const float* g_enc_seg, float* g_shared,
                                   hipStream_t stream);

// nvfp4_gemm and nvfp4_gemm_with_workspace: workspace may be null (then
// workspace_bytes is ignored); a workspace of gemm_workspace_bytes(M, N, K)
// bytes or more enables the K-halves form of a partial last round.
hipError_t launch_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_g,
                       int64_t M, int64_t K, const void* w_packed, int64_t N,
                       const int64_t* seg_offsets, int n_seg, const float* w_g, void* y,
                       int64_t ldy, bool out_f32, void* workspace, size_t workspace_bytes, hipStream_t stream);
size_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K);

// Name of launch `part` (0 or 1) of launch_gemm for this shape on the
// current device, with or without a sufficient workspace; NULL if that
// launch does not exist.
const char* gemm_kernel_for(int64_t M, int64_t N, int64_t K, int part, bool with_ws);

hipError_t launch_gemm_gdn_gates(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_g,
                                 int64_t M, int64_t K, const void* w_packed, int64_t H, const float* w_g,
                                 const float* a_log, const float* dt_bias, void* y, int64_t ldy,
                                 bool out_f32, hipStream_t stream);

// nvfp4_quantize_gemm: M <= 32 with N > 128 takes the fused decode path.
bool quant_gemm_uses_decode_path(int64_t M, int64_t N);
size_t quant_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K);
hipError_t launch_quant_gemm(const void* x, int64_t M, int64_t K, int64_t ldx, float* g_enc, bool dynamic,
                             void* workspace, const void* w_packed, int64_t N, const int64_t* seg_offsets,
                             int n_seg, const float* w_g, uint8_t* codes, uint8_t* scales, void* y, int64_t ldy,
                             bool out_f32, hipStream_t stream);

}  // namespace nvfp4
