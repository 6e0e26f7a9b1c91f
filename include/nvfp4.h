/*
 * nvfp4.h -- C ABI of the MI355X (gfx950) NVFP4 W4A4 linear layer.
 *
 * NVFP4 (paper, section 2 "NVFP4"): E2M1 4-bit values, one E4M3 scale per
 * 16-element block set to the block maximum / 6, and one FP32 scale per
 * tensor.  W4A4: weights and activations are both quantized this way and the
 * GEMM consumes the 4-bit operands.  Fused modules (paper, section 6,
 * "Per-module calibration vs. fused-GEMM scaling"): one GEMM serves several
 * separately calibrated linear modules, so the output columns of each module
 * (a "segment") carry that module's own FP32 weight scale, and the GEMM
 * epilogue applies it per segment.
 *
 * Numerics (identical in every entry point):
 *   G      = fl32(2688 / amax) per tensor (2688 = 6 * 448), 0 if amax = 0,
 *            the largest finite float if the quotient overflows;
 *   S_b    = RNE_E4M3(amax_b * G / 6) per 16-element block along K,
 *            saturating at 448, E4M3 subnormals kept (OCP E4M3FN codes);
 *   code   = sign(x) << 3 | RNE_E2M1(|x| * G / S_b), saturating at 6,
 *            magnitude 0 when S_b = 0; the sign bit of x is always copied.
 *   Each rounding is one round-to-nearest-even of the exact real value.
 *   Codes: byte j of a row holds element 2j in the low nibble and 2j+1 in
 *   the high nibble.
 *   GEMM:  Y[m, n] = sum_k (e S)_A[m, k] (e S)_W[n, k] / (G_A * G_W[s(n)]),
 *          FP32 accumulation; output 0 where G_A * G_W[s] = 0.
 *
 * Conventions.
 *   - All tensor pointers are device pointers, allocated and freed by the
 *     caller, 16-byte aligned (except the GEMM output, see nvfp4_gemm).
 *     The library never allocates device memory, keeps no state between
 *     calls except a per-device property cache, and is safe to call from
 *     several host threads.
 *   - Every call validates its arguments synchronously and returns a status
 *     before anything is enqueued.  Work is enqueued asynchronously on
 *     ``stream`` (a hipStream_t; NULL is the default stream); no call
 *     synchronizes the host.
 *   - Preconditions that are not checked: inputs are finite; buffers do not
 *     overlap; buffers are at least as large as the stated sizes.
 *   - Sizes are element counts unless a name ends in _bytes.
 */
#ifndef NVFP4_H
#define NVFP4_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes returned by every entry point. */
enum nvfp4_status {
  NVFP4_OK = 0,
  NVFP4_EINVAL = 1,        /* null or misaligned pointer, bad shape/stride/mode/segment table */
  NVFP4_EUNSUPPORTED = 2,  /* the current HIP device is not gfx950 */
  NVFP4_EWORKSPACE = 3,    /* workspace or packed buffer smaller than required */
  NVFP4_EHIP = 4           /* a HIP runtime call or kernel launch failed */
};

/* Global-scale mode of a quantization call. */
enum nvfp4_scale_mode {
  NVFP4_DYNAMIC = 0,       /* G computed from the tensor amax on the device and written out */
  NVFP4_STATIC = 1         /* G read from the device scalar(s) passed in (a calibrated scale) */
};

/* Output element type of nvfp4_gemm. */
enum nvfp4_out_dtype {
  NVFP4_BF16 = 0,      /* round-to-nearest-even of the FP32 result */
  NVFP4_F32 = 1
};

#define NVFP4_BLOCK 16          /* elements per block scale, along K */
#define NVFP4_MAX_SEGMENTS 8    /* fused segments per GEMM */

/* Human-readable name of a status code (static string, never NULL). */
const char* nvfp4_status_str(int status);

/* The hipError_t value of the last NVFP4_EHIP failure on the calling host
 * thread (0 if none). */
int nvfp4_last_hip_error(void);

/* Workspace bytes nvfp4_quantize_act needs for an M x K activation (the
 * per-workgroup partial maxima of the dynamic global scale); 0 is a valid
 * answer only in static mode, and the dynamic answer is returned here. */
size_t nvfp4_quantize_act_workspace(int64_t M, int64_t K);

/*
 * Dynamic activation quantization (paper, section 2: NVFP4; section 9
 * "Decode overhead": the activation side is quantized at run time).
 *
 *   x        bf16 [M x K], row stride ldx elements (ldx >= K, ldx % 8 == 0).
 *   codes    out, uint8 [M x K/2] row-major (packed E2M1 pairs, see above).
 *   scales   out, uint8 [M x K/16] row-major E4M3 codes, one per block.
 *   g_enc    one device float: written with G in NVFP4_DYNAMIC mode, read in
 *            NVFP4_STATIC mode (must then be finite and >= 0).
 *   workspace, workspace_bytes: device scratch of at least
 *            nvfp4_quantize_act_workspace(M, K) bytes in dynamic mode;
 *            unused in static mode (may be NULL).  Its contents on entry do
 *            not matter; calls sharing one workspace must be ordered.
 * Requirements: M >= 0, K >= 0, K % 16 == 0, M * K < 2^31.
 * Errors: NVFP4_EINVAL, NVFP4_EWORKSPACE, NVFP4_EUNSUPPORTED, NVFP4_EHIP.
 * M == 0 or K == 0 writes G = 0 in dynamic mode and nothing else.
 */
int nvfp4_quantize_act(const void* x, int64_t M, int64_t K, int64_t ldx,
                       uint8_t* codes, uint8_t* scales, float* g_enc, int mode,
                       void* workspace, size_t workspace_bytes, void* stream);

/*
 * nvfp4_quantize_act without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments (minus the workspace),
 * same kernels, same results as nvfp4_quantize_act.
 *
 * The dynamic global scale's partial maxima go to a scratch array of
 * 4096 bytes per device, which the library holds from its first call on that
 * device until the process ends.  The call allocates nothing and calls no
 * allocating routine.  Every call on a device shares that device's scratch:
 * calls that overlap on one GPU race (order them, e.g. on one stream); calls
 * on different GPUs do not interact.  Its contents between calls do not
 * matter (nothing in it needs to start at zero).
 * Errors: as nvfp4_quantize_act; NVFP4_EWORKSPACE if the call would need more
 * scratch than 4096 bytes (no current shape does).
 */
int nvfp4_quantize_act_noalloc(const void* x, int64_t M, int64_t K, int64_t ldx,
                               uint8_t* codes, uint8_t* scales, float* g_enc,
                               int mode, void* stream);

/*
 * RMSNorm fused with activation quantization under a calibrated (static)
 * global scale: one pass over the activations (the paper serves its W4A4
 * model with activation scales calibrated offline, section 3 "Checkpoints";
 * NVFP4 itself: section 2).
 *
 *   y = RNE_bf16((x * r) * gamma),  r = 1 / sqrt(sum_k x^2 / K + eps),
 *   evaluated in binary32 per row (the sum of squares in a fixed order, r with
 *   correctly rounded division and square root);
 *   codes, scales = the NVFP4 quantization of y under G = *g_enc, exactly as
 *   nvfp4_quantize_act in NVFP4_STATIC mode would write them for y.
 *
 *   x       bf16 [M x K], row stride ldx elements (ldx >= K, ldx % 8 == 0).
 *   gamma   bf16 [K] (device).
 *   eps     >= 0, finite.
 *   codes, scales   out, as for nvfp4_quantize_act (contiguous rows).
 *   g_enc   device float: the calibrated G (read only).
 *   y       optional out (may be NULL): the normalized bf16 [M x K], row
 *           stride ldy elements.
 * Requirements: M >= 0, K >= 16, K % 16 == 0, M * ldx < 2^31; pointers
 * 16-byte aligned (g_enc 4-byte).  M == 0 enqueues nothing.
 * Errors: NVFP4_EINVAL, NVFP4_EUNSUPPORTED, NVFP4_EHIP.
 */
int nvfp4_rmsnorm_quantize_act(const void* x, int64_t M, int64_t K, int64_t ldx,
                               const void* gamma, float eps, uint8_t* codes,
                               uint8_t* scales, const float* g_enc, void* y,
                               int64_t ldy, void* stream);

/* Bytes of the packed weight buffer for an N x K weight: the GEMM-private
 * tile layout of the codes and block scales, N padded to 32 and K to 64. */
size_t nvfp4_packed_weight_bytes(int64_t N, int64_t K);

/* Workspace bytes nvfp4_pack_weight needs (per-segment partial maxima). */
size_t nvfp4_pack_weight_workspace_bytes(int64_t N, int64_t K, int n_seg);

/*
 * Weight quantization and prepack (offline).  The rows of W are the output
 * columns of the GEMM; rows [seg_offsets[s], seg_offsets[s+1]) form segment
 * s, a separately calibrated module with its own global scale (paper,
 * section 6: one FP32 global scale per linear module).
 *
 *   w            bf16 [N x K], row stride ldw elements (ldw >= K, ldw % 8 == 0).
 *   seg_offsets  HOST array of n_seg + 1 entries, strictly increasing from 0
 *                to N; 1 <= n_seg <= NVFP4_MAX_SEGMENTS.
 *   g_enc_seg    device float [n_seg]: written with each segment's G in
 *                NVFP4_DYNAMIC mode (from that segment's amax), read in
 *                NVFP4_STATIC mode.
 *   packed       out, device buffer of packed_bytes >=
 *                nvfp4_packed_weight_bytes(N, K) bytes; its layout is private
 *                to nvfp4_gemm (nvfp4_unpack_weight gives the canonical form).
 *   workspace    device scratch of nvfp4_pack_weight_workspace_bytes bytes
 *                (dynamic mode; may be NULL in static mode).
 * Requirements: N >= 1, K >= 16, K % 16 == 0, N * K < 2^31.
 */
int nvfp4_pack_weight(const void* w, int64_t N, int64_t K, int64_t ldw,
                      const int64_t* seg_offsets, int n_seg, float* g_enc_seg,
                      int mode, void* packed, size_t packed_bytes,
                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * Inverse of the prepack layout, for verification: writes the canonical
 * codes uint8 [N x K/2] and scales uint8 [N x K/16] of a packed weight.
 */
int nvfp4_unpack_weight(const void* packed, int64_t N, int64_t K,
                        uint8_t* codes, uint8_t* scales, void* stream);

/*
 * Global-scale harmonization of a fused weight group (paper, section 6,
 * "Per-module calibration vs. fused-GEMM scaling": the checkpoint-side
 * repair that lets one global scale serve several per-module-calibrated
 * segments).  Rewrites a packed weight IN PLACE so that the whole group uses
 * one shared global scale:
 *   G_shared = the smallest G_s > 0 (the scale of the segment with the
 *              largest amax; 0 if every G_s is 0),
 *   every block scale S of segment s becomes RNE_E4M3(S * G_shared / G_s)
 *   (one round-to-nearest-even of the exact value, ties to the even code,
 *   E4M3 subnormals kept; segments with G_s = 0 or G_s = G_shared are left
 *   as they are).  The E2M1 codes do not change.  Afterwards call nvfp4_gemm
 *   with one segment [0, N] and w_g_enc_seg = g_shared.
 *
 *   packed       in/out, a packed weight for this N and K.
 *   seg_offsets  HOST array, as for nvfp4_pack_weight.
 *   g_enc_seg    device float [n_seg]: the segments' G_s (read only).
 *   g_shared     out, device float: G_shared; must not lie inside g_enc_seg.
 * Requirements: as for nvfp4_unpack_weight; valid segments.
 * Errors: NVFP4_EINVAL, NVFP4_EUNSUPPORTED, NVFP4_EHIP.
 */
int nvfp4_harmonize_weight(void* packed, int64_t N, int64_t K,
                           const int64_t* seg_offsets, int n_seg,
                           const float* g_enc_seg, float* g_shared, void* stream);

/*
 * NVFP4 x NVFP4 GEMM with FP32 accumulation and a per-segment scaled
 * epilogue (paper, section 2: W4A4 GEMM on 4-bit operands; section 6: each
 * fused segment scaled by its own module's global scale).
 *
 *   a_codes, a_scales  the activation as written by nvfp4_quantize_act
 *                      ([M x K/2] and [M x K/16], contiguous rows).
 *   a_g_enc            device float: G_A.
 *   w_packed           the weight as written by nvfp4_pack_weight for the
 *                      same N and K.
 *   seg_offsets        HOST array, as for nvfp4_pack_weight (same segments).
 *   w_g_enc_seg        device float [n_seg]: G_W per segment.
 *   y                  out, [M x N] with row stride ldy elements (ldy >= N),
 *                      bf16 or float per y_dtype, aligned to its element size.
 *   Y[m, n] = (1 / (G_A * G_W[s])) * sum_k (e S)_A[m, k] (e S)_W[n, k]
 *   for the segment s holding column n.
 * Requirements: M >= 0, N >= 1, K >= 16, K % 16 == 0, M*K, N*K, M*ldy < 2^31.
 * M == 0 enqueues nothing.  A bf16 Y of at least 256 MB (the MI355X's
 * last-level cache) is written with non-temporal stores, so it is not left
 * in that cache.
 */
int nvfp4_gemm(const uint8_t* a_codes, const uint8_t* a_scales,
               const float* a_g_enc, int64_t M, int64_t K,
               const void* w_packed, int64_t N,
               const int64_t* seg_offsets, int n_seg, const float* w_g_enc_seg,
               void* y, int64_t ldy, int y_dtype, void* stream);

/*
 * Workspace bytes that let nvfp4_gemm_with_workspace run an M x N x K call
 * in its K-halves form on the current device; 0 when the shape does not use
 * it (then any workspace, or none, gives the nvfp4_gemm launches) or the
 * arguments are invalid.  The form applies when the last round of 256 x 256
 * output tiles (one per compute unit) would be at most half full, those
 * tiles make whole tile columns, and K % 512 == 0 (e.g. 8192 x 5120 x 17408:
 * 2 * 8192 * 1024 * 4 bytes).
 */
size_t nvfp4_gemm_workspace(int64_t M, int64_t N, int64_t K);

/*
 * nvfp4_gemm with a caller workspace (same arguments, same result contract
 * up to the summation order).  For shapes where nvfp4_gemm_workspace is
 * non-zero, the output tiles of the partially filled last round are computed
 * as two K halves on twice as many compute units: each half writes its
 * segment-scaled FP32 partial sums to the workspace ([2][M][tail columns]),
 * and a second pass writes y = half0 + half1 (one FP32 addition; bf16 output
 * is that sum rounded to nearest even).  Three launches on `stream` instead
 * of two; the workspace is overwritten and must not be used by another call
 * in flight.
 *   workspace        device memory, 16-byte aligned, or NULL when
 *                    nvfp4_gemm_workspace(M, N, K) is 0.
 *   workspace_bytes  its size.
 * Errors: as nvfp4_gemm; NVFP4_EWORKSPACE if the workspace is smaller than
 * nvfp4_gemm_workspace(M, N, K); NVFP4_EINVAL for a misaligned workspace.
 */
int nvfp4_gemm_with_workspace(const uint8_t* a_codes, const uint8_t* a_scales,
                              const float* a_g_enc, int64_t M, int64_t K,
                              const void* w_packed, int64_t N,
                              const int64_t* seg_offsets, int n_seg, const float* w_g_enc_seg,
                              void* y, int64_t ldy, int y_dtype,
                              void* workspace, size_t workspace_bytes, void* stream);

/*
 * Which kernels an M x N x K GEMM launches on the current device
 * (diagnostics: benchmarks and profiles name the kernel they time), for
 * nvfp4_gemm (with_workspace = 0) or nvfp4_gemm_with_workspace given a
 * sufficient workspace (with_workspace = 1).  part 0: the first launch;
 * part 1: the launch(es) of a shape whose partially filled last round of
 * tiles runs in another form.  Returns a static string naming the kernel
 * and its tile shape, or NULL when that launch does not exist (M == 0, no
 * second launch) or the arguments are invalid (K % 16 != 0, N < 1, M < 0,
 * part not 0 or 1, with_workspace not 0 or 1) or the device cannot be
 * queried.
 */
const char* nvfp4_gemm_kernel(int64_t M, int64_t N, int64_t K, int part, int with_workspace);

/*
 * The fused GDN gate projection with the gate transform in its epilogue
 * (paper, Eq. 1; the b and a projections are served as one fused GEMM,
 * section 6).  The weight is the fused [b; a] projection packed by
 * nvfp4_pack_weight with N = 2H and segments [0, H, 2H] (b rows first).
 * For token m and head h, with v = the segment-scaled GEMM output:
 *   y[m, h]     = beta  = 1 / (1 + exp(-v_b))
 *   y[m, H + h] = alpha = exp(-exp(A_log[h]) * softplus(v_a + dt_bias[h]))
 * evaluated in binary32 (softplus(x) = log1p(exp(x)), and x for x > 20).
 *
 *   a_codes, a_scales, a_g_enc   as for nvfp4_gemm.
 *   w_packed     the packed [b; a] weight (N = 2H rows).
 *   w_g_enc_seg  device float [2]: G_W of the b and a segments.
 *   a_log, dt_bias   device float [H].
 *   y            out, [M x 2H] (beta | alpha), row stride ldy >= 2H, bf16 or
 *                float per y_dtype.
 * Requirements: as for nvfp4_gemm; K % 64 == 0 (NVFP4_EUNSUPPORTED otherwise).
 */
int nvfp4_gemm_gdn_gates(const uint8_t* a_codes, const uint8_t* a_scales,
                         const float* a_g_enc, int64_t M, int64_t K,
                         const void* w_packed, int64_t H, const float* w_g_enc_seg,
                         const float* a_log, const float* dt_bias,
                         void* y, int64_t ldy, int y_dtype, void* stream);

/* Workspace bytes nvfp4_quantize_gemm needs for an M x N x K call. */
size_t nvfp4_quantize_gemm_workspace(int64_t M, int64_t N, int64_t K);

/*
 * Activation quantization fused into the GEMM, in one call, for the shapes
 * where a separate quantizer launch costs most (paper, section 2 for the
 * format, section 6 for the fused segments; section 4 and section 9
 * "Decode overhead": small-batch activation quantization):
 *   - narrow outputs, N <= 128 (the tall-skinny gate projections), any M:
 *     X is quantized in registers inside the GEMM (read once with a given
 *     G; dynamic mode adds the amax pass in front);
 *   - decode shapes, M <= 32 (any N): for M * K <= 16384 (up to 3 tokens
 *     of width 5120) one launch in which every workgroup quantizes all of
 *     X into its LDS (and takes the dynamic G itself) and the GEMM reads
 *     the activation from there; larger activations take two launches (the
 *     quantizer, then the GEMM), with the codes in a_codes or in the
 *     workspace.
 * The result equals nvfp4_quantize_act followed by nvfp4_gemm: the same
 * codes, scales and G_A, and the GEMM sums in the same order as nvfp4_gemm
 * at these shapes.
 *
 *   x, M, K, ldx   bf16 activation, as for nvfp4_quantize_act.
 *   a_g_enc        one device float: G_A, written (NVFP4_DYNAMIC) or read
 *                  (NVFP4_STATIC), as for nvfp4_quantize_act.
 *   workspace, workspace_bytes   device scratch of at least
 *                  nvfp4_quantize_gemm_workspace(M, N, K) bytes, 16-byte
 *                  aligned; required in dynamic mode and on the decode path
 *                  (M <= 32 and N > 128), else unused (may be NULL).  Its
 *                  contents on entry do not matter; calls sharing one
 *                  workspace must be ordered.
 *   w_packed, N, seg_offsets, n_seg, w_g_enc_seg, y, ldy, y_dtype
 *                  as for nvfp4_gemm.
 *   a_codes, a_scales   optional outputs ([M x K/2], [M x K/16] as written
 *                  by nvfp4_quantize_act); both NULL or both set.
 * Requirements: those of nvfp4_quantize_act and nvfp4_gemm; N > 128 with
 * M > 32, or K % 64 != 0, gives NVFP4_EUNSUPPORTED.
 */
int nvfp4_quantize_gemm(const void* x, int64_t M, int64_t K, int64_t ldx,
                        float* a_g_enc, int mode, void* workspace, size_t workspace_bytes,
                        const void* w_packed, int64_t N,
                        const int64_t* seg_offsets, int n_seg, const float* w_g_enc_seg,
                        uint8_t* a_codes, uint8_t* a_scales,
                        void* y, int64_t ldy, int y_dtype, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* NVFP4_H */
