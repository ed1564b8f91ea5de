/*
 * jq.h -- C ABI of libjq, an MI355X (gfx950) implementation of the plain W4A4
 * linear layer: dynamic per-token symmetric int4 activation quantisation, an
 * int4 x int4 matrix product with exact int32 accumulation and a dequantising
 * epilogue that writes bf16.
 *
 * The operator.  The paper's quantised network keeps the topology of the
 * full-precision one and replaces each module by a low-bit operator of the
 * deployment family (Sec. 3.1 "Quantization as distillation"); for W4A4 that
 * family is INT4 weights and INT4 activations (appendix "Experimental
 * Details", quantization-function rows), executed by quantisation, packing and
 * low-bit matrix-multiplication kernels with no smoothing, rotation,
 * normalisation or SVD branch (appendix FAQ Q7).  The paper states no formula,
 * so the library implements this reading of it, per row r of a bf16 matrix:
 *
 *     a_r    = max_k |x[r,k]|
 *     s_r    = fl32(a_r / 7)                                  (IEEE fp32 division)
 *     q[r,k] = clamp(rne(fl32(x[r,k] / s_r)), -8, 7),  q = 0 if s_r = 0
 *
 * (rne = round half to even).  Activations X[M,K] get one scale per token
 * (row), weights W[N,K] one scale per output channel (row).  The layer is
 *
 *     acc[m,n] = sum_k qx[m,k] * qw[n,k]                       (exact integer)
 *     y[m,n]   = bf16_rne(((fl32(acc) * s_x[m]) * s_w[n]) + bias[n])
 *
 * with each fp32 operation rounded on its own (no fused multiply-add).
 *
 * Packed int4 layout (activations and weights alike): row-major [rows, K/2]
 * bytes; byte j of a row holds code 2j in its low nibble and code 2j+1 in its
 * high nibble, both as 4-bit two's complement.
 *
 * Conventions for every call:
 *   - All tensor pointers are DEVICE pointers, owned by the caller; the library
 *     never allocates device memory, never synchronises and never prints.
 *   - Every call is asynchronous on `stream` (a hipStream_t passed as void*;
 *     NULL means the default stream).  Outputs are valid once the stream has
 *     reached the call.
 *   - Matrices are contiguous and row-major.  bf16 is passed as raw 16-bit
 *     patterns (void*).
 *   - Shapes: rows (M, N) >= 1; K >= 64 and K % 64 == 0, else
 *     JQ_ERR_UNSUPPORTED_SHAPE; K <= 65536 so that every accumulator stays
 *     exact in int32 and in fp32; rows <= 2^30 and, for the GEMM calls,
 *     ceil(M/256) * ceil(N/256) <= 2^26 and each packed operand (M*K/2 and
 *     N*K/2 bytes) below 2 GiB, else JQ_ERR_UNSUPPORTED_SHAPE.
 *     Non-positive sizes or required NULL pointers give JQ_ERR_INVALID_ARG.
 *   - Matrix and packed pointers must be 16-byte aligned and scale/bias pointers
 *     4-/2-byte aligned, else JQ_ERR_MISALIGNED.
 *   - Arguments are checked before anything is launched: on any error nothing
 *     is written.  A failed kernel launch returns JQ_ERR_HIP; faults during
 *     execution surface at the caller's next synchronisation.
 *   - There is no global mutable state apart from the device scratch of
 *     jq_w4a4_f6_linear_noalloc (and the per-device address of it, resolved
 *     once under a lock): calls may be made from several host threads at once
 *     (on one stream they execute in issue order).
 */
#ifndef JQ_H
#define JQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  JQ_OK = 0,
  JQ_ERR_INVALID_ARG = 1,
  JQ_ERR_UNSUPPORTED_SHAPE = 2,
  JQ_ERR_MISALIGNED = 3,
  JQ_ERR_WORKSPACE_TOO_SMALL = 4,
  JQ_ERR_HIP = 5
} jq_status;

/* Human-readable name of a status code (static string, never NULL). */
const char* jq_status_string(jq_status s);

/* Library version as major*10000 + minor*100 + patch. */
int jq_version(void);

/*
 * Activation quantisation (Sec. 3.1; FAQ Q7: the quantisation and packing
 * kernel).  Quantises each row (token) of x_bf16 [M,K] with its own scale.
 *   x_bf16   in   [M,K] bf16, 16-byte aligned
 *   q_packed out  [M,K/2] uint8 in the packed layout above, 16-byte aligned
 *   scale    out  [M] fp32, s_r as defined above
 * Errors: JQ_ERR_INVALID_ARG, JQ_ERR_UNSUPPORTED_SHAPE, JQ_ERR_MISALIGNED, JQ_ERR_HIP.
 */
jq_status jq_quantize_act(const void* x_bf16, int64_t M, int64_t K,
                          void* q_packed, float* scale, void* stream);

/*
 * Weight quantisation and packing (Sec. 3.1; FAQ Q7), done once per layer
 * when a model is loaded.  Per-output-channel scaling of W [N,K] is the same
 * row quantiser applied to the rows of W.
 *   w_bf16    in   [N,K] bf16
 *   wq_packed out  [N,K/2] uint8 (packed layout above)
 *   w_scale   out  [N] fp32
 * Errors: as jq_quantize_act.
 */
jq_status jq_pack_weight_int4(const void* w_bf16, int64_t N, int64_t K,
                              void* wq_packed, float* w_scale, void* stream);

/*
 * Bytes of device workspace jq_w4a4_linear needs for an [M,K] input: the
 * packed activations (M*K/2 bytes) and their scales (4*M bytes), each part
 * rounded up to 256 bytes.  Returns 0 for invalid sizes.
 */
size_t jq_w4a4_workspace_bytes(int64_t M, int64_t K);

/*
 * The whole W4A4 linear (Sec. 3.1, FAQ Q7): quantise x per token into the
 * workspace, then the int4 GEMM with the fused epilogue.
 *   x_bf16      in   [M,K] bf16
 *   wq_packed   in   [N,K/2] uint8 from jq_pack_weight_int4
 *   w_scale     in   [N] fp32 from jq_pack_weight_int4
 *   bias_bf16   in   [N] bf16, or NULL for no bias
 *   y_bf16      out  [M,N] bf16, 16-byte aligned
 *   workspace   scratch of at least jq_w4a4_workspace_bytes(M,K) bytes,
 *               256-byte aligned, owned by the caller; its contents on return
 *               are the packed activations followed by their scales.
 * Errors: as jq_quantize_act, plus JQ_ERR_WORKSPACE_TOO_SMALL.
 */
jq_status jq_w4a4_linear(const void* x_bf16, int64_t M, int64_t K,
                         const void* wq_packed, const float* w_scale, int64_t N,
                         const void* bias_bf16, void* y_bf16,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * GEMM + epilogue on already-quantised activations (Sec. 3.1, FAQ Q7: the
 * low-bit matrix multiplication).  Lets several linears that read the same
 * input share one quantisation.
 *   q_packed, scale   in  [M,K/2] uint8 and [M] fp32 from jq_quantize_act
 *   wq_packed, w_scale, bias_bf16, y_bf16: as jq_w4a4_linear
 * Errors: JQ_ERR_INVALID_ARG, JQ_ERR_UNSUPPORTED_SHAPE, JQ_ERR_MISALIGNED, JQ_ERR_HIP.
 */
jq_status jq_w4a4_gemm(const void* q_packed, const float* scale, int64_t M, int64_t K,
                       const void* wq_packed, const float* w_scale, int64_t N,
                       const void* bias_bf16, void* y_bf16, void* stream);

/*
 * The exact integer contraction alone, for checking (Sec. 3.1, FAQ Q7):
 * acc[m,n] = sum_k qx[m,k] * qw[n,k] written as int32 [M,N] (16-byte aligned),
 * computed by the same kernel as jq_w4a4_gemm with the epilogue replaced by a
 * plain store.
 * Errors: JQ_ERR_INVALID_ARG, JQ_ERR_UNSUPPORTED_SHAPE, JQ_ERR_MISALIGNED, JQ_ERR_HIP.
 */
jq_status jq_w4a4_gemm_i32(const void* q_packed, int64_t M, int64_t K,
                           const void* wq_packed, int64_t N, int32_t* acc, void* stream);

/*
 * ---------------------------------------------------------------------------
 * W1.58A4: ternary weights with the same per-token int4 activations.
 *
 * Ternary (1.58-bit) weights with INT4 activations is the paper's W1.58A4
 * deployment setting (Sec. 4 result tables, W1.58A4 rows; appendix
 * experimental-details tables, "Ternary weights, INT4 activations"), run by
 * the same plain operator: quantise, pack, low-bit GEMM, dequantise (Sec. 3.1,
 * FAQ Q7).  The paper states no ternary formula; the library implements the
 * absmean reading, one scale per output channel (row n of W [N,K]):
 *
 *     g[n]   = fl32(fl64(sum_k |w[n,k]|) / K)       (fp64 sum and division)
 *     t[n,k] = clamp(rne(fl32(w[n,k] / g[n])), -1, 1),  t = 0 if g[n] = 0
 *
 * The fp64 sum is exact (so independent of summation order) when a row's
 * nonzero magnitudes span less than 2^29.  The layer is the W4A4 layer with
 * t and g in place of the int4 weight codes and scales:
 *
 *     acc[m,n] = sum_k qx[m,k] * t[n,k]                        (exact integer)
 *     y[m,n]   = bf16_rne(((fl32(acc) * s_x[m]) * g[n]) + bias[n])
 *
 * Packed ternary layout: row-major [N, K/4] bytes; byte j of a row holds codes
 * 4j .. 4j+3, code 4j+i in bits 2i .. 2i+1 as a 2-bit two's-complement field
 * (0 -> 00, 1 -> 01, -1 -> 11).  Shapes, alignment and errors follow the
 * conventions above; the packed weight operand (N*K/4 bytes) must stay below
 * 2 GiB.
 */

/*
 * Ternary weight quantisation and packing, once per layer at model load.
 *   w_bf16    in   [N,K] bf16, 16-byte aligned
 *   wt_packed out  [N,K/4] uint8 (packed ternary layout above), 16-byte aligned
 *   w_scale   out  [N] fp32, g[n] as defined above
 * Errors: JQ_ERR_INVALID_ARG, JQ_ERR_UNSUPPORTED_SHAPE, JQ_ERR_MISALIGNED, JQ_ERR_HIP.
 */
jq_status jq_pack_weight_ternary(const void* w_bf16, int64_t N, int64_t K,
                                 void* wt_packed, float* w_scale, void* stream);

/*
 * The whole W1.58A4 linear: quantise x per token into the workspace (same
 * size and layout as for jq_w4a4_linear, see jq_w4a4_workspace_bytes), then
 * the int4 x ternary GEMM with the fused epilogue.
 *   wt_packed, w_scale   in  [N,K/4] uint8 and [N] fp32 from jq_pack_weight_ternary
 *   other arguments as jq_w4a4_linear
 * Errors: as jq_w4a4_linear.
 */
jq_status jq_w158a4_linear(const void* x_bf16, int64_t M, int64_t K,
                           const void* wt_packed, const float* w_scale, int64_t N,
                           const void* bias_bf16, void* y_bf16,
                           void* workspace, size_t workspace_bytes, void* stream);

/*
 * GEMM + epilogue on already-quantised activations (from jq_quantize_act)
 * and packed ternary weights.  Arguments as jq_w4a4_gemm with wt_packed
 * [N,K/4] in place of wq_packed.
 * Errors: JQ_ERR_INVALID_ARG, JQ_ERR_UNSUPPORTED_SHAPE, JQ_ERR_MISALIGNED, JQ_ERR_HIP.
 */
jq_status jq_w158a4_gemm(const void* q_packed, const float* scale, int64_t M, int64_t K,
                         const void* wt_packed, const float* w_scale, int64_t N,
                         const void* bias_bf16, void* y_bf16, void* stream);

/*
 * The exact integer contraction alone, for checking: acc[m,n] =
 * sum_k qx[m,k] * t[n,k] as int32 [M,N] (16-byte aligned), by the same kernel
 * as jq_w158a4_gemm with the epilogue replaced by a plain store.
 * Errors: JQ_ERR_INVALID_ARG, JQ_ERR_UNSUPPORTED_SHAPE, JQ_ERR_MISALIGNED, JQ_ERR_HIP.
 */
jq_status jq_w158a4_gemm_i32(const void* q_packed, int64_t M, int64_t K,
                             const void* wt_packed, int64_t N, int32_t* acc, void* stream);

/*
 * ---------------------------------------------------------------------------
 * Group-wise W4A4: one scale per G consecutive k (G = 64 or 128).
 *
 * The paper's own W4A4 runs quantise in groups along K: group128 for the DiT
 * and ELF models, group64 for FLUX (appendix experimental-details tables,
 * quantization-function rows).  The library extends the per-token reading to
 * groups, on activations and weights alike, per row r and group g:
 *
 *     s[r,g]  = fl32(max_{k in g} |x[r,k]| / 7)                (IEEE fp32 division)
 *     q[r,k]  = clamp(rne(fl32(x[r,k] / s[r,g(k)])), -8, 7),  q = 0 where s = 0
 *
 * and the layer sums the exact per-group integer products in k order:
 *
 *     acc_g[m,n] = sum_{k in g} qx[m,k] * qw[n,k]                    (exact)
 *     S[m,n]     = 0;  S = fl32(S + fl32(fl32(fl32(acc_g) * s_x[m,g]) * s_w[n,g]))  for g = 0, 1, ...
 *     y[m,n]     = bf16_rne(fl32(S + bias[n]))
 *
 * each fp32 operation rounded on its own (no fused multiply-add).  Codes use
 * the packed int4 layout above; scales are fp32 [rows, K/G] row-major.
 * Shapes: G must be 64 or 128 and K % G == 0, else JQ_ERR_UNSUPPORTED_SHAPE;
 * for the GEMM calls ceil(M/128) * ceil(N/128) <= 2^26; otherwise the
 * conventions above apply.
 */

/*
 * Group-wise activation quantisation.
 *   x_bf16   in   [M,K] bf16, 16-byte aligned
 *   q_packed out  [M,K/2] uint8 (packed int4 layout), 16-byte aligned
 *   scales   out  [M,K/G] fp32, 4-byte aligned
 * Errors: JQ_ERR_INVALID_ARG, JQ_ERR_UNSUPPORTED_SHAPE (also M*K > 2^41),
 * JQ_ERR_MISALIGNED, JQ_ERR_HIP.
 */
jq_status jq_quantize_act_group(const void* x_bf16, int64_t M, int64_t K, int64_t G,
                                void* q_packed, float* scales, void* stream);

/*
 * Group-wise weight quantisation and packing, once per layer at model load:
 * the same quantiser on the rows of W [N,K].
 *   w_bf16 in [N,K] bf16; wq_packed out [N,K/2] uint8; w_scales out [N,K/G] fp32.
 * Errors: as jq_quantize_act_group.
 */
jq_status jq_pack_weight_int4_group(const void* w_bf16, int64_t N, int64_t K, int64_t G,
                                    void* wq_packed, float* w_scales, void* stream);

/*
 * Bytes of device workspace jq_w4a4g_linear needs for an [M,K] input in
 * groups of G: the packed activations (M*K/2 bytes) and their scales
 * (4*M*K/G bytes), each part rounded up to 256 bytes.  0 for invalid sizes.
 */
size_t jq_w4a4g_workspace_bytes(int64_t M, int64_t K, int64_t G);

/*
 * The whole group-wise W4A4 linear: quantise x in groups into the workspace,
 * then the group GEMM with the fused epilogue.
 *   x_bf16       in   [M,K] bf16
 *   wq_packed    in   [N,K/2] uint8 from jq_pack_weight_int4_group (same G)
 *   w_scales     in   [N,K/G] fp32 from jq_pack_weight_int4_group
 *   bias_bf16    in   [N] bf16, or NULL
 *   y_bf16       out  [M,N] bf16, 16-byte aligned
 *   workspace    at least jq_w4a4g_workspace_bytes(M,K,G) bytes, 256-byte
 *                aligned; on return it holds the packed activations followed
 *                by their scales.
 * Errors: as jq_quantize_act_group, plus JQ_ERR_WORKSPACE_TOO_SMALL.
 */
jq_status jq_w4a4g_linear(const void* x_bf16, int64_t M, int64_t K, int64_t G,
                          const void* wq_packed, const float* w_scales, int64_t N,
                          const void* bias_bf16, void* y_bf16,
                          void* workspace, size_t workspace_bytes, void* stream);

/*
 * Group GEMM + epilogue on already-quantised activations.
 *   q_packed, scales   in  [M,K/2] uint8 and [M,K/G] fp32 from jq_quantize_act_group
 *   other arguments as jq_w4a4g_linear
 * Errors: JQ_ERR_INVALID_ARG, JQ_ERR_UNSUPPORTED_SHAPE, JQ_ERR_MISALIGNED, JQ_ERR_HIP.
 */
jq_status jq_w4a4g_gemm(const void* q_packed, const float* scales, int64_t M, int64_t K, int64_t G,
                        const void* wq_packed, const float* w_scales, int64_t N,
                        const void* bias_bf16, void* y_bf16, void* stream);

/*
 * The fp32 group sum S[m,n] alone (before bias and bf16 rounding), for
 * checking: the same kernel as jq_w4a4g_gemm with the epilogue replaced by a
 * plain fp32 store into s_f32 [M,N] (16-byte aligned).
 * Errors: JQ_ERR_INVALID_ARG, JQ_ERR_UNSUPPORTED_SHAPE, JQ_ERR_MISALIGNED, JQ_ERR_HIP.
 */
jq_status jq_w4a4g_gemm_f32(const void* q_packed, const float* scales, int64_t M, int64_t K, int64_t G,
                            const void* wq_packed, const float* w_scales, int64_t N,
                            float* s_f32, void* stream);

/* ------------------------------------------------------------------------
 * BF6 engine: the same W4A4 layer (Sec. 3.1; FAQ Q7: quantisation, packing
 * and low-bit matrix-multiplication kernels) computed on gfx950's 6-bit
 * matrix cores.  Every int4 code -8..7 is exactly representable in the BF6
 * (E3M2) format and every partial sum of the contraction is an integer below
 * 2^22, so the fp32 accumulators equal the exact integer ones: codes, scales,
 * accumulators and bf16 outputs are identical to the packed-int4 calls above.
 *
 * BF6 operands, 6 bits per code:
 *   - a code c is encoded as sign bit 5 and the E3M2 magnitude
 *     |c| = (1 + m/4) * 2^(e-3) (e in bits 4..2, m in bits 1..0; 0 -> 0);
 *   - 32 codes c[0..31] form a 192-bit group, code p in bits 6p..6p+5
 *     (six little-endian dwords d0..d5);
 *   - rows are padded with zero codes to a multiple of 32 and taken in bands
 *     of 32; K is padded with zero codes to a multiple of 128 and cut into
 *     KS = 2*ceil(K/128) k-steps of 64 codes; band b takes KS*1536 bytes at
 *     b*KS*1536.  G(r, s, h) below is the group of codes 64s+32h ..
 *     64s+32h+31 of row 32b + r, and L = r + 32h (r < 32, h < 2).
 *   - Activation layout: k-step s of a band is 1536 bytes at s*1536; d0..d3
 *     of G(r, s, h) at byte 16L, d4..d5 at byte 1024 + 8L.
 *   - Weight layout: k-steps 2u and 2u+1 of a band share 3072 bytes at
 *     u*3072, three planes of 1024 bytes; the 16 bytes at 1024i + 16L
 *     (i = 0, 1, 2), in plane order, are the six dwords of G(r, 2u, h)
 *     followed by those of G(r, 2u+1, h).
 * Size of either: jq_f6_operand_bytes(rows, K) = ceil(rows/32) * KS * 1536.
 *
 * Shapes, alignment and errors follow the conventions at the top of this
 * file, with each BF6 operand below 2^31 bytes.
 * ------------------------------------------------------------------------ */

/* Bytes of the BF6 operand of a [rows,K] matrix (0 for invalid sizes). */
size_t jq_f6_operand_bytes(int64_t rows, int64_t K);

/*
 * Activation quantisation into the BF6 operand (Sec. 3.1; FAQ Q7): the
 * quantiser of jq_quantize_act (same scale, same codes) written in the BF6
 * layout; padding rows get zero codes.
 *   x_bf16  in   [M,K] bf16, 16-byte aligned
 *   xf6     out  jq_f6_operand_bytes(M,K) bytes, 16-byte aligned
 *   scale   out  [M] fp32
 * Errors: as jq_quantize_act.
 */
jq_status jq_quantize_act_f6(const void* x_bf16, int64_t M, int64_t K,
                             void* xf6, float* scale, void* stream);

/*
 * Re-encode packed int4 codes (any codes -8..7) as a BF6 operand in the
 * activation layout; lossless.  Serves activation codes from
 * jq_quantize_act (e.g. to check the GEMM on chosen codes).
 *   q_packed in   [rows,K/2] uint8, 16-byte aligned
 *   f6       out  jq_f6_operand_bytes(rows,K) bytes, 16-byte aligned
 *            (padding rows and codes are written as zeros)
 * Errors: JQ_ERR_INVALID_ARG, JQ_ERR_UNSUPPORTED_SHAPE, JQ_ERR_MISALIGNED, JQ_ERR_HIP.
 */
jq_status jq_int4_to_f6(const void* q_packed, int64_t rows, int64_t K, void* f6, void* stream);

/*
 * The same re-encoding into the weight layout: done once per layer at model
 * load, after jq_pack_weight_int4, whose scales stay the weight scales.
 *   q_packed in   [rows,K/2] uint8, 16-byte aligned
 *   wf6      out  jq_f6_operand_bytes(rows,K) bytes, 16-byte aligned
 * Errors: as jq_int4_to_f6.
 */
jq_status jq_int4_to_f6_weight(const void* q_packed, int64_t rows, int64_t K, void* wf6, void* stream);

/*
 * W1.58A4 on the BF6 engine.  Ternary codes -1, 0, 1 are int4 codes, so the
 * W1.58A4 layer (acc = sum_k qx[m,k] * t[n,k], epilogue with g[n] in place of
 * the int4 weight scale) is jq_w4a4_f6_linear / jq_w4a4_f6_gemm given the
 * ternary codes in the BF6 weight layout and g as w_scale; the result is
 * bit-identical to jq_w158a4_linear / jq_w158a4_gemm.  This re-encodes the
 * packed ternary codes once per layer at model load, losslessly.
 *   wt_packed in   [rows,K/4] uint8 from jq_pack_weight_ternary, 16-byte aligned
 *   wf6       out  jq_f6_operand_bytes(rows,K) bytes, 16-byte aligned
 * Errors: as jq_int4_to_f6.
 */
jq_status jq_ternary_to_f6_weight(const void* wt_packed, int64_t rows, int64_t K, void* wf6, void* stream);

/*
 * Bytes of device workspace jq_w4a4_f6_linear needs for an [M,K] input: the
 * BF6 activation operand and the scales (4*M bytes), each part rounded up to
 * 256 bytes.  0 for invalid sizes.
 */
size_t jq_w4a4_f6_workspace_bytes(int64_t M, int64_t K);

/*
 * The whole W4A4 linear on the BF6 engine: quantise x per token into the
 * workspace (BF6 operand, then scales), then the GEMM with the fused epilogue
 * y = bf16_rne(((fl32(acc) * s_x[m]) * s_w[n]) + bias[n]).
 *   x_bf16      in   [M,K] bf16
 *   wf6         in   BF6 weight operand (weight layout) from jq_int4_to_f6_weight
 *   w_scale     in   [N] fp32 from jq_pack_weight_int4
 *   bias_bf16   in   [N] bf16, or NULL
 *   y_bf16      out  [M,N] bf16, 16-byte aligned
 *   workspace   at least jq_w4a4_f6_workspace_bytes(M,K) bytes, 256-byte aligned
 * Errors: as jq_w4a4_linear.
 */
jq_status jq_w4a4_f6_linear(const void* x_bf16, int64_t M, int64_t K,
                            const void* wf6, const float* w_scale, int64_t N,
                            const void* bias_bf16, void* y_bf16,
                            void* workspace, size_t workspace_bytes, void* stream);

/*
 * The per-token quantiser of jq_quantize_act_f6 on several independent
 * inputs at once (at most JQ_QUANT_BATCH_MAX): input i, x_bf16[i] [M[i], K[i]]
 * bf16, is quantised into xf6[i] (jq_f6_operand_bytes(M[i], K[i]) bytes, the
 * activation layout) and scale[i] [M[i]] fp32, exactly as jq_quantize_act_f6
 * would.  Inputs of up to 16384 codes per row share one launch, so the short
 * quantisation of one input runs inside the bandwidth-bound pass over
 * another instead of as a launch of its own, e.g. the inputs of two linears
 * that do not depend on each other; longer rows get a launch each, on the
 * same stream.  The quantisation and packing kernels are part of the
 * deployed low-bit operator (appendix FAQ Q7); the paper names the
 * non-GEMM time of a step as what makes speed-ups hard to reach on small
 * models (deployment-summary figure caption, Sec. 1).
 *   count   1 .. JQ_QUANT_BATCH_MAX
 *   x_bf16, M, K, xf6, scale   host arrays of count entries; every entry
 *           obeys jq_quantize_act_f6's rules; no output may overlap another
 *           entry's input or output
 * Errors: JQ_ERR_INVALID_ARG (count out of range, a NULL array or entry,
 * non-positive sizes), JQ_ERR_UNSUPPORTED_SHAPE, JQ_ERR_MISALIGNED, JQ_ERR_HIP;
 * every entry is checked before anything is launched.
 */
#define JQ_QUANT_BATCH_MAX 8
jq_status jq_quantize_act_f6_batch(int count, const void* const* x_bf16, const int64_t* M, const int64_t* K,
                                   void* const* xf6, float* const* scale, void* stream);

/*
 * Size of the device scratch that libjq holds for jq_w4a4_f6_linear_noalloc
 * on each device it runs on (96 MiB): room for the BF6 activation operand and
 * the scales of an input of up to about 128 M elements, e.g. the FLUX-12B
 * MLP-down input of two images, 9216 x 12288 (81 MiB).
 */
#define JQ_NOALLOC_SCRATCH_BYTES ((size_t)96 << 20)

/*
 * jq_w4a4_f6_linear for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same layer, kernels and result, with the quantised
 * activations (BF6 operand, then scales) in a scratch array the library
 * holds on each device instead of a caller workspace.  The call allocates
 * nothing and calls no allocating routine; its first call on a device looks
 * up the scratch's address there.  The caller still passes inputs and
 * outputs, with the meaning and layout of jq_w4a4_f6_linear.
 * Nothing in the scratch needs to start at zero: every byte the GEMM reads
 * (the whole operand, padding included, and M scales) is written by the
 * call's own quantiser first.  All calls on one device share the one scratch
 * and it keeps the last call's contents: calls that can overlap on one device
 * (other streams, other host threads) race and must be ordered by the caller.
 * Errors: as jq_w4a4_f6_linear; JQ_ERR_WORKSPACE_TOO_SMALL when
 * jq_w4a4_f6_workspace_bytes(M,K) exceeds JQ_NOALLOC_SCRATCH_BYTES (checked
 * before anything is launched).
 */
jq_status jq_w4a4_f6_linear_noalloc(const void* x_bf16, int64_t M, int64_t K,
                                    const void* wf6, const float* w_scale, int64_t N,
                                    const void* bias_bf16, void* y_bf16, void* stream);

/*
 * GEMM + epilogue of the BF6 engine on an already-quantised activation
 * operand (activation layout, from jq_quantize_act_f6 or jq_int4_to_f6) and
 * its scales; wf6 as in jq_w4a4_f6_linear.
 * Errors: JQ_ERR_INVALID_ARG, JQ_ERR_UNSUPPORTED_SHAPE, JQ_ERR_MISALIGNED, JQ_ERR_HIP.
 */
jq_status jq_w4a4_f6_gemm(const void* xf6, const float* scale, int64_t M, int64_t K,
                          const void* wf6, const float* w_scale, int64_t N,
                          const void* bias_bf16, void* y_bf16, void* stream);

/*
 * The exact contraction alone on the BF6 engine, for checking:
 * acc [M,N] int32 (16-byte aligned) = sum_k qx[m,k] * qw[n,k].
 * Errors: as jq_w4a4_f6_gemm.
 */
jq_status jq_w4a4_f6_gemm_i32(const void* xf6, int64_t M, int64_t K,
                              const void* wf6, int64_t N, int32_t* acc, void* stream);

/*
 * The tile height the int8 engine's GEMM (jq_w4a4_gemm, _linear, _gemm_i32 and
 * their W1.58A4 forms) takes for an M x K by K x N product on a device with
 * `cus` compute units, for checking and tuning: *tile_rows = 128 or 112 rows
 * of activations per output tile (256 columns).  Host-only; launches nothing.
 * Errors: JQ_ERR_INVALID_ARG, JQ_ERR_UNSUPPORTED_SHAPE.
 */
jq_status jq_gemm_plan(int64_t M, int64_t N, int64_t K, int cus, int* tile_rows);

/*
 * The block shape the BF6 GEMM (jq_w4a4_f6_gemm, _linear, _gemm_i32) takes for
 * an M x K by K x N product on a device with `cus` compute units, for checking
 * and tuning: *waves = 8 (one 8-wave block per CU) or 4 (two 4-wave blocks per
 * CU), *tile_rows = the rows of activations per output tile (256 columns).
 * Host-only; launches nothing.
 * Errors: JQ_ERR_INVALID_ARG, JQ_ERR_UNSUPPORTED_SHAPE.
 */
jq_status jq_f6_gemm_plan(int64_t M, int64_t N, int64_t K, int cus, int* waves, int* tile_rows);

/*
 * ---------------------------------------------------------------------------
 * Group-wise W4A4 on the BF6 engine.
 *
 * The group-wise layer defined above (the same codes, scales [rows, K/G],
 * the fp32 group sum in k order and the epilogue), with the codes held as
 * BF6 operands: the matrix cores return each group's exact integer product
 * in fp32, so the result is bit-identical to jq_w4a4g_linear.  Weights:
 * jq_pack_weight_int4_group, then jq_int4_to_f6_weight on its codes; its
 * scales are used as they are.  Shapes and errors as for the group-wise
 * layer, plus the BF6 operand limits (each operand below 2 GiB).
 */

/*
 * Group-wise activation quantisation into the BF6 activation layout.
 *   x_bf16  in   [M,K] bf16, 16-byte aligned
 *   xf6     out  jq_f6_operand_bytes(M,K) bytes, 16-byte aligned
 *   scales  out  [M,K/G] fp32, 4-byte aligned
 * Errors: JQ_ERR_INVALID_ARG, JQ_ERR_UNSUPPORTED_SHAPE, JQ_ERR_MISALIGNED, JQ_ERR_HIP.
 */
jq_status jq_quantize_act_group_f6(const void* x_bf16, int64_t M, int64_t K, int64_t G,
                                   void* xf6, float* scales, void* stream);

/*
 * Bytes of device workspace jq_w4a4g_f6_linear needs: the BF6 activation
 * operand and its scales (4*M*K/G bytes), each rounded up to 256 bytes.
 * 0 for invalid sizes.
 */
size_t jq_w4a4g_f6_workspace_bytes(int64_t M, int64_t K, int64_t G);

/*
 * The whole group-wise W4A4 linear on the BF6 engine.
 *   wf6        in   BF6 weight operand (weight layout) of the group-packed codes
 *   w_scales   in   [N,K/G] fp32 from jq_pack_weight_int4_group
 *   workspace  at least jq_w4a4g_f6_workspace_bytes(M,K,G) bytes, 256-byte aligned
 *   other arguments as jq_w4a4g_linear
 * Errors: as jq_w4a4g_linear.
 */
jq_status jq_w4a4g_f6_linear(const void* x_bf16, int64_t M, int64_t K, int64_t G,
                             const void* wf6, const float* w_scales, int64_t N,
                             const void* bias_bf16, void* y_bf16,
                             void* workspace, size_t workspace_bytes, void* stream);

/*
 * Group GEMM + epilogue on a BF6 activation operand and its scales (from
 * jq_quantize_act_group_f6); other arguments as jq_w4a4g_f6_linear.
 * Errors: JQ_ERR_INVALID_ARG, JQ_ERR_UNSUPPORTED_SHAPE, JQ_ERR_MISALIGNED, JQ_ERR_HIP.
 */
jq_status jq_w4a4g_f6_gemm(const void* xf6, const float* scales, int64_t M, int64_t K, int64_t G,
                           const void* wf6, const float* w_scales, int64_t N,
                           const void* bias_bf16, void* y_bf16, void* stream);

/*
 * The fp32 group sum S[m,n] alone, for checking: the same kernel as
 * jq_w4a4g_f6_gemm storing S into s_f32 [M,N] (16-byte aligned).
 * Errors: as jq_w4a4g_f6_gemm.
 */
jq_status jq_w4a4g_f6_gemm_f32(const void* xf6, const float* scales, int64_t M, int64_t K, int64_t G,
                               const void* wf6, const float* w_scales, int64_t N, float* s_f32, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* JQ_H */
