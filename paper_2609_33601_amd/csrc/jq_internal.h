// Internal launch interface between the C ABI layer and the gfx950 kernels.
#ifndef JQ_INTERNAL_H
#define JQ_INTERNAL_H

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace jq {

// Largest supported reduction length.  With codes in [-8, 7] the kernel's
// int8 operands are 16 * code, so its int32 accumulator holds 256 * acc with
// |256 * acc| <= 256 * 64 * K = 2^30 at K = 65536, and |acc| < 2^24 keeps the
// epilogue's int -> fp32 conversion exact.
constexpr int64_t kMaxK = 65536;
// Rows are addressed with 32-bit block indices.
constexpr int64_t kMaxRows = int64_t(1) << 30;

// Row quantiser: x [M,K] bf16 -> q [M,K/2] packed int4, scale [M] fp32.
hipError_t launch_quantize_rows(const uint16_t* x, int64_t M, int64_t K, uint8_t* q, float* scale,
                                hipStream_t st);

// Ternary weight quantiser: w [N,K] bf16 -> t [N,K/4] 2-bit codes, g [N] fp32.
hipError_t launch_ternary_rows(const uint16_t* w, int64_t N, int64_t K, uint8_t* t, float* g, hipStream_t st);

// Group-wise quantiser (G = 64 or 128): x [M,K] bf16 -> q [M,K/2], scale [M, K/G] fp32.
hipError_t launch_quantize_groups(const uint16_t* x, int64_t M, int64_t K, int G, uint8_t* q, float* scale,
                                  hipStream_t st);

// kBf16: bf16 output; kInt32: raw accumulators; kF32: the group kernel's fp32 sum before bias.
enum class Epilogue { kBf16, kInt32, kF32 };

// Weight operand of the GEMM: packed int4 [N,K/2] or packed ternary [N,K/4].
enum class WeightFormat { kInt4, kTernary };

// Packed low-bit GEMM: acc[m,n] = sum_k qx[m,k] * qw[n,k] followed by the epilogue.
//   kBf16:  y[m,n] = bf16(((fp32(acc) * sx[m]) * sw[n]) + bias[n])  (bias may be null)
//   kInt32: out[m,n] = acc
hipError_t launch_w4a4_gemm(Epilogue epi, const uint8_t* qx, const float* sx, int64_t M, int64_t K,
                            const uint8_t* qw, const float* sw, int64_t N, const uint16_t* bias,
                            void* out, hipStream_t st, WeightFormat wf = WeightFormat::kInt4);
// Its tile height (128 or 112 activation rows) for an M x N output with
// `slots` block slots (two per CU).
int gemm_tile_rows(int64_t M, int64_t N, int64_t slots);

// Group-wise GEMM: scales sx [M, K/G] and sw [N, K/G]; epi is kBf16 or kF32.
hipError_t launch_w4a4g_gemm(Epilogue epi, const uint8_t* qx, const float* sx, int64_t M, int64_t K, int G,
                             const uint8_t* qw, const float* sw, int64_t N, const uint16_t* bias, void* out,
                             hipStream_t st);

// BF6 engine (6-bit MFMA operands).  Activations and weights take
// f6_operand_bytes(rows, K) bytes each (rows padded to 32, K to 128), in the
// activation layout and the weight layout respectively.
int64_t f6_ksteps(int64_t K);
int64_t f6_operand_bytes(int64_t rows, int64_t K);
// GEMM block shape for an M x K by K x N product on `slots` CUs: 4 (two 4-wave
// blocks per CU) or 8 (one 8-wave block) waves.
int f6_block_waves(int64_t M, int64_t N, int64_t K, int64_t slots);
// GEMM tile height in bands of 32 rows (7 or 8) for an M x N output on `slots` CUs.
int f6_tile_bands(int64_t M, int64_t N, int64_t slots);

// Per-token quantiser writing the BF6 activation operand and the scales.
hipError_t launch_quantize_rows_f6(const uint16_t* x, int64_t M, int64_t K, uint8_t* out, float* scale,
                                   hipStream_t st);

// The per-token BF6 quantiser on `count` (<= 8) independent inputs at once
// (one launch for those with K <= 16384, one each for longer rows).
hipError_t launch_quantize_rows_f6_batch(int count, const uint16_t* const* x, const int64_t* M, const int64_t* K,
                                         uint8_t* const* out, float* const* scale, hipStream_t st);

// Group-wise BF6 engine (G = 64 or 128): the group quantiser writing the BF6
// activation operand and scales [M, K/G]; the group GEMM on BF6 operands with
// scales [M, K/G] and [N, K/G] (epi kBf16 or kF32).
hipError_t launch_quantize_groups_f6(const uint16_t* x, int64_t M, int64_t K, int G, uint8_t* out, float* scale,
                                     hipStream_t st);
hipError_t launch_w4a4g_f6_gemm(Epilogue epi, const uint8_t* xf6, const float* sx, int64_t M, int64_t K, int G,
                                const uint8_t* wf6, const float* sw, int64_t N, const uint16_t* bias, void* out,
                                hipStream_t st);

// Canonical packed int4 codes ([rows, K/2]) or packed ternary codes
// ([rows, K/4], `ternary`) -> BF6 operand in the activation layout or the
// weight layout (padding written as zeros).
hipError_t launch_int4_to_f6(const uint8_t* q, int64_t rows, int64_t K, uint8_t* out, bool weight_layout,
                             bool ternary, hipStream_t st);

// GEMM on BF6 operands (xf6 in the activation layout, wf6 in the weight
// layout); epi is kBf16 (y = bf16(((acc*sx)*sw)+bias)) or kInt32 (acc).
hipError_t launch_w4a4_f6_gemm(Epilogue epi, const uint8_t* xf6, const float* sx, int64_t M, int64_t K,
                               const uint8_t* wf6, const float* sw, int64_t N, const uint16_t* bias, void* out,
                               hipStream_t st);

// Device address of the library-held scratch (JQ_NOALLOC_SCRATCH_BYTES) on
// the current device, resolved once per device.
hipError_t noalloc_scratch(void** ptr);

}  // namespace jq

#endif  // JQ_INTERNAL_H
