// C ABI of libjq: argument checks, workspace layout and kernel launches.
// Every check runs before any launch, so a rejected call writes nothing.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "jq.h"
#include "jq_internal.h"

namespace {

constexpr size_t kWsAlign = 256;

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Shape checks shared by every entry point: rows >= 1, 64 <= K <= kMaxK, K % 64 == 0.
jq_status check_shape(int64_t rows, int64_t K) {
  if (rows <= 0 || K <= 0) return JQ_ERR_INVALID_ARG;
  if (rows > jq::kMaxRows) return JQ_ERR_UNSUPPORTED_SHAPE;
  if (K < 64 || K % 64 != 0 || K > jq::kMaxK) return JQ_ERR_UNSUPPORTED_SHAPE;
  return JQ_OK;
}

jq_status from_hip(hipError_t e) { return e == hipSuccess ? JQ_OK : JQ_ERR_HIP; }

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

jq_status quantize_common(const void* x, int64_t rows, int64_t K, void* q, float* scale, void* stream) {
  if (x == nullptr || q == nullptr || scale == nullptr) return JQ_ERR_INVALID_ARG;
  const jq_status st = check_shape(rows, K);
  if (st != JQ_OK) return st;
  if (!aligned(x, 16) || !aligned(q, 16) || !aligned(scale, 4)) return JQ_ERR_MISALIGNED;
  return from_hip(jq::launch_quantize_rows(static_cast<const uint16_t*>(x), rows, K,
                                           static_cast<uint8_t*>(q), scale, as_stream(stream)));
}

jq_status check_gemm(const void* qx, const float* sx, int64_t M, int64_t K, const void* qw,
                     const float* sw, int64_t N, const void* bias, const void* y, bool need_scales,
                     jq::WeightFormat wf = jq::WeightFormat::kInt4) {
  if (qx == nullptr || qw == nullptr || y == nullptr) return JQ_ERR_INVALID_ARG;
  if (need_scales && (sx == nullptr || sw == nullptr)) return JQ_ERR_INVALID_ARG;
  jq_status st = check_shape(M, K);
  if (st != JQ_OK) return st;
  st = check_shape(N, K);
  if (st != JQ_OK) return st;
  // The tile grid is indexed with 32-bit integers, and each packed operand is
  // addressed through a buffer descriptor with a 31-bit size.
  if (((M + 255) / 256) * ((N + 255) / 256) > (int64_t(1) << 26)) return JQ_ERR_UNSUPPORTED_SHAPE;
  const int64_t wrow = wf == jq::WeightFormat::kTernary ? K / 4 : K / 2;
  if (M * (K / 2) >= (int64_t(1) << 31) || N * wrow >= (int64_t(1) << 31)) return JQ_ERR_UNSUPPORTED_SHAPE;
  if (!aligned(qx, 16) || !aligned(qw, 16) || !aligned(y, 16)) return JQ_ERR_MISALIGNED;
  if ((sx != nullptr && !aligned(sx, 4)) || (sw != nullptr && !aligned(sw, 4))) return JQ_ERR_MISALIGNED;
  if (bias != nullptr && !aligned(bias, 2)) return JQ_ERR_MISALIGNED;
  return JQ_OK;
}

size_t workspace_bytes(int64_t M, int64_t K) {
  if (check_shape(M, K) != JQ_OK) return 0;
  return round_up(static_cast<size_t>(M) * static_cast<size_t>(K / 2), kWsAlign) +
         round_up(static_cast<size_t>(M) * sizeof(float), kWsAlign);
}

// Quantise x into the workspace, then the GEMM with the fused epilogue.
jq_status linear_common(const void* x_bf16, int64_t M, int64_t K, const void* w_packed, const float* w_scale,
                        int64_t N, const void* bias_bf16, void* y_bf16, void* workspace, size_t ws_bytes,
                        void* stream, jq::WeightFormat wf) {
  if (x_bf16 == nullptr || workspace == nullptr) return JQ_ERR_INVALID_ARG;
  jq_status st = check_gemm(x_bf16, w_scale, M, K, w_packed, w_scale, N, bias_bf16, y_bf16, true, wf);
  if (st != JQ_OK) return st;
  if (!aligned(workspace, kWsAlign)) return JQ_ERR_MISALIGNED;
  if (ws_bytes < workspace_bytes(M, K)) return JQ_ERR_WORKSPACE_TOO_SMALL;

  uint8_t* qx = static_cast<uint8_t*>(workspace);
  float* sx = reinterpret_cast<float*>(qx + round_up(static_cast<size_t>(M) * static_cast<size_t>(K / 2), kWsAlign));
  hipError_t e = jq::launch_quantize_rows(static_cast<const uint16_t*>(x_bf16), M, K, qx, sx,
                                          as_stream(stream));
  if (e != hipSuccess) return JQ_ERR_HIP;
  e = jq::launch_w4a4_gemm(jq::Epilogue::kBf16, qx, sx, M, K, static_cast<const uint8_t*>(w_packed), w_scale, N,
                           static_cast<const uint16_t*>(bias_bf16), y_bf16, as_stream(stream), wf);
  return from_hip(e);
}

jq_status gemm_common(const void* q_packed, const float* scale, int64_t M, int64_t K, const void* w_packed,
                      const float* w_scale, int64_t N, const void* bias_bf16, void* y_bf16, void* stream,
                      jq::WeightFormat wf) {
  const jq_status st = check_gemm(q_packed, scale, M, K, w_packed, w_scale, N, bias_bf16, y_bf16, true, wf);
  if (st != JQ_OK) return st;
  return from_hip(jq::launch_w4a4_gemm(jq::Epilogue::kBf16, static_cast<const uint8_t*>(q_packed), scale, M, K,
                                       static_cast<const uint8_t*>(w_packed), w_scale, N,
                                       static_cast<const uint16_t*>(bias_bf16), y_bf16, as_stream(stream), wf));
}

jq_status gemm_i32_common(const void* q_packed, int64_t M, int64_t K, const void* w_packed, int64_t N,
                          int32_t* acc, void* stream, jq::WeightFormat wf) {
  const jq_status st = check_gemm(q_packed, nullptr, M, K, w_packed, nullptr, N, nullptr, acc, false, wf);
  if (st != JQ_OK) return st;
  return from_hip(jq::launch_w4a4_gemm(jq::Epilogue::kInt32, static_cast<const uint8_t*>(q_packed), nullptr, M,
                                       K, static_cast<const uint8_t*>(w_packed), nullptr, N, nullptr, acc,
                                       as_stream(stream), wf));
}

}  // namespace

extern "C" {

const char* jq_status_string(jq_status s) {
  switch (s) {
    case JQ_OK: return "JQ_OK";
    case JQ_ERR_INVALID_ARG: return "JQ_ERR_INVALID_ARG";
    case JQ_ERR_UNSUPPORTED_SHAPE: return "JQ_ERR_UNSUPPORTED_SHAPE";
    case JQ_ERR_MISALIGNED: return "JQ_ERR_MISALIGNED";
    case JQ_ERR_WORKSPACE_TOO_SMALL: return "JQ_ERR_WORKSPACE_TOO_SMALL";
    case JQ_ERR_HIP: return "JQ_ERR_HIP";
  }
  return "JQ_ERR_UNKNOWN";
}

int jq_version(void) { return 100; }

jq_status jq_quantize_act(const void* x_bf16, int64_t M, int64_t K, void* q_packed, float* scale,
                          void* stream) {
  return quantize_common(x_bf16, M, K, q_packed, scale, stream);
}

jq_status jq_pack_weight_int4(const void* w_bf16, int64_t N, int64_t K, void* wq_packed,
                              float* w_scale, void* stream) {
  return quantize_common(w_bf16, N, K, wq_packed, w_scale, stream);
}

size_t jq_w4a4_workspace_bytes(int64_t M, int64_t K) { return workspace_bytes(M, K); }

jq_status jq_w4a4_linear(const void* x_bf16, int64_t M, int64_t K, const void* wq_packed,
                         const float* w_scale, int64_t N, const void* bias_bf16, void* y_bf16,
                         void* workspace, size_t workspace_bytes, void* stream) {
  return linear_common(x_bf16, M, K, wq_packed, w_scale, N, bias_bf16, y_bf16, workspace, workspace_bytes, stream,
                       jq::WeightFormat::kInt4);
}

jq_status jq_w4a4_gemm(const void* q_packed, const float* scale, int64_t M, int64_t K,
                       const void* wq_packed, const float* w_scale, int64_t N, const void* bias_bf16,
                       void* y_bf16, void* stream) {
  return gemm_common(q_packed, scale, M, K, wq_packed, w_scale, N, bias_bf16, y_bf16, stream,
                     jq::WeightFormat::kInt4);
}

jq_status jq_w4a4_gemm_i32(const void* q_packed, int64_t M, int64_t K, const void* wq_packed, int64_t N,
                           int32_t* acc, void* stream) {
  return gemm_i32_common(q_packed, M, K, wq_packed, N, acc, stream, jq::WeightFormat::kInt4);
}

jq_status jq_pack_weight_ternary(const void* w_bf16, int64_t N, int64_t K, void* wt_packed, float* w_scale,
                                 void* stream) {
  if (w_bf16 == nullptr || wt_packed == nullptr || w_scale == nullptr) return JQ_ERR_INVALID_ARG;
  const jq_status st = check_shape(N, K);
  if (st != JQ_OK) return st;
  if (!aligned(w_bf16, 16) || !aligned(wt_packed, 16) || !aligned(w_scale, 4)) return JQ_ERR_MISALIGNED;
  return from_hip(jq::launch_ternary_rows(static_cast<const uint16_t*>(w_bf16), N, K,
                                          static_cast<uint8_t*>(wt_packed), w_scale, as_stream(stream)));
}

jq_status jq_w158a4_linear(const void* x_bf16, int64_t M, int64_t K, const void* wt_packed,
                           const float* w_scale, int64_t N, const void* bias_bf16, void* y_bf16,
                           void* workspace, size_t workspace_bytes, void* stream) {
  return linear_common(x_bf16, M, K, wt_packed, w_scale, N, bias_bf16, y_bf16, workspace, workspace_bytes, stream,
                       jq::WeightFormat::kTernary);
}

jq_status jq_w158a4_gemm(const void* q_packed, const float* scale, int64_t M, int64_t K,
                         const void* wt_packed, const float* w_scale, int64_t N, const void* bias_bf16,
                         void* y_bf16, void* stream) {
  return gemm_common(q_packed, scale, M, K, wt_packed, w_scale, N, bias_bf16, y_bf16, stream,
                     jq::WeightFormat::kTernary);
}

jq_status jq_w158a4_gemm_i32(const void* q_packed, int64_t M, int64_t K, const void* wt_packed, int64_t N,
                             int32_t* acc, void* stream) {
  return gemm_i32_common(q_packed, M, K, wt_packed, N, acc, stream, jq::WeightFormat::kTernary);
}


// ---------------------------------------------------------------------------
// group-wise W4A4

}  // extern "C"

namespace {

jq_status check_group(int64_t rows, int64_t K, int64_t G) {
  const jq_status st = check_shape(rows, K);
  if (st != JQ_OK) return st;
  if ((G != 64 && G != 128) || K % G != 0) return JQ_ERR_UNSUPPORTED_SHAPE;
  return JQ_OK;
}

jq_status quantize_group_common(const void* x, int64_t rows, int64_t K, int64_t G, void* q, float* scales,
                                void* stream) {
  if (x == nullptr || q == nullptr || scales == nullptr) return JQ_ERR_INVALID_ARG;
  const jq_status st = check_group(rows, K, G);
  if (st != JQ_OK) return st;
  if (rows * K > (int64_t(1) << 41)) return JQ_ERR_UNSUPPORTED_SHAPE;  // the grid counts 2048-element blocks
  if (!aligned(x, 16) || !aligned(q, 16) || !aligned(scales, 4)) return JQ_ERR_MISALIGNED;
  return from_hip(jq::launch_quantize_groups(static_cast<const uint16_t*>(x), rows, K, static_cast<int>(G),
                                             static_cast<uint8_t*>(q), scales, as_stream(stream)));
}

jq_status check_group_gemm(const void* qx, const float* sx, int64_t M, int64_t K, int64_t G, const void* qw,
                           const float* sw, int64_t N, const void* bias, const void* y) {
  if (qx == nullptr || qw == nullptr || y == nullptr || sx == nullptr || sw == nullptr) return JQ_ERR_INVALID_ARG;
  jq_status st = check_group(M, K, G);
  if (st != JQ_OK) return st;
  st = check_group(N, K, G);
  if (st != JQ_OK) return st;
  // 32-bit tile indices; 31-bit buffer descriptors over the codes and scales.
  if (((M + 127) / 128) * ((N + 127) / 128) > (int64_t(1) << 26)) return JQ_ERR_UNSUPPORTED_SHAPE;
  if (M * (K / 2) >= (int64_t(1) << 31) || N * (K / 2) >= (int64_t(1) << 31)) return JQ_ERR_UNSUPPORTED_SHAPE;
  if (!aligned(qx, 16) || !aligned(qw, 16) || !aligned(y, 16)) return JQ_ERR_MISALIGNED;
  if (!aligned(sx, 4) || !aligned(sw, 4)) return JQ_ERR_MISALIGNED;
  if (bias != nullptr && !aligned(bias, 2)) return JQ_ERR_MISALIGNED;
  return JQ_OK;
}

size_t group_workspace_bytes(int64_t M, int64_t K, int64_t G) {
  if (check_group(M, K, G) != JQ_OK) return 0;
  return round_up(static_cast<size_t>(M) * static_cast<size_t>(K / 2), kWsAlign) +
         round_up(static_cast<size_t>(M) * static_cast<size_t>(K / G) * sizeof(float), kWsAlign);
}

}  // namespace

extern "C" {

jq_status jq_quantize_act_group(const void* x_bf16, int64_t M, int64_t K, int64_t G, void* q_packed, float* scales,
                                void* stream) {
  return quantize_group_common(x_bf16, M, K, G, q_packed, scales, stream);
}

jq_status jq_pack_weight_int4_group(const void* w_bf16, int64_t N, int64_t K, int64_t G, void* wq_packed,
                                    float* w_scales, void* stream) {
  return quantize_group_common(w_bf16, N, K, G, wq_packed, w_scales, stream);
}

size_t jq_w4a4g_workspace_bytes(int64_t M, int64_t K, int64_t G) { return group_workspace_bytes(M, K, G); }

jq_status jq_w4a4g_linear(const void* x_bf16, int64_t M, int64_t K, int64_t G, const void* wq_packed,
                          const float* w_scales, int64_t N, const void* bias_bf16, void* y_bf16, void* workspace,
                          size_t workspace_bytes, void* stream) {
  if (x_bf16 == nullptr || workspace == nullptr) return JQ_ERR_INVALID_ARG;
  // the activation operands live in the workspace; check the rest with stand-ins
  jq_status st = check_group_gemm(x_bf16, w_scales, M, K, G, wq_packed, w_scales, N, bias_bf16, y_bf16);
  if (st != JQ_OK) return st;
  if (!aligned(workspace, kWsAlign)) return JQ_ERR_MISALIGNED;
  if (workspace_bytes < group_workspace_bytes(M, K, G)) return JQ_ERR_WORKSPACE_TOO_SMALL;
  uint8_t* qx = static_cast<uint8_t*>(workspace);
  float* sx = reinterpret_cast<float*>(qx + round_up(static_cast<size_t>(M) * static_cast<size_t>(K / 2), kWsAlign));
  hipError_t e = jq::launch_quantize_groups(static_cast<const uint16_t*>(x_bf16), M, K, static_cast<int>(G), qx, sx,
                                            as_stream(stream));
  if (e != hipSuccess) return JQ_ERR_HIP;
  e = jq::launch_w4a4g_gemm(jq::Epilogue::kBf16, qx, sx, M, K, static_cast<int>(G),
                            static_cast<const uint8_t*>(wq_packed), w_scales, N,
                            static_cast<const uint16_t*>(bias_bf16), y_bf16, as_stream(stream));
  return from_hip(e);
}

jq_status jq_w4a4g_gemm(const void* q_packed, const float* scales, int64_t M, int64_t K, int64_t G,
                        const void* wq_packed, const float* w_scales, int64_t N, const void* bias_bf16, void* y_bf16,
                        void* stream) {
  const jq_status st = check_group_gemm(q_packed, scales, M, K, G, wq_packed, w_scales, N, bias_bf16, y_bf16);
  if (st != JQ_OK) return st;
  return from_hip(jq::launch_w4a4g_gemm(jq::Epilogue::kBf16, static_cast<const uint8_t*>(q_packed), scales, M, K,
                                        static_cast<int>(G), static_cast<const uint8_t*>(wq_packed), w_scales, N,
                                        static_cast<const uint16_t*>(bias_bf16), y_bf16, as_stream(stream)));
}

jq_status jq_w4a4g_gemm_f32(const void* q_packed, const float* scales, int64_t M, int64_t K, int64_t G,
                            const void* wq_packed, const float* w_scales, int64_t N, float* s_f32, void* stream) {
  const jq_status st = check_group_gemm(q_packed, scales, M, K, G, wq_packed, w_scales, N, nullptr, s_f32);
  if (st != JQ_OK) return st;
  return from_hip(jq::launch_w4a4g_gemm(jq::Epilogue::kF32, static_cast<const uint8_t*>(q_packed), scales, M, K,
                                        static_cast<int>(G), static_cast<const uint8_t*>(wq_packed), w_scales, N,
                                        nullptr, s_f32, as_stream(stream)));
}

}  // extern "C"

// ---------------------------------------------------------------------------
// BF6 engine: the same layer on the 6-bit matrix cores

namespace {

jq_status check_f6_operands(int64_t M, int64_t N, int64_t K) {
  jq_status st = check_shape(M, K);
  if (st != JQ_OK) return st;
  st = check_shape(N, K);
  if (st != JQ_OK) return st;
  // 32-bit tile indices; 31-bit buffer descriptors over both operands.
  if (((M + 255) / 256) * ((N + 255) / 256) > (int64_t(1) << 26)) return JQ_ERR_UNSUPPORTED_SHAPE;
  if (jq::f6_operand_bytes(M, K) >= (int64_t(1) << 31) || jq::f6_operand_bytes(N, K) >= (int64_t(1) << 31))
    return JQ_ERR_UNSUPPORTED_SHAPE;
  return JQ_OK;
}

jq_status check_f6_gemm(const void* xf6, const float* sx, int64_t M, int64_t K, const void* wf6, const float* sw,
                        int64_t N, const void* bias, const void* y, bool need_scales) {
  if (xf6 == nullptr || wf6 == nullptr || y == nullptr) return JQ_ERR_INVALID_ARG;
  if (need_scales && (sx == nullptr || sw == nullptr)) return JQ_ERR_INVALID_ARG;
  const jq_status st = check_f6_operands(M, N, K);
  if (st != JQ_OK) return st;
  if (!aligned(xf6, 16) || !aligned(wf6, 16) || !aligned(y, 16)) return JQ_ERR_MISALIGNED;
  if ((sx != nullptr && !aligned(sx, 4)) || (sw != nullptr && !aligned(sw, 4))) return JQ_ERR_MISALIGNED;
  if (bias != nullptr && !aligned(bias, 2)) return JQ_ERR_MISALIGNED;
  return JQ_OK;
}

size_t f6_workspace_bytes(int64_t M, int64_t K) {
  if (check_shape(M, K) != JQ_OK) return 0;
  return round_up(static_cast<size_t>(jq::f6_operand_bytes(M, K)), kWsAlign) +
         round_up(static_cast<size_t>(M) * sizeof(float), kWsAlign);
}

// Quantise x into a checked workspace (BF6 operand, then scales), then the
// GEMM with the fused epilogue.
jq_status f6_linear_launch(const void* x_bf16, int64_t M, int64_t K, const void* wf6, const float* w_scale,
                           int64_t N, const void* bias_bf16, void* y_bf16, void* workspace, void* stream) {
  uint8_t* xf6 = static_cast<uint8_t*>(workspace);
  float* sx = reinterpret_cast<float*>(xf6 + round_up(static_cast<size_t>(jq::f6_operand_bytes(M, K)), kWsAlign));
  hipError_t e = jq::launch_quantize_rows_f6(static_cast<const uint16_t*>(x_bf16), M, K, xf6, sx,
                                             as_stream(stream));
  if (e != hipSuccess) return JQ_ERR_HIP;
  e = jq::launch_w4a4_f6_gemm(jq::Epilogue::kBf16, xf6, sx, M, K, static_cast<const uint8_t*>(wf6), w_scale, N,
                              static_cast<const uint16_t*>(bias_bf16), y_bf16, as_stream(stream));
  return from_hip(e);
}

jq_status check_group_f6_gemm(const void* xf6, const float* sx, int64_t M, int64_t K, int64_t G, const void* wf6,
                              const float* sw, int64_t N, const void* bias, const void* y) {
  if (xf6 == nullptr || wf6 == nullptr || y == nullptr || sx == nullptr || sw == nullptr) return JQ_ERR_INVALID_ARG;
  jq_status st = check_group(M, K, G);
  if (st != JQ_OK) return st;
  st = check_group(N, K, G);
  if (st != JQ_OK) return st;
  st = check_f6_operands(M, N, K);
  if (st != JQ_OK) return st;
  // 32-bit tile indices over 128 x 128 tiles
  if (((M + 127) / 128) * ((N + 127) / 128) > (int64_t(1) << 26)) return JQ_ERR_UNSUPPORTED_SHAPE;
  if (!aligned(xf6, 16) || !aligned(wf6, 16) || !aligned(y, 16)) return JQ_ERR_MISALIGNED;
  if (!aligned(sx, 4) || !aligned(sw, 4)) return JQ_ERR_MISALIGNED;
  if (bias != nullptr && !aligned(bias, 2)) return JQ_ERR_MISALIGNED;
  return JQ_OK;
}

size_t group_f6_workspace_bytes(int64_t M, int64_t K, int64_t G) {
  if (check_group(M, K, G) != JQ_OK) return 0;
  return round_up(static_cast<size_t>(jq::f6_operand_bytes(M, K)), kWsAlign) +
         round_up(static_cast<size_t>(M) * static_cast<size_t>(K / G) * sizeof(float), kWsAlign);
}

}  // namespace

extern "C" {

size_t jq_f6_operand_bytes(int64_t rows, int64_t K) {
  if (check_shape(rows, K) != JQ_OK) return 0;
  return static_cast<size_t>(jq::f6_operand_bytes(rows, K));
}

jq_status jq_quantize_act_f6(const void* x_bf16, int64_t M, int64_t K, void* xf6, float* scale, void* stream) {
  if (x_bf16 == nullptr || xf6 == nullptr || scale == nullptr) return JQ_ERR_INVALID_ARG;
  const jq_status st = check_shape(M, K);
  if (st != JQ_OK) return st;
  if (!aligned(x_bf16, 16) || !aligned(xf6, 16) || !aligned(scale, 4)) return JQ_ERR_MISALIGNED;
  return from_hip(jq::launch_quantize_rows_f6(static_cast<const uint16_t*>(x_bf16), M, K,
                                              static_cast<uint8_t*>(xf6), scale, as_stream(stream)));
}

jq_status jq_quantize_act_f6_batch(int count, const void* const* x_bf16, const int64_t* M, const int64_t* K,
                                   void* const* xf6, float* const* scale, void* stream) {
  if (count < 1 || count > JQ_QUANT_BATCH_MAX) return JQ_ERR_INVALID_ARG;
  if (x_bf16 == nullptr || M == nullptr || K == nullptr || xf6 == nullptr || scale == nullptr)
    return JQ_ERR_INVALID_ARG;
  for (int i = 0; i < count; ++i) {
    if (x_bf16[i] == nullptr || xf6[i] == nullptr || scale[i] == nullptr) return JQ_ERR_INVALID_ARG;
    const jq_status st = check_shape(M[i], K[i]);
    if (st != JQ_OK) return st;
    if (!aligned(x_bf16[i], 16) || !aligned(xf6[i], 16) || !aligned(scale[i], 4)) return JQ_ERR_MISALIGNED;
  }
  const uint16_t* xs[JQ_QUANT_BATCH_MAX];
  uint8_t* outs[JQ_QUANT_BATCH_MAX];
  for (int i = 0; i < count; ++i) {
    xs[i] = static_cast<const uint16_t*>(x_bf16[i]);
    outs[i] = static_cast<uint8_t*>(xf6[i]);
  }
  return from_hip(jq::launch_quantize_rows_f6_batch(count, xs, M, K, outs, scale, as_stream(stream)));
}

jq_status jq_int4_to_f6(const void* q_packed, int64_t rows, int64_t K, void* f6, void* stream) {
  if (q_packed == nullptr || f6 == nullptr) return JQ_ERR_INVALID_ARG;
  const jq_status st = check_shape(rows, K);
  if (st != JQ_OK) return st;
  if (!aligned(q_packed, 16) || !aligned(f6, 16)) return JQ_ERR_MISALIGNED;
  return from_hip(jq::launch_int4_to_f6(static_cast<const uint8_t*>(q_packed), rows, K, static_cast<uint8_t*>(f6),
                                        false, false, as_stream(stream)));
}

jq_status jq_int4_to_f6_weight(const void* q_packed, int64_t rows, int64_t K, void* wf6, void* stream) {
  if (q_packed == nullptr || wf6 == nullptr) return JQ_ERR_INVALID_ARG;
  const jq_status st = check_shape(rows, K);
  if (st != JQ_OK) return st;
  if (!aligned(q_packed, 16) || !aligned(wf6, 16)) return JQ_ERR_MISALIGNED;
  return from_hip(jq::launch_int4_to_f6(static_cast<const uint8_t*>(q_packed), rows, K, static_cast<uint8_t*>(wf6),
                                        true, false, as_stream(stream)));
}

jq_status jq_ternary_to_f6_weight(const void* wt_packed, int64_t rows, int64_t K, void* wf6, void* stream) {
  if (wt_packed == nullptr || wf6 == nullptr) return JQ_ERR_INVALID_ARG;
  const jq_status st = check_shape(rows, K);
  if (st != JQ_OK) return st;
  if (!aligned(wt_packed, 16) || !aligned(wf6, 16)) return JQ_ERR_MISALIGNED;
  return from_hip(jq::launch_int4_to_f6(static_cast<const uint8_t*>(wt_packed), rows, K, static_cast<uint8_t*>(wf6),
                                        true, true, as_stream(stream)));
}

size_t jq_w4a4_f6_workspace_bytes(int64_t M, int64_t K) { return f6_workspace_bytes(M, K); }

jq_status jq_w4a4_f6_linear(const void* x_bf16, int64_t M, int64_t K, const void* wf6, const float* w_scale,
                            int64_t N, const void* bias_bf16, void* y_bf16, void* workspace,
                            size_t workspace_bytes, void* stream) {
  if (x_bf16 == nullptr || workspace == nullptr) return JQ_ERR_INVALID_ARG;
  // the activation operand lives in the workspace; check the rest with stand-ins
  const jq_status st = check_f6_gemm(x_bf16, w_scale, M, K, wf6, w_scale, N, bias_bf16, y_bf16, true);
  if (st != JQ_OK) return st;
  if (!aligned(workspace, kWsAlign)) return JQ_ERR_MISALIGNED;
  if (workspace_bytes < f6_workspace_bytes(M, K)) return JQ_ERR_WORKSPACE_TOO_SMALL;
  return f6_linear_launch(x_bf16, M, K, wf6, w_scale, N, bias_bf16, y_bf16, workspace, stream);
}

jq_status jq_w4a4_f6_linear_noalloc(const void* x_bf16, int64_t M, int64_t K, const void* wf6,
                                    const float* w_scale, int64_t N, const void* bias_bf16, void* y_bf16,
                                    void* stream) {
  if (x_bf16 == nullptr) return JQ_ERR_INVALID_ARG;
  // the activation operand lives in the library's scratch; check the rest with stand-ins
  const jq_status st = check_f6_gemm(x_bf16, w_scale, M, K, wf6, w_scale, N, bias_bf16, y_bf16, true);
  if (st != JQ_OK) return st;
  if (f6_workspace_bytes(M, K) > JQ_NOALLOC_SCRATCH_BYTES) return JQ_ERR_WORKSPACE_TOO_SMALL;
  void* scratch = nullptr;
  if (jq::noalloc_scratch(&scratch) != hipSuccess) return JQ_ERR_HIP;
  return f6_linear_launch(x_bf16, M, K, wf6, w_scale, N, bias_bf16, y_bf16, scratch, stream);
}

jq_status jq_w4a4_f6_gemm(const void* xf6, const float* scale, int64_t M, int64_t K, const void* wf6,
                          const float* w_scale, int64_t N, const void* bias_bf16, void* y_bf16, void* stream) {
  const jq_status st = check_f6_gemm(xf6, scale, M, K, wf6, w_scale, N, bias_bf16, y_bf16, true);
  if (st != JQ_OK) return st;
  return from_hip(jq::launch_w4a4_f6_gemm(jq::Epilogue::kBf16, static_cast<const uint8_t*>(xf6), scale, M, K,
                                          static_cast<const uint8_t*>(wf6), w_scale, N,
                                          static_cast<const uint16_t*>(bias_bf16), y_bf16, as_stream(stream)));
}

jq_status jq_w4a4_f6_gemm_i32(const void* xf6, int64_t M, int64_t K, const void* wf6, int64_t N, int32_t* acc,
                              void* stream) {
  const jq_status st = check_f6_gemm(xf6, nullptr, M, K, wf6, nullptr, N, nullptr, acc, false);
  if (st != JQ_OK) return st;
  return from_hip(jq::launch_w4a4_f6_gemm(jq::Epilogue::kInt32, static_cast<const uint8_t*>(xf6), nullptr, M, K,
                                          static_cast<const uint8_t*>(wf6), nullptr, N, nullptr, acc,
                                          as_stream(stream)));
}


jq_status jq_quantize_act_group_f6(const void* x_bf16, int64_t M, int64_t K, int64_t G, void* xf6, float* scales,
                                   void* stream) {
  if (x_bf16 == nullptr || xf6 == nullptr || scales == nullptr) return JQ_ERR_INVALID_ARG;
  const jq_status st = check_group(M, K, G);
  if (st != JQ_OK) return st;
  if (!aligned(x_bf16, 16) || !aligned(xf6, 16) || !aligned(scales, 4)) return JQ_ERR_MISALIGNED;
  return from_hip(jq::launch_quantize_groups_f6(static_cast<const uint16_t*>(x_bf16), M, K, static_cast<int>(G),
                                                static_cast<uint8_t*>(xf6), scales, as_stream(stream)));
}

size_t jq_w4a4g_f6_workspace_bytes(int64_t M, int64_t K, int64_t G) { return group_f6_workspace_bytes(M, K, G); }

jq_status jq_w4a4g_f6_linear(const void* x_bf16, int64_t M, int64_t K, int64_t G, const void* wf6,
                             const float* w_scales, int64_t N, const void* bias_bf16, void* y_bf16, void* workspace,
                             size_t workspace_bytes, void* stream) {
  if (x_bf16 == nullptr || workspace == nullptr) return JQ_ERR_INVALID_ARG;
  // the activation operand lives in the workspace; check the rest with stand-ins
  const jq_status st = check_group_f6_gemm(x_bf16, w_scales, M, K, G, wf6, w_scales, N, bias_bf16, y_bf16);
  if (st != JQ_OK) return st;
  if (!aligned(workspace, kWsAlign)) return JQ_ERR_MISALIGNED;
  if (workspace_bytes < group_f6_workspace_bytes(M, K, G)) return JQ_ERR_WORKSPACE_TOO_SMALL;
  uint8_t* xf6 = static_cast<uint8_t*>(workspace);
  float* sx = reinterpret_cast<float*>(xf6 + round_up(static_cast<size_t>(jq::f6_operand_bytes(M, K)), kWsAlign));
  hipError_t e = jq::launch_quantize_groups_f6(static_cast<const uint16_t*>(x_bf16), M, K, static_cast<int>(G), xf6,
                                               sx, as_stream(stream));
  if (e != hipSuccess) return JQ_ERR_HIP;
  return from_hip(jq::launch_w4a4g_f6_gemm(jq::Epilogue::kBf16, xf6, sx, M, K, static_cast<int>(G),
                                           static_cast<const uint8_t*>(wf6), w_scales, N,
                                           static_cast<const uint16_t*>(bias_bf16), y_bf16, as_stream(stream)));
}

jq_status jq_w4a4g_f6_gemm(const void* xf6, const float* scales, int64_t M, int64_t K, int64_t G, const void* wf6,
                           const float* w_scales, int64_t N, const void* bias_bf16, void* y_bf16, void* stream) {
  const jq_status st = check_group_f6_gemm(xf6, scales, M, K, G, wf6, w_scales, N, bias_bf16, y_bf16);
  if (st != JQ_OK) return st;
  return from_hip(jq::launch_w4a4g_f6_gemm(jq::Epilogue::kBf16, static_cast<const uint8_t*>(xf6), scales, M, K,
                                           static_cast<int>(G), static_cast<const uint8_t*>(wf6), w_scales, N,
                                           static_cast<const uint16_t*>(bias_bf16), y_bf16, as_stream(stream)));
}

jq_status jq_w4a4g_f6_gemm_f32(const void* xf6, const float* scales, int64_t M, int64_t K, int64_t G,
                               const void* wf6, const float* w_scales, int64_t N, float* s_f32, void* stream) {
  const jq_status st = check_group_f6_gemm(xf6, scales, M, K, G, wf6, w_scales, N, nullptr, s_f32);
  if (st != JQ_OK) return st;
  return from_hip(jq::launch_w4a4g_f6_gemm(jq::Epilogue::kF32, static_cast<const uint8_t*>(xf6), scales, M, K,
                                           static_cast<int>(G), static_cast<const uint8_t*>(wf6), w_scales, N,
                                           nullptr, s_f32, as_stream(stream)));
}

jq_status jq_gemm_plan(int64_t M, int64_t N, int64_t K, int cus, int* tile_rows) {
  if (tile_rows == nullptr || cus < 1) return JQ_ERR_INVALID_ARG;
  jq_status st = check_shape(M, K);
  if (st != JQ_OK) return st;
  st = check_shape(N, K);
  if (st != JQ_OK) return st;
  *tile_rows = jq::gemm_tile_rows(M, N, 2 * std::max<int64_t>(8, cus / 8 * 8));
  return JQ_OK;
}

jq_status jq_f6_gemm_plan(int64_t M, int64_t N, int64_t K, int cus, int* waves, int* tile_rows) {
  if (waves == nullptr || tile_rows == nullptr || cus < 1) return JQ_ERR_INVALID_ARG;
  const jq_status st = check_f6_operands(M, N, K);
  if (st != JQ_OK) return st;
  const int64_t slots = std::max<int64_t>(8, cus / 8 * 8);
  *waves = jq::f6_block_waves(M, N, K, slots);
  *tile_rows = 32 * (*waves == 4 ? 4 : jq::f6_tile_bands(M, N, slots));
  return JQ_OK;
}

}  // extern "C"
