// Ternary (1.58-bit) weight quantisation and 2-bit packing for gfx950.
//
// Ternary weights with INT4 activations is the W1.58A4 deployment setting of
// the paper (Sec. 4 result tables; appendix experimental-details tables,
// "Ternary weights, INT4 activations").  The paper states no formula for the
// weight quantiser; the library uses the absmean reading, one scale per output
// channel (row n of W [N,K]):
//
//   g[n]   = fl32(fl64(sum_k |w[n,k]|) / K)      (fp64 sum and division, RNE to fp32)
//   t[n,k] = clamp(rne(fl32(w[n,k] / g[n])), -1, 1),  t = 0 when g = 0
//
// Packing: byte j of a row holds codes 4j .. 4j+3, code 4j+i in bits
// 2i .. 2i+1 as a two's-complement 2-bit field (0 -> 00, 1 -> 01, -1 -> 11).
//
// The fp64 sum is exact, and so independent of the order the block adds in,
// whenever a row's nonzero magnitudes span less than 2^29 (8 significant bits
// per bf16 value plus at most 16 bits of growth for K <= 65536 fit the 53-bit
// significand).  This runs once per layer when a model is loaded.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "jq_internal.h"

namespace jq {

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xFFFF0000u); }

__device__ __forceinline__ double abs_sum8(uint4 v) {
  return static_cast<double>(fabsf(bf16_lo(v.x))) + static_cast<double>(fabsf(bf16_hi(v.x))) +
         static_cast<double>(fabsf(bf16_lo(v.y))) + static_cast<double>(fabsf(bf16_hi(v.y))) +
         static_cast<double>(fabsf(bf16_lo(v.z))) + static_cast<double>(fabsf(bf16_hi(v.z))) +
         static_cast<double>(fabsf(bf16_lo(v.w))) + static_cast<double>(fabsf(bf16_hi(v.w)));
}

// Code of one element as a 2-bit field: rne(w / g) (IEEE division) clamped to [-1, 1].
__device__ __forceinline__ uint32_t tcode(float w, float g) {
  float q = rintf(w / g);
  q = fminf(fmaxf(q, -1.0f), 1.0f);
  return static_cast<uint32_t>(static_cast<int>(q)) & 3u;
}

__device__ __forceinline__ uint32_t pack8(uint4 v, float g) {
  return tcode(bf16_lo(v.x), g) | (tcode(bf16_hi(v.x), g) << 2) | (tcode(bf16_lo(v.y), g) << 4) |
         (tcode(bf16_hi(v.y), g) << 6) | (tcode(bf16_lo(v.z), g) << 8) | (tcode(bf16_hi(v.z), g) << 10) |
         (tcode(bf16_lo(v.w), g) << 12) | (tcode(bf16_hi(v.w), g) << 14);
}

// One block per row.  Pass 1: fp64 sum of |w| (each thread 8 elements per
// 16-byte load), reduced over the block.  Pass 2: 16 codes per thread per
// step, written as one 32-bit word (4 packed bytes).
__global__ __launch_bounds__(kThreads) void ternary_rows_kernel(const uint16_t* __restrict__ w, int64_t K,
                                                                uint8_t* __restrict__ t, float* __restrict__ g) {
  __shared__ double partial[kThreads / 64];
  const int64_t row = blockIdx.x;
  const uint16_t* wr = w + row * K;
  const int tid = threadIdx.x;

  double s = 0.0;
  for (int64_t k = 8 * static_cast<int64_t>(tid); k < K; k += 8 * kThreads)
    s += abs_sum8(*reinterpret_cast<const uint4*>(wr + k));
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off);
  if ((tid & 63) == 0) partial[tid >> 6] = s;
  __syncthreads();
  double total = 0.0;
#pragma unroll
  for (int i = 0; i < kThreads / 64; ++i) total += partial[i];
  const float gs = static_cast<float>(total / static_cast<double>(K));
  if (tid == 0) g[row] = gs;

  uint32_t* tr = reinterpret_cast<uint32_t*>(t + row * (K / 4));
  for (int64_t j = tid; j < K / 16; j += kThreads) {
    uint32_t word = 0;
    if (gs != 0.0f) {
      const uint4* src = reinterpret_cast<const uint4*>(wr + 16 * j);
      word = pack8(src[0], gs) | (pack8(src[1], gs) << 16);
    }
    tr[j] = word;
  }
}

}  // namespace

hipError_t launch_ternary_rows(const uint16_t* w, int64_t N, int64_t K, uint8_t* t, float* g, hipStream_t st) {
  hipLaunchKernelGGL(ternary_rows_kernel, dim3(static_cast<unsigned>(N)), dim3(kThreads), 0, st, w, K, t, g);
  return hipGetLastError();
}

}  // namespace jq
