// Per-row symmetric int4 quantiser and nibble packer for gfx950.
//
// Implements the activation/weight quantisation of the plain W4A4 linear
// (Sec. 3.1: every module becomes a low-bit operator of the deployment family;
// appendix FAQ Q7: quantisation and packing kernels; appendix experimental-
// details tables: INT4 weights and activations).  Per row r of a bf16 matrix:
//   a_r = max_k |x[r,k]|,  s_r = fl32(a_r / 7),
//   q[r,k] = clamp(rne(fl32(x[r,k] / s_r)), -8, 7)   (q = 0 when s_r = 0),
// packed two codes per byte, even k in the low nibble.
//
// Mapping: one wavefront per row.  Lane l owns elements [c*512 + 8l, +8) for
// chunk c = 0..NC-1, loaded with one 16-byte global load per chunk (a wave
// reads 1 KiB contiguous per chunk) and held in registers, so the row is read
// from HBM exactly once.  The absmax is a packed-u16 max over sign-cleared
// bf16 bits followed by a butterfly reduction across the wave.
//
// Exact quotient without a division per element.  With r = fl32(1/s) (one
// IEEE division per row) and t = fl32(x * r), both t and fl32(x/s) lie within
// 21 * 2^-24 < 2^-19.6 of x/s, because |x/s| <= 7.0004 for every finite bf16
// row (s is within one fp32 rounding of a/7, or within 2^-149 of it for the
// smallest subnormal rows).  Their rne() can therefore differ only when t is
// within 2^-19.6 of a half-integer.  Elements with |t - rne(t)| >= 1/2 - 2^-17
// are recomputed with the IEEE division; all others take rne(t), which then
// equals rne(fl32(x/s)) exactly.  Rows whose reciprocal overflows (s < 2^-128)
// use the division for every element.  The same bound shows |rne(t)| <= 7, so
// the clamp to [-8, 7] can only bind on the division path, where it is applied.
//
// rne(t) is taken with the float "magic number" 1.5 * 2^23: t + 1.5*2^23 is
// rounded to an integer by the fp32 adder (round-to-nearest-even), and the low
// byte of its bit pattern is rne(t) as an 8-bit two's complement value.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "jq_internal.h"

namespace jq {

namespace {

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

constexpr float kMagic = 12582912.0f;         // 1.5 * 2^23
constexpr float kNearTie = 0.5f - 0x1p-17f;   // |t - rne(t)| at or above this -> exact path

__device__ __forceinline__ float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }

// Exact code of one element by the definition: IEEE fp32 division, rne, clamp.
__device__ __forceinline__ uint32_t exact_nibble(float x, float s) {
  float t = __builtin_rintf(x / s);
  t = fminf(fmaxf(t, -8.0f), 7.0f);
  return static_cast<uint32_t>(static_cast<int>(t)) & 0xFu;
}

// Pack 8 elements (4 dwords of bf16 pairs) by the exact division path.
__device__ __forceinline__ uint32_t pack8_exact(uint4 v, float s) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  uint32_t out = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    out |= exact_nibble(bf16_lo(w[j]), s) << (8 * j);
    out |= exact_nibble(bf16_hi(w[j]), s) << (8 * j + 4);
  }
  return out;
}

// Pack 8 elements by the reciprocal path; sets *near if any element sits next
// to a rounding decision point and must be redone exactly.
__device__ __forceinline__ uint32_t pack8_fast(uint4 v, float rcp, bool* near) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  uint32_t ev[4], od[4];
  float dmax = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float te = bf16_lo(w[j]) * rcp;
    const float to = bf16_hi(w[j]) * rcp;
    const float me = te + kMagic;
    const float mo = to + kMagic;
    dmax = fmaxf(dmax, fmaxf(fabsf(te - (me - kMagic)), fabsf(to - (mo - kMagic))));
    ev[j] = __float_as_uint(me);
    od[j] = __float_as_uint(mo);
  }
  *near = !(dmax < kNearTie);
  // Gather the low bytes: e = [q0, q2, q4, q6], o = [q1, q3, q5, q7].
  const uint32_t e01 = __builtin_amdgcn_perm(ev[1], ev[0], 0x0C0C0400u);
  const uint32_t e23 = __builtin_amdgcn_perm(ev[3], ev[2], 0x0C0C0400u);
  const uint32_t o01 = __builtin_amdgcn_perm(od[1], od[0], 0x0C0C0400u);
  const uint32_t o23 = __builtin_amdgcn_perm(od[3], od[2], 0x0C0C0400u);
  const uint32_t e = __builtin_amdgcn_perm(e23, e01, 0x05040100u);
  const uint32_t o = __builtin_amdgcn_perm(o23, o01, 0x05040100u);
  // Byte j = (q_{2j} & 0xF) | (q_{2j+1} & 0xF) << 4.
  return (e & 0x0F0F0F0Fu) | ((o << 4) & 0xF0F0F0F0u);
}

typedef unsigned v4u32 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint32_t o = static_cast<uint32_t>(__shfl_xor(static_cast<int>(v), off, 64));
    v = v > o ? v : o;
  }
  return v;
}

// One block per row: W = blockDim.x / 64 waves share the row, wave w owning
// chunks w*NC .. w*NC + NC - 1 (chunk c = elements [c*512, c*512 + 512)).
// The input is read once, with non-temporal loads, so that it does not evict
// the operands of the GEMM that follows; chunks past K load the first chunk
// of x and are discarded.
template <int NC>
__global__ __launch_bounds__(512) void quantize_rows_kernel(
    const uint16_t* __restrict__ x, int64_t M, int64_t K,
    uint8_t* __restrict__ q, float* __restrict__ scale) {
  __shared__ uint32_t wave_max[8];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  const int64_t row = blockIdx.x;

  const uint16_t* xr = x + row * K;
  uint8_t* qr = q + row * (K / 2);

  uint4 v[NC];
  u16x2 am = {0, 0};  // two u16 lanes of sign-cleared bf16 bits
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int64_t k = static_cast<int64_t>(wave * NC + c) * 512 + lane * 8;
    {
      const bool ok = k < K;
      const v4u32 t = __builtin_nontemporal_load(reinterpret_cast<const v4u32*>(ok ? xr + k : x));
      v[c] = ok ? make_uint4(t.x, t.y, t.z, t.w) : make_uint4(0, 0, 0, 0);
    }
    am = __builtin_elementwise_max(am, __builtin_bit_cast(u16x2, v[c].x & 0x7FFF7FFFu));
    am = __builtin_elementwise_max(am, __builtin_bit_cast(u16x2, v[c].y & 0x7FFF7FFFu));
    am = __builtin_elementwise_max(am, __builtin_bit_cast(u16x2, v[c].z & 0x7FFF7FFFu));
    am = __builtin_elementwise_max(am, __builtin_bit_cast(u16x2, v[c].w & 0x7FFF7FFFu));
  }
  uint32_t amax = am.x > am.y ? am.x : am.y;
  amax = wave_max_u32(amax);
  if (nwaves > 1) {
    if (lane == 0) wave_max[wave] = amax;
    __syncthreads();
    amax = wave_max[0];
    for (int w = 1; w < nwaves; ++w) amax = amax > wave_max[w] ? amax : wave_max[w];
  }

  // Non-negative floats order like their bit patterns, so the u16 max of the
  // sign-cleared bf16 bits is the bit pattern of the absolute maximum.
  const float a = __uint_as_float(amax << 16);
  const float s = a / 7.0f;
  if (threadIdx.x == 0) scale[row] = s;

  if (s == 0.0f) {
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int64_t k = static_cast<int64_t>(wave * NC + c) * 512 + lane * 8;
      if (k < K) *reinterpret_cast<uint32_t*>(qr + k / 2) = 0u;
    }
    return;
  }

  const float rcp = 1.0f / s;
  if (__builtin_isinf(rcp)) {
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int64_t k = static_cast<int64_t>(wave * NC + c) * 512 + lane * 8;
      if (k < K) *reinterpret_cast<uint32_t*>(qr + k / 2) = pack8_exact(v[c], s);
    }
    return;
  }

#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int64_t k = static_cast<int64_t>(wave * NC + c) * 512 + lane * 8;
    bool near = false;
    uint32_t p = pack8_fast(v[c], rcp, &near);
    if (near) p = pack8_exact(v[c], s);
    if (k < K) *reinterpret_cast<uint32_t*>(qr + k / 2) = p;
  }
}

// Rows longer than the register-resident variants: two passes over the row
// (absmax, then quantise), the second mostly served from cache.
__global__ __launch_bounds__(256) void quantize_rows_stream_kernel(
    const uint16_t* __restrict__ x, int64_t M, int64_t K,
    uint8_t* __restrict__ q, float* __restrict__ scale) {
  const int lane = threadIdx.x & 63;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const uint16_t* xr = x + row * K;
  uint8_t* qr = q + row * (K / 2);

  uint32_t amax = 0;
  for (int64_t k = lane * 8; k < K; k += 512) {
    const uint4 v = *reinterpret_cast<const uint4*>(xr + k);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t lo = w[j] & 0x7FFFu, hi = (w[j] >> 16) & 0x7FFFu;
      amax = amax > lo ? amax : lo;
      amax = amax > hi ? amax : hi;
    }
  }
  amax = wave_max_u32(amax);
  const float a = __uint_as_float(amax << 16);
  const float s = a / 7.0f;
  if (lane == 0) scale[row] = s;
  const float rcp = 1.0f / s;
  const bool exact_row = __builtin_isinf(rcp);
  for (int64_t k = lane * 8; k < K; k += 512) {
    const uint4 v = *reinterpret_cast<const uint4*>(xr + k);
    uint32_t p = 0;
    if (s != 0.0f) {
      bool near = true;
      if (!exact_row) p = pack8_fast(v, rcp, &near);
      if (near) p = pack8_exact(v, s);
    }
    *reinterpret_cast<uint32_t*>(qr + k / 2) = p;
  }
}

// Group-wise variant: one scale per G consecutive k of a row (G = 64 or 128),
// s[r,g] = fl32(max |x| over the group / 7), the same codes and packing.
// The matrix is treated as flat 8-element units: thread i loads elements
// 8i .. 8i+7 (one 16-byte load; a wave reads 1 KiB contiguous) and the
// G/8 lanes of a group reduce their maxima with shuffles.  Since K % G == 0
// no group straddles two rows, so the scale of unit i is scale[i / (G/8)]
// in the row-major [rows, K/G] layout.  The quotient uses the same
// reciprocal-with-exact-fallback path as the per-row kernel, with one
// reciprocal per group.  Non-temporal loads, as in the per-row kernel.
template <int G>
__global__ __launch_bounds__(256) void quantize_groups_kernel(const uint16_t* __restrict__ x, int64_t units,
                                                              uint8_t* __restrict__ q, float* __restrict__ scale) {
  constexpr int kLanes = G / 8;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const bool live = i < units;
  uint4 v = make_uint4(0, 0, 0, 0);
  if (live) {
    const v4u32 t = __builtin_nontemporal_load(reinterpret_cast<const v4u32*>(x) + i);
    v = make_uint4(t.x, t.y, t.z, t.w);
  }
  u16x2 am = __builtin_bit_cast(u16x2, v.x & 0x7FFF7FFFu);
  am = __builtin_elementwise_max(am, __builtin_bit_cast(u16x2, v.y & 0x7FFF7FFFu));
  am = __builtin_elementwise_max(am, __builtin_bit_cast(u16x2, v.z & 0x7FFF7FFFu));
  am = __builtin_elementwise_max(am, __builtin_bit_cast(u16x2, v.w & 0x7FFF7FFFu));
  uint32_t amax = am.x > am.y ? am.x : am.y;
#pragma unroll
  for (int off = 1; off < kLanes; off <<= 1) {
    const uint32_t o = static_cast<uint32_t>(__shfl_xor(static_cast<int>(amax), off, 64));
    amax = amax > o ? amax : o;
  }
  const float a = __uint_as_float(amax << 16);
  const float s = a / 7.0f;
  if (live && (threadIdx.x % kLanes) == 0) scale[i / kLanes] = s;
  uint32_t p = 0;
  if (s != 0.0f) {
    const float rcp = 1.0f / s;
    bool near = true;
    if (!__builtin_isinf(rcp)) p = pack8_fast(v, rcp, &near);
    if (near) p = pack8_exact(v, s);
  }
  if (live) reinterpret_cast<uint32_t*>(q)[i] = p;
}

template <int NC>
hipError_t launch_nc(const uint16_t* x, int64_t M, int64_t K, uint8_t* q, float* s, int waves, hipStream_t st) {
  hipLaunchKernelGGL(quantize_rows_kernel<NC>, dim3(static_cast<unsigned>(M)), dim3(64 * waves), 0, st, x, M, K,
                     q, s);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_quantize_rows(const uint16_t* x, int64_t M, int64_t K, uint8_t* q, float* s,
                                hipStream_t st) {
  // A row of K elements is 'chunks' chunks of 512; it is split over up to 8
  // waves of at most 4 chunks each, so that many small waves keep enough
  // loads in flight and the last round of waves is short.
  const int64_t chunks = (K + 511) / 512;
  if (chunks <= 32) {
    const int waves = static_cast<int>(chunks <= 4 ? 1 : (chunks + 3) / 4);
    const int nc = static_cast<int>((chunks + waves - 1) / waves);
    switch (nc) {
      case 1: return launch_nc<1>(x, M, K, q, s, waves, st);
      case 2: return launch_nc<2>(x, M, K, q, s, waves, st);
      case 3: return launch_nc<3>(x, M, K, q, s, waves, st);
      default: return launch_nc<4>(x, M, K, q, s, waves, st);
    }
  }
  const dim3 grid(static_cast<unsigned>((M + 3) / 4));
  hipLaunchKernelGGL(quantize_rows_stream_kernel, grid, dim3(256), 0, st, x, M, K, q, s);
  return hipGetLastError();
}

hipError_t launch_quantize_groups(const uint16_t* x, int64_t M, int64_t K, int G, uint8_t* q, float* s,
                                  hipStream_t st) {
  const int64_t units = M * K / 8;
  const dim3 grid(static_cast<unsigned>((units + 255) / 256));
  if (G == 64) {
    hipLaunchKernelGGL(quantize_groups_kernel<64>, grid, dim3(256), 0, st, x, units, q, s);
  } else {
    hipLaunchKernelGGL(quantize_groups_kernel<128>, grid, dim3(256), 0, st, x, units, q, s);
  }
  return hipGetLastError();
}

}  // namespace jq
