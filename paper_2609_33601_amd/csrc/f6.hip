// The W4A4 layer on gfx950's 6-bit matrix cores (v_mfma_scale_f32_32x32x64_f8f6f4
// with BF6 = E3M2 operands), an exact alternative to the int8 MFMA path.
//
// Why it is exact.  Every int4 code -8..7 is a BF6 E3M2 value (|c| = 1.m * 2^e
// with two mantissa bits and e <= 3), so the matrix core multiplies the codes
// exactly.  Each product is an integer of magnitude <= 64 and every partial sum
// of a row of K <= 65536 products is an integer below 2^22, which fp32 holds
// exactly whatever the order of the additions.  The fp32 accumulator therefore
// equals the integer contraction acc[m,n] = sum_k qx[m,k] * qw[n,k], and the
// epilogue ((acc * s_x) * s_w) + bias sees the same operands as on the int8
// path.  Outputs are bit-identical to it.
//
// Why it is faster.  gfx950 issues the 6-bit MFMA at twice the int8 rate, and the
// operands reach it already encoded, so the loop holds no widening
// arithmetic at all:
//   * activations are quantised straight into BF6 by quantize_rows4_f6_kernel
//     (four rows per block) or quantize_rows_f6_kernel (longer rows), with
//     the same scale and codes as the packed-int4 quantiser;
//   * weights are converted once, offline, from the canonical packed int4
//     (or ternary) codes.
//
// The file also holds the group-wise form of the layer (one scale per G = 64
// or 128 codes): the same quantisers with group scales, and
// w4a4g_f6_gemm_kernel, which folds each group's exact product into fp32
// sums in k order.
//
// BF6 groups.  32 codes c[0..31] form a group of 192 bits, code p in bits
// 6p .. 6p+5 (six little-endian dwords d0..d5).  Rows are padded with zero
// codes to a multiple of 32 and taken in bands of 32; K is padded with zero
// codes to a multiple of 128 and cut into k-steps of 64 codes (KS of them, an
// even number).  Lane L = r + 32h of a v_mfma_*_32x32x64_f8f6f4 operand holds
// the group of codes 64s + 32h .. 64s + 32h + 31 of row r of the band for
// k-step s; A and B lanes use the same assignment, so the contraction is
// summed correctly.  Both operands take KS * 1536 bytes per band, band b at
// b * KS * 1536, in one of two orders within the band:
//   * activation layout (read by the GEMM through LDS): the fragment of
//     k-step s is 1536 bytes at s * 1536, lane L's d0..d3 at byte 16L and
//     d4, d5 at byte 1024 + 8L;
//   * weight layout (loaded by the GEMM straight into registers): k-steps 2u
//     and 2u + 1 share 3072 bytes at u * 3072, three planes of 1 KiB; lane L's
//     16 bytes of plane i are at 1024i + 16L, and its 48 bytes in plane order
//     are the six dwords of k-step 2u followed by those of k-step 2u + 1.
//     A wave thus loads two k-steps of a band with three 16-byte accesses per
//     lane (the vector memory path costs about the same per instruction
//     whatever its width).
//
// GEMM structure.  Persistent blocks walk the output tiles (256 n columns
// each) in an XCD-aware order, in one of two shapes:
//   * one 8-wave block per CU (two waves per SIMD) on tiles of
//     32 * tile_bands rows, tile_bands 7 or 8 picked per shape to spread the
//     tiles evenly over the CUs.  Wave (wm, wn) owns weight bands 2wn,
//     2wn + 1 of the tile and the activation bands of half wm (four bands,
//     or tile_bands - 4 in the second half; the two waves on a SIMD belong
//     to different halves, so every SIMD gets the same work).  Each XCD's
//     blocks walk K from stage x T / 8 of it (XCD x) round to it, so that
//     the eight XCDs read different slices of the operands at any moment
//     (FLUX MLP-down in the benchmark step: 157 -> 145 us);
//   * two 4-wave blocks per CU on tiles of 128 rows, wave wn owning weight
//     bands 2wn, 2wn + 1 and all four activation bands.  Taken where 256-row
//     tiles would not cover M evenly and K is not long: each block's epilogue
//     then runs beside the other block's MFMAs.  So that the two blocks of a
//     CU stay out of step, the blocks in the second half of each XCD's share
//     walk K from its middle stage round to it (the sum is exact in any
//     order).
// Either way a wave holds up to 2 x 4 tiles of 32x32, 128 fp32 accumulators
// per lane.
//   * Activations: shared by the four waves that read the same bands, staged
//     through LDS.  A stage is 128 codes of K (two k-steps x the block's
//     activation bands: 16 fragments, 24 KiB, or 8 fragments, 12 KiB),
//     moved by buffer_load ... lds (no registers) into a ring of three stage
//     slots, three stages ahead.
//   * Weights: loaded straight into registers one stage ahead, two register
//     sets (so the stage loop is unrolled by six, a multiple of both ring
//     sizes).
//   * Per stage: the eight MFMAs of k-step 0 run while the wave reads its
//     k-step 1 fragments from LDS and issues the next stage's weight loads,
//     one or two after each fragment's MFMAs; then it waits for its share
//     of the next stage's DMA and meets the others at a barrier (no memory
//     fence); then the MFMAs of k-step 1 run while the next stage's k-step 0
//     fragments are read and the DMA three stages ahead goes into the slot
//     just read, one instruction after each of the first fragments.  Issued
//     in one burst per wave at the stage's start and middle, the same loads
//     queued up behind each other and held the waves' MFMAs back (the
//     spread issue took the FLUX MLP-down GEMM from 147 to 131 us on zero
//     codes).  No VALU work sits between the MFMAs.
//   * Every vector-memory instruction of the stage loop (the weight loads
//     and the buffer -> LDS transfers) is issued as an instruction of its
//     own, and the loop orders it with explicit waits only: at a stage's
//     start, vmcnt(3) (this stage's weights, issued before the previous
//     stage's DMA, have landed); at its middle, vmcnt(9), lgkmcnt(0) and the
//     barrier (the next slot's DMA has landed and every read of the slot
//     about to be refilled has completed).  Left to the compiler, the
//     transfers made it wait for every DMA in flight before each LDS read.
//     The compiler does not know that these loads complete after they
//     issue, so the loaded registers pass through an empty asm after their
//     wait before any use, and the build checks the generated code: no
//     instruction may touch a load's registers before a wait retires it
//     (check_waits.py).  The file is also built without machine sinking,
//     which otherwise moved the first k-step's MFMAs below the stage's
//     barrier (into the block after the tile's first-stage branch), leaving
//     the matrix pipes idle while both waves of a SIMD waited there.
//   * An activation fragment's 16- and 8-byte parts land next to each other
//     in registers (the 8-byte part read on its own, not paired with another
//     fragment's), and a band's three 16-byte weight parts of a stage are
//     the two k-steps' operands as two overlapping 6-dword windows.
//   * The weight fragment is operand A and the activation fragment operand B,
//     so the 32x32 result is y^T: lane L holds column m = L % 32 and rows
//     n = 8j + 4(L / 32) + r (j, r = 0..3).  The epilogue scales them, packs
//     bf16 and stages them through LDS to store whole 128-byte rows.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>
#include <type_traits>
#include <utility>

#include "gemm_common.h"
#include "jq.h"
#include "jq_internal.h"

namespace jq {

namespace {

using namespace gemm_detail;

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef unsigned v6u __attribute__((ext_vector_type(6)));
typedef float v16f32 __attribute__((ext_vector_type(16)));
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
typedef unsigned v4u32 __attribute__((ext_vector_type(4)));

constexpr int kFragBytes = 1536;          // one 32-row x 64-code fragment
constexpr int kFBN = 256;                 // block tile columns
constexpr int kDmaPerWave = 3;            // stage DMA instructions per wave
constexpr int64_t kShortK = 6144;          // largest K that may take the two-block shape
constexpr int kQuantBatchMax = 8;          // inputs of one batched quantiser launch

// The GEMM comes in two block shapes (WAVES = 8 or 4 waves of 64): one
// 8-wave block per CU on a tile of up to 256 activation rows, or two 4-wave
// blocks per CU on tiles of 128 rows.  Per wave the work is the same (two
// weight bands, four activation bands); a stage holds the block's
// activation bands for two k-steps.
template <int WAVES>
struct F6Shape {
  static constexpr int kThreads = 64 * WAVES;
  static constexpr int kBands = WAVES;                          // activation bands staged per tile
  static constexpr int kFBM = 32 * kBands;                      // tile rows at most
  static constexpr int kStageU4 = 2 * kBands * kFragBytes / 16;  // one stage slot, 16-byte units
  static_assert(kStageU4 == 64 * kDmaPerWave * WAVES, "a stage is 3 DMA instructions per wave");
};

// 32 codes (as exact fp32 integers, code p in q[p]) -> six dwords, code p in bits 6p..6p+5.
// The converter interleaves its two sources (field 2i <- src0[i], field 2i+1 <- src1[i]).
__device__ __forceinline__ v6u bf6_group(const float* q) {
  v16f32 ev, od;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    ev[i] = q[2 * i];
    od[i] = q[2 * i + 1];
  }
  return __builtin_amdgcn_cvt_scalef32_2xpk16_bf6_f32(ev, od, 1.0f);
}

constexpr float kMagic = 12582912.0f;         // 1.5 * 2^23
constexpr float kNearTie = 0.5f - 0x1p-17f;

__device__ __forceinline__ float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }

// Codes of one 32-element group (16 dwords of bf16 pairs).  Reciprocal path
// with the exact IEEE division wherever the product sits next to a rounding
// decision point (the argument is that of the packed-int4 quantiser), or the
// division for every element when the reciprocal overflows.
__device__ __forceinline__ void codes32(const uint32_t* w, float s, float rcp, bool exact_row, float* q) {
  bool near = exact_row;
  if (!exact_row) {
    float dmax = 0.0f;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const float te = bf16_lo(w[j]) * rcp;
      const float to = bf16_hi(w[j]) * rcp;
      const float re = (te + kMagic) - kMagic;
      const float ro = (to + kMagic) - kMagic;
      dmax = fmaxf(dmax, fmaxf(fabsf(te - re), fabsf(to - ro)));
      q[2 * j] = re;
      q[2 * j + 1] = ro;
    }
    near = !(dmax < kNearTie);
  }
  if (near) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      q[2 * j] = fminf(fmaxf(__builtin_rintf(bf16_lo(w[j]) / s), -8.0f), 7.0f);
      q[2 * j + 1] = fminf(fmaxf(__builtin_rintf(bf16_hi(w[j]) / s), -8.0f), 7.0f);
    }
  }
}

// Store the BF6 group gi (= 2 * kstep + half) of row `row` into the
// activation layout (WLAYOUT false) or the weight layout (true).
template <bool WLAYOUT>
__device__ __forceinline__ void store_group(uint8_t* out, int64_t ksteps, int64_t row, int gi, v6u d) {
  const int s = gi >> 1, h = gi & 1;
  const int L = static_cast<int>(row & 31) + 32 * h;
  if constexpr (!WLAYOUT) {
    uint8_t* p = out + ((row >> 5) * ksteps + s) * kFragBytes;
    *reinterpret_cast<uint4*>(p + 16 * L) = make_uint4(d[0], d[1], d[2], d[3]);
    *reinterpret_cast<uint2*>(p + 1024 + 8 * L) = make_uint2(d[4], d[5]);
  } else {
    uint8_t* p = out + (row >> 5) * ksteps * kFragBytes + (s >> 1) * (2 * kFragBytes) + 16 * L;
    if ((s & 1) == 0) {
      *reinterpret_cast<uint4*>(p) = make_uint4(d[0], d[1], d[2], d[3]);
      *reinterpret_cast<uint2*>(p + 1024) = make_uint2(d[4], d[5]);
    } else {
      *reinterpret_cast<uint2*>(p + 1024 + 8) = make_uint2(d[0], d[1]);
      *reinterpret_cast<uint4*>(p + 2048) = make_uint4(d[2], d[3], d[4], d[5]);
    }
  }
}

// Row of block b.  Blocks are dealt round-robin to the 8 XCDs; the 32 rows of
// a band all go to the blocks of one XCD, so the partial cache lines of a
// fragment are completed in one L2 before they are written back.
__device__ __forceinline__ int64_t row_of_block(int64_t b) {
  const int64_t x = b % kNumXcd, j = b / kNumXcd;
  return 32 * (kNumXcd * (j / 32) + x) + (j % 32);
}

// Per-token quantiser writing the BF6 operand.  One block per row of the
// padded operand; thread i handles groups i + T j (j < NJ) of 32 codes and
// keeps them in registers between the absmax and the quantisation.  A wave
// reads its 64 groups (4 KiB) as four 1 KiB loads of whole cache lines and
// hands each lane its own 64 bytes through LDS (the 16-byte chunk q of the
// wave's 256 at slot q ^ ((q >> 4) & 15), so that neither the writes nor the
// reads conflict).  The loads are non-temporal: the input is read once, and
// left to the caches it would evict the operands of the GEMM that follows.
// The scale and the codes are those of quantize_rows_kernel.  Padding rows
// (M <= row < 32 * ceil(M/32)) get zero codes and no scale.
//
// G = 64 or 128: one scale per G consecutive codes instead (scale [M, K/G]
// row-major, the codes and scales of quantize_groups_kernel).  A group is the
// 32-code groups of G/32 neighbouring lanes, which meet with shuffles.
template <int NJ, int G>
__global__ __launch_bounds__(512) void quantize_rows_f6_kernel(const uint16_t* __restrict__ x, int64_t M, int64_t K,
                                                               int64_t rows_padded, int64_t ksteps,
                                                               uint8_t* __restrict__ out, float* __restrict__ scale) {
  __shared__ uint32_t wave_max[8];
  const int T = blockDim.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nwaves = T >> 6;
  const int64_t row = row_of_block(blockIdx.x);
  if (row >= rows_padded) return;
  const bool live = row < M;
  const int groups = static_cast<int>(2 * ksteps);
  const uint16_t* xr = x + (live ? row : 0) * K;

  extern __shared__ v4u32 xt[];  // 256 chunks of 16 bytes per wave
  v4u32* xw = xt + 256 * wave;
  auto swz = [](int q) { return q ^ ((q >> 4) & 15); };
  uint4 v[NJ][4];
  u16x2 am = {0, 0};
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int64_t base = 32 * static_cast<int64_t>(T * j + 64 * wave);
    v4u32 t[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      // Out-of-range chunks (K padding, padding rows) load the first chunk
      // of x and are zeroed; no branch, so the four loads issue together.
      const int64_t e = base + 512 * c + 8 * lane;
      const bool ok = live && e < K;
      t[c] = __builtin_nontemporal_load(reinterpret_cast<const v4u32*>(ok ? xr + e : x));
      if (!ok) t[c] = v4u32{0, 0, 0, 0};
      am = __builtin_elementwise_max(am, __builtin_bit_cast(u16x2, t[c].x & 0x7FFF7FFFu));
      am = __builtin_elementwise_max(am, __builtin_bit_cast(u16x2, t[c].y & 0x7FFF7FFFu));
      am = __builtin_elementwise_max(am, __builtin_bit_cast(u16x2, t[c].z & 0x7FFF7FFFu));
      am = __builtin_elementwise_max(am, __builtin_bit_cast(u16x2, t[c].w & 0x7FFF7FFFu));
    }
    // Only this wave touches its chunks, and LDS runs a wave's accesses in
    // order: the fences just keep the compiler from moving them.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int c = 0; c < 4; ++c) xw[swz(64 * c + lane)] = t[c];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const v4u32 r = xw[swz(4 * lane + c)];
      v[j][c] = make_uint4(r.x, r.y, r.z, r.w);
    }
  }
  if constexpr (G != 0) {
    (void)am;
    (void)wave_max;
    constexpr int kLanes = G / 32;  // lanes per group
    const int64_t KG = K / G;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      u16x2 gm = {0, 0};
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        gm = __builtin_elementwise_max(gm, __builtin_bit_cast(u16x2, v[j][c].x & 0x7FFF7FFFu));
        gm = __builtin_elementwise_max(gm, __builtin_bit_cast(u16x2, v[j][c].y & 0x7FFF7FFFu));
        gm = __builtin_elementwise_max(gm, __builtin_bit_cast(u16x2, v[j][c].z & 0x7FFF7FFFu));
        gm = __builtin_elementwise_max(gm, __builtin_bit_cast(u16x2, v[j][c].w & 0x7FFF7FFFu));
      }
      uint32_t gmax = gm.x > gm.y ? gm.x : gm.y;
#pragma unroll
      for (int off = 1; off < kLanes; off <<= 1) {
        const uint32_t o = static_cast<uint32_t>(__shfl_xor(static_cast<int>(gmax), off, 64));
        gmax = gmax > o ? gmax : o;
      }
      const int gi = threadIdx.x + T * j;
      if (gi >= groups) continue;
      const float sg = __uint_as_float(gmax << 16) / 7.0f;
      if (live && gi % kLanes == 0 && 32 * static_cast<int64_t>(gi) < K) scale[row * KG + gi / kLanes] = sg;
      const float rcp = (sg == 0.0f) ? 0.0f : 1.0f / sg;
      float q[32];
      if (sg == 0.0f) {
#pragma unroll
        for (int p = 0; p < 32; ++p) q[p] = 0.0f;
      } else {
        const uint32_t w[16] = {v[j][0].x, v[j][0].y, v[j][0].z, v[j][0].w, v[j][1].x, v[j][1].y,
                                v[j][1].z, v[j][1].w, v[j][2].x, v[j][2].y, v[j][2].z, v[j][2].w,
                                v[j][3].x, v[j][3].y, v[j][3].z, v[j][3].w};
        codes32(w, sg, rcp, __builtin_isinf(rcp), q);
      }
      store_group<false>(out, ksteps, row, gi, bf6_group(q));
    }
    return;
  }
  uint32_t amax = am.x > am.y ? am.x : am.y;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint32_t o = static_cast<uint32_t>(__shfl_xor(static_cast<int>(amax), off, 64));
    amax = amax > o ? amax : o;
  }
  if (nwaves > 1) {
    if (lane == 0) wave_max[wave] = amax;
    __syncthreads();
    amax = wave_max[0];
    for (int w = 1; w < nwaves; ++w) amax = amax > wave_max[w] ? amax : wave_max[w];
  }
  // Non-negative floats order like their bit patterns.
  const float a = __uint_as_float(amax << 16);
  const float s = a / 7.0f;
  if (live && threadIdx.x == 0) scale[row] = s;
  const float rcp = (s == 0.0f) ? 0.0f : 1.0f / s;
  const bool exact_row = __builtin_isinf(rcp);

#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int gi = threadIdx.x + T * j;
    if (gi >= groups) continue;
    float q[32];
    if (s == 0.0f) {
#pragma unroll
      for (int p = 0; p < 32; ++p) q[p] = 0.0f;
    } else {
      const uint32_t w[16] = {v[j][0].x, v[j][0].y, v[j][0].z, v[j][0].w, v[j][1].x, v[j][1].y,
                              v[j][1].z, v[j][1].w, v[j][2].x, v[j][2].y, v[j][2].z, v[j][2].w,
                              v[j][3].x, v[j][3].y, v[j][3].z, v[j][3].w};
      codes32(w, s, rcp, exact_row, q);
    }
    store_group<false>(out, ksteps, row, gi, bf6_group(q));
  }
}

// First row of block b in the four-rows-per-block quantiser: the eight
// blocks of a band are consecutive blocks of one XCD, so the lines of a
// fragment that they write piecewise meet in one L2.
__device__ __forceinline__ int64_t row0_of_block4(int64_t b) {
  const int64_t x = b % kNumXcd, j = b / kNumXcd;
  return 32 * (kNumXcd * (j / 8) + x) + 4 * (j % 8);
}

// The same quantiser for rows of up to 512 groups (K <= 16384), four rows
// per block: lane l of a wave takes row l % 4 and group slot l / 4, so that
// the four lanes of a group slot store the same fragment piece of four
// consecutive rows, 64 (and 32) contiguous bytes, instead of four scattered
// 16- and 8-byte pieces.  Wave w's j-th set of groups is the 16 groups from
// 16 (W j + w) in each of the four rows: four 1 KiB loads of whole lines (one
// per row), regrouped per lane through LDS (chunk q = 64 row + 4 slot +
// quarter at slot q ^ ((q >> 6) & 3): conflict-free both ways).  Per-row
// maxima meet by shuffles within a wave and through LDS across waves; group
// maxima (G = 64, 128) by shuffles between the lanes of a group.  The scales
// and codes are those of quantize_rows_f6_kernel.
//
// The body is shared with the batched form (several inputs in one launch):
// block b of the input, and nj <= NJ sets of groups per wave (the rest of the
// register arrays idle).
template <int NJ, int G>
__device__ __forceinline__ void q4_rows(const uint16_t* __restrict__ x, int64_t M, int64_t K, int64_t rows_padded,
                                        int64_t ksteps, uint8_t* __restrict__ out, float* __restrict__ scale,
                                        int64_t b, int nj) {
  __shared__ uint32_t wave_max[8][4];
  const int T = blockDim.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nwaves = T >> 6;
  const int64_t row0 = row0_of_block4(b);
  if (row0 >= rows_padded) return;
  const int rr = lane & 3, gslot = lane >> 2;
  const int64_t row = row0 + rr;
  const bool live = row < M;
  const int groups = static_cast<int>(2 * ksteps);

  extern __shared__ v4u32 xt[];  // 256 chunks of 16 bytes per wave
  v4u32* xw = xt + 256 * wave;
  auto swz = [](int q) { return q ^ ((q >> 6) & 3); };
  // All loads first (NJ x 4 of them in flight), then the regrouping.
  v4u32 t[NJ][4];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    if (j >= nj) break;
    const int g0 = 16 * (nwaves * j + wave);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      // row row0 + c, elements 32 g0 + 8 lane .. + 7; out-of-range chunks load
      // the first chunk of x and are zeroed (no branch between the loads)
      const int64_t e = 32 * static_cast<int64_t>(g0) + 8 * lane;
      const bool ok = row0 + c < M && e < K;
      t[j][c] = __builtin_nontemporal_load(reinterpret_cast<const v4u32*>(ok ? x + (row0 + c) * K + e : x));
      if (!ok) t[j][c] = v4u32{0, 0, 0, 0};
    }
  }
  uint4 v[NJ][4];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    if (j >= nj) break;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int c = 0; c < 4; ++c) xw[swz(64 * c + lane)] = t[j][c];
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const v4u32 r = xw[swz(64 * rr + 4 * gslot + c)];
      v[j][c] = make_uint4(r.x, r.y, r.z, r.w);
    }
  }
  // The lane's maximum over each of its groups.
  uint32_t gmax[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) gmax[j] = 0;  // sets past nj stay 0
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    if (j >= nj) break;
    u16x2 gm = {0, 0};
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      gm = __builtin_elementwise_max(gm, __builtin_bit_cast(u16x2, v[j][c].x & 0x7FFF7FFFu));
      gm = __builtin_elementwise_max(gm, __builtin_bit_cast(u16x2, v[j][c].y & 0x7FFF7FFFu));
      gm = __builtin_elementwise_max(gm, __builtin_bit_cast(u16x2, v[j][c].z & 0x7FFF7FFFu));
      gm = __builtin_elementwise_max(gm, __builtin_bit_cast(u16x2, v[j][c].w & 0x7FFF7FFFu));
    }
    gmax[j] = gm.x > gm.y ? gm.x : gm.y;
  }
  float srow = 0.0f;
  if constexpr (G == 0) {
    uint32_t amax = 0;
#pragma unroll
    for (int j = 0; j < NJ; ++j) amax = amax > gmax[j] ? amax : gmax[j];
#pragma unroll
    for (int off = 4; off <= 32; off <<= 1) {  // the 16 lanes of this row
      const uint32_t o = static_cast<uint32_t>(__shfl_xor(static_cast<int>(amax), off, 64));
      amax = amax > o ? amax : o;
    }
    if (nwaves > 1) {
      if (gslot == 0) wave_max[wave][rr] = amax;
      __syncthreads();
      amax = wave_max[0][rr];
      for (int w = 1; w < nwaves; ++w) amax = amax > wave_max[w][rr] ? amax : wave_max[w][rr];
    }
    srow = __uint_as_float(amax << 16) / 7.0f;
    if (live && wave == 0 && gslot == 0) scale[row] = srow;
  } else {
    (void)wave_max;
  }
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    if (j >= nj) break;
    float s = srow;
    if constexpr (G != 0) {
      constexpr int kLanes = G / 32;  // group slots per group, 4 lanes apart
      uint32_t gm = gmax[j];
#pragma unroll
      for (int off = 4; off < 4 * kLanes; off <<= 1) {
        const uint32_t o = static_cast<uint32_t>(__shfl_xor(static_cast<int>(gm), off, 64));
        gm = gm > o ? gm : o;
      }
      s = __uint_as_float(gm << 16) / 7.0f;
    }
    const int gi = 16 * (nwaves * j + wave) + gslot;
    if (gi >= groups) continue;
    if constexpr (G != 0) {
      constexpr int kLanes = G / 32;
      if (live && gi % kLanes == 0 && 32 * static_cast<int64_t>(gi) < K) scale[row * (K / G) + gi / kLanes] = s;
    }
    const float rcp = (s == 0.0f) ? 0.0f : 1.0f / s;
    float q[32];
    if (s == 0.0f) {
#pragma unroll
      for (int p = 0; p < 32; ++p) q[p] = 0.0f;
    } else {
      const uint32_t w[16] = {v[j][0].x, v[j][0].y, v[j][0].z, v[j][0].w, v[j][1].x, v[j][1].y,
                              v[j][1].z, v[j][1].w, v[j][2].x, v[j][2].y, v[j][2].z, v[j][2].w,
                              v[j][3].x, v[j][3].y, v[j][3].z, v[j][3].w};
      codes32(w, s, rcp, __builtin_isinf(rcp), q);
    }
    store_group<false>(out, ksteps, row, gi, bf6_group(q));
  }
}

template <int NJ, int G>
__global__ __launch_bounds__(512) void quantize_rows4_f6_kernel(const uint16_t* __restrict__ x, int64_t M, int64_t K,
                                                                int64_t rows_padded, int64_t ksteps,
                                                                uint8_t* __restrict__ out, float* __restrict__ scale) {
  q4_rows<NJ, G>(x, M, K, rows_padded, ksteps, out, scale, blockIdx.x, NJ);
}

// Several independent inputs quantised per token in one launch (rows of up
// to 512 groups each): input i takes the blocks from first[i] on, a multiple
// of 64 so that each band's blocks stay on one XCD, and runs with nj[i] of
// the NJ sets of groups per wave.  Each input's codes and scales are those
// of its own launch of quantize_rows4_f6_kernel.
struct Q4Input {
  const uint16_t* x;
  uint8_t* out;
  float* scale;
  int64_t M, K, rows_padded, ksteps, first;
  int nj;
};
struct Q4Batch {
  Q4Input in[kQuantBatchMax];
  int count;
};

template <int NJ>
__global__ __launch_bounds__(512) void quantize_rows4_f6_batch_kernel(Q4Batch b) {
  int i = 0;
  while (i + 1 < b.count && static_cast<int64_t>(blockIdx.x) >= b.in[i + 1].first) ++i;
  const Q4Input& e = b.in[i];
  q4_rows<NJ, 0>(e.x, e.M, e.K, e.rows_padded, e.ksteps, e.out, e.scale, blockIdx.x - e.first, e.nj);
}

// Canonical packed int4 codes (TERNARY false) or packed ternary codes (true)
// -> BF6 operand in the activation or the weight layout.  One thread per
// (row, 32-code group) of the padded operand; padding rows and codes are
// written as zeros.
template <bool WLAYOUT, bool TERNARY>
__global__ __launch_bounds__(256) void int4_to_f6_kernel(const uint8_t* __restrict__ q, int64_t rows,
                                                         int64_t rows_padded, int64_t K, int64_t ksteps,
                                                         uint8_t* __restrict__ out) {
  const int groups = static_cast<int>(2 * ksteps);
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= rows_padded * groups) return;
  const int64_t row = i / groups;
  const int gi = static_cast<int>(i % groups);
  const bool live = row < rows && 32 * static_cast<int64_t>(gi) < K;
  float c[32];
  if constexpr (!TERNARY) {
    uint4 p = make_uint4(0, 0, 0, 0);
    if (live) p = *reinterpret_cast<const uint4*>(q + row * (K / 2) + 16 * static_cast<int64_t>(gi));
    const uint32_t w[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int n = 0; n < 8; ++n)  // nibble n of dword d is code 8d + n (even codes in low nibbles)
        c[8 * d + n] = static_cast<float>(static_cast<int>(w[d] << (28 - 4 * n)) >> 28);
  } else {
    uint2 p = make_uint2(0, 0);
    if (live) p = *reinterpret_cast<const uint2*>(q + row * (K / 4) + 8 * static_cast<int64_t>(gi));
    const uint32_t w[2] = {p.x, p.y};
#pragma unroll
    for (int d = 0; d < 2; ++d)
#pragma unroll
      for (int n = 0; n < 16; ++n)  // 2-bit field n of dword d is code 16d + n
        c[16 * d + n] = static_cast<float>(static_cast<int>(w[d] << (30 - 2 * n)) >> 30);
  }
  store_group<WLAYOUT>(out, ksteps, row, gi, bf6_group(c));
}

// ---------------------------------------------------------------------------
// GEMM

typedef int v4i32 __attribute__((ext_vector_type(4)));
typedef unsigned v2u32 __attribute__((ext_vector_type(2)));
typedef int v2i32 __attribute__((ext_vector_type(2)));

struct WFrag {
  v8i f[2][2];  // [k-step][band]; dwords 0..5 used
};
// A wave's weights of one stage as loaded: three 16-byte parts per band
// (the six dwords of k-step 0, then those of k-step 1), turned into MFMA
// operands only once the stage's wait has passed.
struct WRaw {
  v4i32 p[2][3];  // [band][part]
};

__device__ __forceinline__ v8i join(v4i32 a, v2i32 b) { return v8i{a.x, a.y, a.z, a.w, b.x, b.y, 0, 0}; }

// f(integral_constant<int, i>) for i = 0 .. N - 1, in order, as straight-line code.
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Buffer -> LDS transfers issued as instructions of their own (M0 set
// alongside), so that the compiler neither tracks them nor orders LDS reads
// behind them: the GEMM orders them against its LDS reads with its own
// explicit waits, and is the only user of M0 in its kernel.
typedef unsigned v4u32r __attribute__((ext_vector_type(4)));
struct RawRsrc {
  v4u32r w;  // the four descriptor words of a raw (unswizzled, stride 0) buffer
};
__device__ __forceinline__ RawRsrc raw_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  RawRsrc r;
  r.w = v4u32r{static_cast<uint32_t>(a), static_cast<uint32_t>(a >> 32) & 0xFFFFu, bytes,
               static_cast<uint32_t>(kBufferFlags)};
  return r;
}
// The LDS byte address of a __shared__ object: the low 32 bits of its generic address.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p));
}
__device__ __forceinline__ void dma16_raw(const RawRsrc& r, uint32_t lds, uint32_t voffset, uint32_t soffset) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :: "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(voffset), "s"(r.w), "s"(soffset) : "memory");
}
__device__ __forceinline__ v4i32 load16_raw(const RawRsrc& r, uint32_t voffset, uint32_t soffset) {
  v4i32 v;
  asm volatile("buffer_load_dwordx4 %0, %1, %2, %3 offen" : "=v"(v) : "v"(voffset), "s"(r.w), "s"(soffset));
  return v;
}
__device__ __forceinline__ void dma4_raw(const RawRsrc& r, uint32_t lds, uint32_t voffset) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, 0 offen lds"
               :: "s"(__builtin_amdgcn_readfirstlane(lds)), "v"(voffset), "s"(r.w) : "memory");
}

constexpr int kWaitcntBase = (0x7 << 4) | (0xF << 8);  // expcnt, lgkmcnt: no wait
constexpr int vmcnt_imm(int n) { return kWaitcntBase | (n & 0xF) | ((n >> 4) << 14); }
constexpr int kLgkm0 = 0xC07F;                          // lgkmcnt(0), vmcnt and expcnt: no wait
constexpr int kWLoads = 6;                              // weight loads per wave per stage
constexpr uint32_t kOutside = 0x80000000u;              // a buffer offset past every operand

// BIAS_TAIL: a bias with odd N, whose last value the epilogue of a ragged
// tile reads from memory (its staged pair reads past the buffer as zero);
// otherwise every bias value comes from LDS and the epilogue has no branch.
template <int WAVES, Epilogue EPI, bool HAS_BIAS, bool BIAS_TAIL>
__global__ __launch_bounds__(64 * WAVES, 8 / WAVES) void w4a4_f6_gemm_kernel(
    const uint8_t* __restrict__ xf6, const float* __restrict__ sx, int M, int mbands,
    const uint8_t* __restrict__ wf6, const float* __restrict__ sw, int N, int nbands, int ksteps,
    const uint16_t* __restrict__ bias, void* __restrict__ out, int tile_bands, int tiles_m, int tiles_n,
    int grid_blocks) {
  // The ring (72 or 36 KiB) as three separate arrays.  With the stage loop
  // unrolled by six every slot is known at compile time, so the compiler
  // can tell the slot being read from the one the DMA is writing.
  using S = F6Shape<WAVES>;
  constexpr int kStageU4 = S::kStageU4, kFBM = S::kFBM, kF6Threads = S::kThreads;
  __shared__ uint4 lds0[kStageU4];
  __shared__ uint4 lds1[kStageU4];
  __shared__ uint4 lds2[kStageU4];
  // Output staging for the epilogue: per wave 64 rows x 64 bf16 (128 bytes a
  // row), 16-byte chunk c of row r at chunk c ^ ((r >> 1) & 7).  Accessed
  // only as stg[i] / stg2[i] with a computed index, so that every access
  // keeps the alias information that tells it apart from the DMA targets
  // (an access without it would wait for every load in flight).
  __shared__ v4u32 stg[kF6Threads / 64 * 512];
  // The current tile's scales and bias, moved in by DMA for the epilogue.
  __shared__ float sc_x[kFBM];
  __shared__ float sc_w[kFBN];
  __shared__ float sc_b[kFBN / 2];  // bf16 pairs
  auto slot = [&](int k) __attribute__((always_inline)) { return k == 0 ? lds0 : (k == 1 ? lds1 : lds2); };

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = WAVES == 8 ? wave >> 2 : 0, wn = wave & 3;  // activation half, weight quarter (2 bands)
  // A tile has tile_bands (7 or 8) bands of 32 activation rows: the first
  // half takes four of them, the second half the rest, so each SIMD (one wave
  // of each half) does the same work whatever the tile height.
  const int tile_rows = 32 * tile_bands;
  const int T = ksteps / 2;                  // stages of 128 codes per tile
  const int last = T - 1;

  // The block's tiles: virtual block ids v = blockIdx.x + i * grid_blocks of
  // a grid of 8 * ceil(tiles / 8) blocks in the XCD-aware order (grid_blocks
  // is a multiple of 8, so the XCD of every tile of this block is the
  // block's own).  The launch makes every block walk a single tile when a
  // tile has fewer than three stages, since the loads run three stages ahead
  // and must not reach past the next tile.
  int ntiles = 0;
  {
    const int vmax = (tiles_m * tiles_n + kNumXcd - 1) / kNumXcd * kNumXcd;
    TileCoord tc;
    for (int v = blockIdx.x; v < vmax && tile_of_block(v, tiles_m, tiles_n, &tc); v += grid_blocks) ++ntiles;
  }
  if (ntiles == 0) return;
  auto tile_at = [&](int i, int* m0, int* n0) __attribute__((always_inline)) {
    TileCoord tc;
    tile_of_block(blockIdx.x + i * grid_blocks, tiles_m, tiles_n, &tc);
    *m0 = tc.tm * tile_rows;
    *n0 = tc.tn * kFBN;
  };

  const RawRsrc rsx = raw_rsrc(xf6, static_cast<uint32_t>(static_cast<int64_t>(mbands) * ksteps * kFragBytes));
  const RawRsrc rsw = raw_rsrc(wf6, static_cast<uint32_t>(static_cast<int64_t>(nbands) * ksteps * kFragBytes));

  // Activation DMA: the 16 fragments of a stage ((k-step s, band b) in order
  // 8s + b) are contiguous 1536-byte blocks in LDS; slot part
  // Q = 64 (3 wave + j) + lane of the stage is byte 16 (Q % 96) of fragment
  // Q / 96.  Per lane: the band within the tile and the byte offset within
  // the band's stage.  Bands past the operand are clamped (their results are
  // discarded); bands past the tile get an offset outside the operand, which
  // the buffer load answers with zeros without touching memory.
  int rband[kDmaPerWave];
  uint32_t rpart[kDmaPerWave];
#pragma unroll
  for (int j = 0; j < kDmaPerWave; ++j) {
    const int Q = 64 * (kDmaPerWave * wave + j) + lane;
    const int R = Q / 96, q = Q % 96;
    rband[j] = R % S::kBands;
    rpart[j] = (R % S::kBands) < tile_bands ? (R / S::kBands) * kFragBytes + 16 * q : kOutside;
  }
  const uint32_t band_bytes = static_cast<uint32_t>(ksteps) * kFragBytes;
  // The blocks walk the stages of their tiles from a point of K of their
  // own (the fp32 sums of integers do not depend on the order).  One block
  // per CU: each XCD starts an eighth of K after the one before, so that at
  // any moment the XCDs read different slices of the operands rather than
  // all requesting the same weight lines together.  Two blocks per CU: the
  // second half of each XCD's blocks starts from the middle of K, so the two
  // blocks on a CU reach their epilogues half a tile apart and one runs its
  // MFMAs while the other stores.
  const int koff =
      WAVES == 8 ? static_cast<int>(blockIdx.x % kNumXcd) * T / kNumXcd
                 : ((static_cast<int>(blockIdx.x / kNumXcd) >= grid_blocks / kNumXcd / 2) ? T / 2 : 0);
  auto rot = [&](int st) __attribute__((always_inline)) { return st + koff < T ? st + koff : st + koff - T; };

  // Stage `st` of the tile at (m0, n0): part j of the wave's share of its
  // activations into slot k, or part pp (band pp / 3, 16-byte part pp % 3)
  // of its weights into w.
  auto issue_dma = [&](int m0, int st, int k, int j) __attribute__((always_inline)) {
    uint4* dst = slot(k) + 64 * kDmaPerWave * wave;
    const uint32_t band = static_cast<uint32_t>(min(m0 / 32 + rband[j], mbands - 1));
    dma16_raw(rsx, lds_addr(dst + 64 * j), rpart[j] == kOutside ? kOutside : band * band_bytes + rpart[j],
              2 * kFragBytes * rot(st));
  };
  auto load_w = [&](WRaw& w, int n0, int st, int pp) __attribute__((always_inline)) {
    const int f = pp / 3, q = pp % 3;
    const uint32_t wb = static_cast<uint32_t>(min(n0 / 32 + 2 * wn + f, nbands - 1)) * band_bytes;
    const uint32_t so = static_cast<uint32_t>(2 * rot(st) * kFragBytes);
    w.p[f][q] = load16_raw(rsw, wb + 1024 * q + 16 * lane, so);
  };
  // The MFMA operands of a loaded stage, once the wait for its loads has
  // passed.  The compiler takes an asm load's result as ready when the asm
  // is issued, so the parts first pass through an empty asm placed after the
  // wait: any copy it makes to assemble an operand then reads them after the
  // wait, not in the register a load may still be writing.
  auto frags = [&](WRaw& w) __attribute__((always_inline)) {
    asm volatile("" : "+v"(w.p[0][0]), "+v"(w.p[0][1]), "+v"(w.p[0][2]), "+v"(w.p[1][0]), "+v"(w.p[1][1]),
                 "+v"(w.p[1][2]));
    WFrag r;
#pragma unroll
    for (int f = 0; f < 2; ++f) {
      // the k-steps are the 6-dword windows of the 12 loaded dwords
      r.f[0][f] = __builtin_shufflevector(w.p[f][0], w.p[f][1], 0, 1, 2, 3, 4, 5, -1, -1);
      r.f[1][f] = __builtin_shufflevector(w.p[f][1], w.p[f][2], 2, 3, 4, 5, 6, 7, -1, -1);
    }
    return r;
  };
  // Scales and bias of the tile at (m0, n0) into LDS: waves 0..3 take a
  // quarter of s_x each, waves 4..7 a quarter of s_w, waves 0..1 half of the
  // bias.  Entries past M or N read as zero (outside the buffers).
  auto issue_scales = [&](int m0, int n0) __attribute__((always_inline)) {
    if constexpr (EPI == Epilogue::kBf16 && WAVES == 4) {
      // every wave a quarter of s_w; waves 0, 1 half of s_x each, waves 2, 3
      // half of the bias each
      {
        const RawRsrc r = raw_rsrc(sw, 4 * N);
        dma4_raw(r, lds_addr(sc_w + 64 * wave), 4 * static_cast<uint32_t>(n0 + 64 * wave + lane));
      }
      if (wave < 2) {
        const RawRsrc r = raw_rsrc(sx, 4 * M);
        dma4_raw(r, lds_addr(sc_x + 64 * wave), 4 * static_cast<uint32_t>(m0 + 64 * wave + lane));
      } else if (HAS_BIAS) {
        const RawRsrc r = raw_rsrc(bias, 2 * N);
        dma4_raw(r, lds_addr(sc_b + 64 * (wave - 2)), 2 * static_cast<uint32_t>(n0 + 128 * (wave - 2) + 2 * lane));
      }
    } else if constexpr (EPI == Epilogue::kBf16) {
      const int q = wave & 3;
      if (wave < 4) {
        const RawRsrc r = raw_rsrc(sx, 4 * M);
        dma4_raw(r, lds_addr(sc_x + 64 * q), 4 * static_cast<uint32_t>(m0 + 64 * q + lane));
      } else {
        const RawRsrc r = raw_rsrc(sw, 4 * N);
        dma4_raw(r, lds_addr(sc_w + 64 * q), 4 * static_cast<uint32_t>(n0 + 64 * q + lane));
      }
      if (HAS_BIAS && wave < 2) {
        const RawRsrc r = raw_rsrc(bias, 2 * N);
        dma4_raw(r, lds_addr(sc_b + 64 * wave), 2 * static_cast<uint32_t>(n0 + 128 * wave + 2 * lane));
      }
    }
  };
  // B fragment (k-step s, band 4 wm + fm) from slot k: the 16-byte part and
  // the 8-byte part.
  auto read_b = [&](int k, int s, int fm) __attribute__((always_inline)) {
    const uint8_t* p = reinterpret_cast<const uint8_t*>(slot(k)) + (s * S::kBands + 4 * wm + fm) * kFragBytes;
    // the 8-byte part as a relaxed atomic load, which the compiler does not
    // pair with another fragment's (a paired read lands both parts apart from
    // their 16-byte parts and costs moves to join them)
    const uint64_t hi = __hip_atomic_load(reinterpret_cast<const uint64_t*>(p + 1024 + 8 * lane), __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_WAVEFRONT);
    return join(*reinterpret_cast<const v4i32*>(p + 16 * lane), __builtin_bit_cast(v2i32, hi));
  };

  // The rest of the kernel, for a wave with NFM activation bands (four in
  // the first half; tile_bands - 4 in the second).  Each count gets its own
  // straight-line code, so no branch sits between the MFMAs.
  auto run = [&](auto NFM) __attribute__((always_inline)) {
  constexpr int nfm = decltype(NFM)::value;
  v16f acc[2][4];
#pragma unroll
  for (int f = 0; f < 2; ++f)
#pragma unroll
    for (int fm = 0; fm < 4; ++fm) acc[f][fm] = v16f{};

  // The block walks one stream of stages g = i * T + t over its tiles i.
  // Loads run ahead across tile boundaries: the weights of stage g + 1 and
  // the activations of stage g + 3.  Past the block's last stage they are
  // issued anyway, for its last stage again (every address stays inside the
  // operands), which keeps the wait counts below constant.
  int cm0, cn0, xm0, xn0;  // current and next tile
  tile_at(0, &cm0, &cn0);
  if (ntiles > 1) tile_at(1, &xm0, &xn0);
  else xm0 = cm0, xn0 = cn0;
  // Tile and stage of g + k for k < 2T, clamped to the block's last stage.
  auto ahead = [&](int t, int ti, int k, int* m0, int* n0, int* st) __attribute__((always_inline)) {
    const int u = t + k;
    if (u < T) {
      *m0 = cm0, *n0 = cn0, *st = u;
    } else if (ti + 1 < ntiles) {
      *m0 = xm0, *n0 = xn0, *st = min(u - T, last);
    } else {
      *m0 = cm0, *n0 = cn0, *st = last;
    }
  };

  WRaw w0, w1;
  {
    int m0, n0, st;
    static_for<kWLoads>([&](auto PP) __attribute__((always_inline)) { load_w(w0, cn0, 0, decltype(PP)::value); });
    static_for<kDmaPerWave>([&](auto J) __attribute__((always_inline)) { issue_dma(cm0, 0, 0, decltype(J)::value); });
    ahead(0, 0, 1, &m0, &n0, &st);
    static_for<kDmaPerWave>([&](auto J) __attribute__((always_inline)) { issue_dma(m0, st, 1, decltype(J)::value); });
    ahead(0, 0, 2, &m0, &n0, &st);
    static_for<kDmaPerWave>([&](auto J) __attribute__((always_inline)) { issue_dma(m0, st, 2, decltype(J)::value); });
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * kDmaPerWave));  // DMA(0)
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  // A wave's activation fragments of a stage, (k-step s, band fm) in order
  // nfm s + fm, roll through a window of nfm register sets: fragment i is
  // read (into the set fragment i - nfm has just left) while the MFMAs of
  // fragment i - nfm run.
  v8i bq[4];
#pragma unroll
  for (int fm = 0; fm < nfm; ++fm) bq[fm] = read_b(0, 0, fm);

  // Epilogue of the current tile: lane holds column m = m0 + 128 wm + 32 fm +
  // (lane & 31) and rows n = n0 + 64 wn + 32 f + 8 j + 4 (lane >> 5) + r of
  // y^T.  Then the accumulators restart from zero.
  auto epilogue = [&]() __attribute__((always_inline)) {
    // The lane index is passed through an empty asm so that the per-lane
    // addresses below are computed here, not hoisted out of the stage loop
    // into registers the loop needs (or into scratch, whose reloads would
    // wait for every load in flight).
    int lane = threadIdx.x & 63;
    asm volatile("" : "+v"(lane));
    const int mb = cm0 + 128 * wm + (lane & 31);
    const int nl = 64 * wn + 4 * (lane >> 5);  // within the tile
    const int mlim = min(M, cm0 + tile_rows);  // rows of this tile
    const bool full = (cm0 + tile_rows <= M) && (cn0 + kFBN <= N) && (N % 4 == 0);
    if constexpr (EPI == Epilogue::kInt32) {
      int32_t* o = static_cast<int32_t*>(out);
#pragma unroll
      for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int fm = 0; fm < 4; ++fm) {
          const int m = mb + 32 * fm;
          if (fm >= nfm) continue;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int n = cn0 + nl + 32 * f + 8 * j;
            const int v0 = static_cast<int>(acc[f][fm][4 * j]), v1 = static_cast<int>(acc[f][fm][4 * j + 1]);
            const int v2 = static_cast<int>(acc[f][fm][4 * j + 2]), v3 = static_cast<int>(acc[f][fm][4 * j + 3]);
            int32_t* p = o + static_cast<int64_t>(m) * N + n;
            if (full) {
              *reinterpret_cast<int4*>(p) = make_int4(v0, v1, v2, v3);
            } else if (m < mlim) {
              if (n + 0 < N) p[0] = v0;
              if (n + 1 < N) p[1] = v1;
              if (n + 2 < N) p[2] = v2;
              if (n + 3 < N) p[3] = v3;
            }
          }
        }
    } else {
      // Through LDS: a wave's 128 x 64 outputs in two halves of 64 rows; each
      // half is written to LDS as the accumulators hold it and stored to
      // memory as whole 128-byte rows, eight rows per instruction (in a ragged
      // tile, element by element where a row runs past M or N).
      uint16_t* o = static_cast<uint16_t*>(out);
      v2u32* stg2 = reinterpret_cast<v2u32*>(stg);
      const int sbase = 512 * wave;  // the wave's area, in 16-byte units
      const bool vec = full && (N % 8 == 0);
#pragma unroll
      for (int ph = 0; ph < 2; ++ph) {
        if (2 * ph >= nfm) break;  // a short second half (a compile-time test)
#pragma unroll
        for (int f = 0; f < 2; ++f)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int c = nl + 32 * f + 8 * j;  // column within the tile
            const float4 swv = *reinterpret_cast<const float4*>(sc_w + c);
            const float swa[4] = {swv.x, swv.y, swv.z, swv.w};
            float bv[4] = {0.0f, 0.0f, 0.0f, 0.0f};
            if (HAS_BIAS) {
              if (!BIAS_TAIL || full) {
                const float2 bf = *reinterpret_cast<const float2*>(sc_b + c / 2);
                const uint32_t b0 = __float_as_uint(bf.x), b1 = __float_as_uint(bf.y);
                bv[0] = __uint_as_float(b0 << 16);
                bv[1] = __uint_as_float(b0 & 0xFFFF0000u);
                bv[2] = __uint_as_float(b1 << 16);
                bv[3] = __uint_as_float(b1 & 0xFFFF0000u);
              } else {
                // a ragged tile (with odd N the last staged pair of bias values
                // reads past the buffer as zero): straight from memory
#pragma unroll
                for (int r = 0; r < 4; ++r)
                  bv[r] = __uint_as_float(static_cast<uint32_t>(bias[min(cn0 + c + r, N - 1)]) << 16);
                // settle these loads here, in the ragged branch: otherwise the
                // wait for them lands after the branches join and, in every
                // tile, waits for all the prefetches in flight
                __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
              }
            }
#pragma unroll
            for (int fh = 0; fh < 2; ++fh) {
              const int fm = 2 * ph + fh;
              const float sxv = sc_x[128 * wm + 32 * fm + (lane & 31)];
              uint16_t h[4];
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                float v = acc[f][fm][4 * j + r];
                v = v * sxv;
                v = v * swa[r];
                if (HAS_BIAS) v = v + bv[r];
                h[r] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(v));
              }
              const int row = 32 * fh + (lane & 31);
              const int col = c - 64 * wn;  // within the wave's 64 columns
              const int chunk = (col >> 3) ^ ((row >> 1) & 7);
              stg2[2 * (sbase + 8 * row + chunk) + ((col & 7) >> 2)] =
                  v2u32{h[0] | (static_cast<uint32_t>(h[1]) << 16), h[2] | (static_cast<uint32_t>(h[3]) << 16)};
            }
          }
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int it = 0; it < 8; ++it) {
          const int row = 8 * it + (lane >> 3);
          const int c = lane & 7;
          const v4u32 vv = stg[sbase + 8 * row + (c ^ ((row >> 1) & 7))];
          const uint4 v = make_uint4(vv.x, vv.y, vv.z, vv.w);
          const int m = cm0 + 128 * wm + 64 * ph + row;
          const int n = cn0 + 64 * wn + 8 * c;
          uint16_t* p = o + static_cast<int64_t>(m) * N + n;
          if (m >= mlim) {
          } else if (vec) {
            __builtin_nontemporal_store(vv, reinterpret_cast<v4u32*>(p));
          } else {
            const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 8; ++e)
              if (n + e < N) p[e] = static_cast<uint16_t>(w[e >> 1] >> (16 * (e & 1)));
          }
        }
        __builtin_amdgcn_wave_barrier();
      }
    }
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
      for (int fm = 0; fm < 4; ++fm) acc[f][fm] = v16f{};
  };

  // One stage g = g0 + I, g0 a multiple of 6: slot I % 3 and weight set
  // I % 2, both known at compile time; t is its stage within tile ti.
  //   * At its start, the wait for this stage's weights (loaded during the
  //     previous stage's first k-step): vmcnt(kDmaPerWave) leaves in flight
  //     only the DMA issued after them (vector loads complete in order).
  //   * Then the stage's fragments j = nfm s + fm (k-step s, band fm) in
  //     turn: the two MFMAs of fragment j, the read of fragment j + nfm into
  //     the register set fragment j has left (past the stage's last
  //     fragment, those of the next stage, from the next slot), and a share
  //     of the stage's vector-memory loads, so that they reach the memory
  //     system spread over the stage rather than in one burst per wave:
  //     stage g + 1's weights (into the other set, done with at stage g - 1)
  //     among the first k-step's fragments, and the DMA of stage g + 3
  //     among the second's.
  //   * Between the k-steps, once every wave has read the whole slot
  //     (lgkmcnt(0) + barrier) and DMA(g + 1) has landed, the slot is free
  //     for that DMA (at a tile's first stage, the tile's scales are moved
  //     first).  The wait there, vmcnt(kWLoads + kDmaPerWave) = 9, leaves in
  //     flight at most the loads issued since this stage's weights (which
  //     have landed): DMA(g + 2) and stage g + 1's weights.  DMA(g + 1),
  //     issued before them, has therefore landed (the stores of an epilogue
  //     in between only add to the count).
  // After a tile's last stage comes its epilogue.
  WRaw* wset[2] = {&w0, &w1};
  int t = 0, ti = 0;
  auto stage = [&](auto I) __attribute__((always_inline)) {
    constexpr int i = decltype(I)::value;
    constexpr int cur = i % 3, nxt = (i + 1) % 3;
    int wm0, wn0, wst, dm0 = 0, dst = 0;  // the tile and stage of the weights and the DMA issued here
    ahead(t, ti, 1, &wm0, &wn0, &wst);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(kDmaPerWave));
    __builtin_amdgcn_sched_barrier(0);
    const WFrag wc = frags(*wset[i % 2]);
    static_for<2 * nfm>([&](auto J) __attribute__((always_inline)) {
      constexpr int j = decltype(J)::value;
      constexpr int ks = j / nfm, fm = j % nfm, r = j + nfm;
      acc[0][fm] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(wc.f[ks][0], bq[fm], acc[0][fm], 3, 3, 0, 127, 0,
                                                                   127);
      acc[1][fm] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(wc.f[ks][1], bq[fm], acc[1][fm], 3, 3, 0, 127, 0,
                                                                   127);
      if constexpr (r < 2 * nfm) bq[fm] = read_b(cur, 1, fm);
      else bq[fm] = read_b(nxt, 0, fm);
      if constexpr (ks == 0) {
        // weight parts pp with pp nfm / kWLoads == j
        static_for<kWLoads>([&](auto PP) __attribute__((always_inline)) {
          constexpr int pp = decltype(PP)::value;
          if constexpr (pp * nfm / kWLoads == j) load_w(*wset[(i + 1) % 2], wn0, wst, pp);
        });
      } else if constexpr (fm < kDmaPerWave) {
        issue_dma(dm0, dst, cur, fm);
      }
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (j == nfm - 1) {
        __builtin_amdgcn_s_waitcnt(kLgkm0);
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(kWLoads + kDmaPerWave));
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        if (t == 0) issue_scales(cm0, cn0);
        int dn0;
        ahead(t, ti, 3, &dm0, &dn0, &dst);
      }
    });
    // (past the block's last stage the reads of the next slot are of data
    // that is not used)
    static_assert(kDmaPerWave <= 3, "the DMA parts go with the second k-step's fragments");
    __builtin_amdgcn_sched_barrier(0);
    if (t == last) {
      if (T == 1) {
        // the scales were moved at this very stage
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
        __builtin_amdgcn_s_barrier();
      }
      epilogue();
      ++ti;
      t = 0;
      cm0 = xm0, cn0 = xn0;
      if (ti + 1 < ntiles) tile_at(ti + 1, &xm0, &xn0);
    } else {
      ++t;
    }
  };
  const int G = ntiles * T;
  for (int g = 0; g < G; g += 6) {
    stage(std::integral_constant<int, 0>{});
#define JQ_F6_NEXT(N) \
    if (g + N < G) stage(std::integral_constant<int, N>{});
    JQ_F6_NEXT(1) JQ_F6_NEXT(2) JQ_F6_NEXT(3) JQ_F6_NEXT(4) JQ_F6_NEXT(5)
#undef JQ_F6_NEXT
  }
  // no load may still be writing LDS or registers when the wave ends
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  };
  if (wm == 0 || tile_bands == 8) run(std::integral_constant<int, 4>{});
  else run(std::integral_constant<int, 3>{});
}

// ---------------------------------------------------------------------------
// Group-wise GEMM on BF6 operands
//
// S[m,n] = sum over the groups g in k order of fl32(fl32(acc_g * s_x[m,g]) *
// s_w[n,g]), acc_g the exact integer product over the G codes of group g (a
// single k-step for G = 64, two for G = 128), then y = bf16(S + bias) (or S
// itself, EPI kF32).  The matrix cores deliver acc_g in fp32, exactly, so the
// fold after each group is two multiplies and an add per output: the kernel
// is bound by that vector arithmetic, not by the MFMAs.
//
// Block tile 128 (m) x 128 (n), four waves, two blocks per CU; wave (wm, wn)
// owns activation bands 2wm, 2wm + 1 and weight bands 2wn, 2wn + 1 of the
// tile: 2 x 2 tiles of 32x32, 64 fp32 sums per lane.  A stage is 128 codes of
// K: both operands' fragments (activation layout and weight layout, 12 KiB
// each) and the stage's scales (s_x and s_w of its groups, gathered from the
// [rows, K/G] arrays by 4-byte transfers) move into LDS by buffer_load ...
// lds, issued as instructions of their own two stages ahead into a ring of
// three slots.  A stage waits only for its own loads (vmcnt counts the next
// stage's as still in flight) and then meets the other waves at a barrier
// with no memory fence, after which the slot read two stages ago takes the
// loads of the stage two ahead.  Operand bands, rows or columns past M or N
// read as zero (outside the buffers).
template <int G, Epilogue EPI, bool HAS_BIAS>
__global__ __launch_bounds__(256, 2) void w4a4g_f6_gemm_kernel(
    const uint8_t* __restrict__ xf6, const float* __restrict__ sx, int M, int mbands,
    const uint8_t* __restrict__ wf6, const float* __restrict__ sw, int N, int nbands, int ksteps, int KG,
    const uint16_t* __restrict__ bias, void* __restrict__ out, int tiles_m, int tiles_n) {
  constexpr int kGps = 128 / G;                    // groups per stage
  constexpr int kOpU4 = 4 * 2 * kFragBytes / 16;   // one operand's stage: 4 bands x 3072 bytes
  constexpr int kScF = 2 * kGps * 128;             // one stage's scales: s_x then s_w, [group][row]
  constexpr int kScDma = kScF / 64 / 4;            // 4-byte scale transfers per wave per stage
  constexpr int kLoads = 6 + kScDma;               // vector-memory instructions per wave per stage
  // Three slots, each the operand fragments of a stage (activations, then
  // weights) and its scales.  The transfers are asm the compiler does not
  // track, so the slot may be computed at run time.
  __shared__ uint4 ops[3 * 2 * kOpU4];
  __shared__ float scs[3 * kScF];
  auto opk = [&](int k) __attribute__((always_inline)) { return ops + 2 * kOpU4 * k; };
  auto sck = [&](int k) __attribute__((always_inline)) { return scs + kScF * k; };

  TileCoord tc;
  if (!tile_of_block(blockIdx.x, tiles_m, tiles_n, &tc)) return;
  const int m0 = 128 * tc.tm, n0 = 128 * tc.tn;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int T = ksteps / 2;
  const uint32_t band_bytes = static_cast<uint32_t>(ksteps) * kFragBytes;

  const RawRsrc rsx = raw_rsrc(xf6, static_cast<uint32_t>(static_cast<int64_t>(mbands) * band_bytes));
  const RawRsrc rsw = raw_rsrc(wf6, static_cast<uint32_t>(static_cast<int64_t>(nbands) * band_bytes));
  const RawRsrc rssx = raw_rsrc(sx, static_cast<uint32_t>(4 * static_cast<int64_t>(M) * KG));
  const RawRsrc rssw = raw_rsrc(sw, static_cast<uint32_t>(4 * static_cast<int64_t>(N) * KG));

  // Operand DMA: the 12 KiB of a stage are 12 instructions of 1 KiB, three
  // per wave; instruction i = 3 wave + j is part i % 3 of band i / 3.  Bands
  // past the operand read as zero.
  uint32_t xoff[3], woff[3];
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    const int i = 3 * wave + j;
    const int b = i / 3, part = i % 3;
    const int xb = m0 / 32 + b, wb = n0 / 32 + b;
    xoff[j] = xb < mbands ? static_cast<uint32_t>(xb) * band_bytes + 1024 * part + 16 * lane : kOutside;
    woff[j] = wb < nbands ? static_cast<uint32_t>(wb) * band_bytes + 1024 * part + 16 * lane : kOutside;
  }
  // Scale DMA: entry e of a stage's kScF (s_x entries, then s_w) is group
  // e % (kGps 128) / 128 of row (column) e % 128 of the tile; instruction
  // i = kScDma wave + j moves entries 64 i .. 64 i + 63, all of one array.
  // Per lane: the array's row and the group within the stage; entries past
  // M or N read as zero.
  int sc_row[kScDma], sc_gl[kScDma];
  bool sc_w[kScDma];  // wave-uniform: whether instruction j moves s_w entries
#pragma unroll
  for (int j = 0; j < kScDma; ++j) {
    sc_w[j] = 64 * (kScDma * wave + j) >= kGps * 128;
    const int ee = (64 * (kScDma * wave + j) + lane) % (kGps * 128);
    sc_gl[j] = ee / 128;
    sc_row[j] = (sc_w[j] ? n0 : m0) + ee % 128;
  }
  auto issue = [&](int u, int k) __attribute__((always_inline)) {
    const uint32_t xa = lds_addr(opk(k)), wa = lds_addr(opk(k) + kOpU4);
    const uint32_t so = 2 * kFragBytes * u;
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      dma16_raw(rsx, xa + 16 * 64 * (3 * wave + j), xoff[j], so);  // kOutside + so stays outside
      dma16_raw(rsw, wa + 16 * 64 * (3 * wave + j), woff[j], so);
    }
#pragma unroll
    for (int j = 0; j < kScDma; ++j) {
      const int g = kGps * u + sc_gl[j];
      const bool in = sc_row[j] < (sc_w[j] ? N : M) && g < KG;
      const uint32_t off = in ? 4u * static_cast<uint32_t>(sc_row[j] * KG + g) : kOutside;
      const uint32_t dst = lds_addr(sck(k) + 64 * (kScDma * wave + j));
      if (sc_w[j]) dma4_raw(rssw, dst, off);
      else dma4_raw(rssx, dst, off);
    }
  };

  v16f S[2][2];  // [weight band f][activation band fb]
#pragma unroll
  for (int f = 0; f < 2; ++f)
#pragma unroll
    for (int fb = 0; fb < 2; ++fb) S[f][fb] = v16f{};

  // Fold one group into the sums: lane holds column m = 32 (2wm + fb) +
  // (lane & 31) and rows n = 32 (2wn + f) + 8 j + 4 (lane >> 5) + r of y^T,
  // with the lane's scales of the stage read from its scale slot.
  float xsr[kGps][2];
  float4 wsr[kGps][2][4];
  auto read_scales = [&](int k) __attribute__((always_inline)) {
#pragma unroll
    for (int gl = 0; gl < kGps; ++gl)
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        xsr[gl][b] = sck(k)[128 * gl + 32 * (2 * wm + b) + (lane & 31)];
#pragma unroll
        for (int j = 0; j < 4; ++j)
          wsr[gl][b][j] = *reinterpret_cast<const float4*>(sck(k) + kGps * 128 + 128 * gl + 32 * (2 * wn + b) +
                                                           8 * j + 4 * (lane >> 5));
      }
  };
  auto fold = [&](const v16f& acc, int f, int fb, int gl) __attribute__((always_inline)) {
    const float xs = xsr[gl][fb];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float wsa[4] = {wsr[gl][f][j].x, wsr[gl][f][j].y, wsr[gl][f][j].z, wsr[gl][f][j].w};
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float t = acc[4 * j + r] * xs;
        t = t * wsa[r];
        S[f][fb][4 * j + r] = S[f][fb][4 * j + r] + t;
      }
    }
  };
  auto read_x = [&](int k, int t, int fb) __attribute__((always_inline)) {
    const uint8_t* p = reinterpret_cast<const uint8_t*>(opk(k)) + (2 * wm + fb) * 2 * kFragBytes + t * kFragBytes;
    return join(*reinterpret_cast<const v4i32*>(p + 16 * lane), *reinterpret_cast<const v2i32*>(p + 1024 + 8 * lane));
  };
  auto read_w = [&](int k, int t, int f) __attribute__((always_inline)) {
    const uint8_t* p = reinterpret_cast<const uint8_t*>(opk(k) + kOpU4) + (2 * wn + f) * 2 * kFragBytes;
    if (t == 0) {
      const v4i32 a = *reinterpret_cast<const v4i32*>(p + 16 * lane);
      const v2i32 b = *reinterpret_cast<const v2i32*>(p + 1024 + 16 * lane);
      return v8i{a.x, a.y, a.z, a.w, b.x, b.y, 0, 0};
    }
    const v2i32 a = *reinterpret_cast<const v2i32*>(p + 1024 + 16 * lane + 8);
    const v4i32 b = *reinterpret_cast<const v4i32*>(p + 2048 + 16 * lane);
    return v8i{a.x, a.y, b.x, b.y, b.z, b.w, 0, 0};
  };

  // Stage u from slot (xa, wa, sxa, swa): the stage's loads have landed
  // and every wave has passed the barrier after them.
  auto compute = [&](int u, int k) __attribute__((always_inline)) {
    if constexpr (G == 64) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        if (kGps * u + t >= KG) break;  // K % 128 == 64: the last stage's second half is padding
        const v8i b0 = read_x(k, t, 0), b1 = read_x(k, t, 1);
#pragma unroll
        for (int f = 0; f < 2; ++f) {
          const v8i a = read_w(k, t, f);
          const v16f c0 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b0, v16f{}, 3, 3, 0, 127, 0, 127);
          const v16f c1 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b1, v16f{}, 3, 3, 0, 127, 0, 127);
          fold(c0, f, 0, t);
          fold(c1, f, 1, t);
        }
      }
    } else {
      const v8i b00 = read_x(k, 0, 0), b01 = read_x(k, 0, 1);
      const v8i b10 = read_x(k, 1, 0), b11 = read_x(k, 1, 1);
#pragma unroll
      for (int f = 0; f < 2; ++f) {
        const v8i a0 = read_w(k, 0, f), a1 = read_w(k, 1, f);
        v16f c0 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a0, b00, v16f{}, 3, 3, 0, 127, 0, 127);
        v16f c1 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a0, b01, v16f{}, 3, 3, 0, 127, 0, 127);
        c0 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a1, b10, c0, 3, 3, 0, 127, 0, 127);
        c1 = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a1, b11, c1, 3, 3, 0, 127, 0, 127);
        fold(c0, f, 0, 0);
        fold(c1, f, 1, 0);
      }
    }
  };

  // Stage u from slot u % 3: wait for its loads (those of stage u + 1, issued
  // after them, may still be in flight: vector loads complete in order),
  // meet the other waves (every wave is then also done with slot (u - 1) % 3,
  // read at the previous stage), issue stage u + 2 into that slot, compute.
  issue(0, 0);
  if (T > 1) issue(1, 1);
  for (int u = 0; u < T; ++u) {
    const int k = u % 3;
    if (u + 1 < T) __builtin_amdgcn_s_waitcnt(vmcnt_imm(kLoads));
    else __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    __builtin_amdgcn_s_barrier();
    // no LDS read of the slot may be moved above the wait and the barrier
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    if (u + 2 < T) issue(u + 2, (u + 2) % 3);
    read_scales(k);
    compute(u, k);
  }

  if constexpr (EPI == Epilogue::kF32) {
    // S as it is (the checking path): four consecutive n per store.
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int n = n0 + 32 * (2 * wn + f) + 8 * j + 4 * (lane >> 5);
#pragma unroll
        for (int fb = 0; fb < 2; ++fb) {
          const int m = m0 + 32 * (2 * wm + fb) + (lane & 31);
          if (m >= M) continue;
          float* p = static_cast<float*>(out) + static_cast<int64_t>(m) * N + n;
          if (n + 3 < N && N % 4 == 0) {
            *reinterpret_cast<float4*>(p) =
                make_float4(S[f][fb][4 * j], S[f][fb][4 * j + 1], S[f][fb][4 * j + 2], S[f][fb][4 * j + 3]);
          } else {
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (n + r < N) p[r] = S[f][fb][4 * j + r];
          }
        }
      }
  } else {
    // bf16(S + bias), staged through LDS (the first slot, free once every
    // wave is past the last stage) and stored as whole 128-byte rows: per
    // wave two passes of 32 rows x 64 columns, 16-byte chunk c of row r at
    // chunk c ^ ((r >> 1) & 7).
    __syncthreads();
    v4u32* stg = reinterpret_cast<v4u32*>(ops) + 256 * wave;
    v2u32* stg2 = reinterpret_cast<v2u32*>(stg);
    float bv[2][4][4];
#pragma unroll
    for (int f = 0; f < 2; ++f)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int n = n0 + 32 * (2 * wn + f) + 8 * j + 4 * (lane >> 5) + r;
          bv[f][j][r] = HAS_BIAS ? __uint_as_float(static_cast<uint32_t>(bias[min(n, N - 1)]) << 16) : 0.0f;
        }
    const bool vec = (n0 + 128 <= N) && (N % 8 == 0);
#pragma unroll
    for (int fb = 0; fb < 2; ++fb) {
      const int row = lane & 31;
#pragma unroll
      for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int c = 32 * f + 8 * j + 4 * (lane >> 5);  // column within the wave's 64
          uint16_t h[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            float v = S[f][fb][4 * j + r];
            if (HAS_BIAS) v = v + bv[f][j][r];
            h[r] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(v));
          }
          stg2[2 * (8 * row + ((c >> 3) ^ ((row >> 1) & 7))) + ((c & 7) >> 2)] =
              v2u32{h[0] | (static_cast<uint32_t>(h[1]) << 16), h[2] | (static_cast<uint32_t>(h[3]) << 16)};
        }
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int it = 0; it < 4; ++it) {
        const int rr = 8 * it + (lane >> 3), ch = lane & 7;
        const v4u32 vv = stg[8 * rr + (ch ^ ((rr >> 1) & 7))];
        const int m = m0 + 32 * (2 * wm + fb) + rr;
        const int n = n0 + 64 * wn + 8 * ch;
        uint16_t* p = static_cast<uint16_t*>(out) + static_cast<int64_t>(m) * N + n;
        if (m >= M) {
        } else if (vec) {
          __builtin_nontemporal_store(vv, reinterpret_cast<v4u32*>(p));
        } else {
          const uint32_t w[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (n + e < N) p[e] = static_cast<uint16_t>(w[e >> 1] >> (16 * (e & 1)));
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
  }
}

// Four rows per block, W waves of 16 group slots, NJ sets of groups each.
template <int NJ, int G>
hipError_t launch_q4f6(const uint16_t* x, int64_t M, int64_t K, int64_t ksteps, uint8_t* out, float* s, int waves,
                       hipStream_t st) {
  const int64_t rows_padded = (M + 31) / 32 * 32;
  const int64_t groups_of_8_bands = (rows_padded / 32 + kNumXcd - 1) / kNumXcd;
  const dim3 grid(static_cast<unsigned>(groups_of_8_bands * 8 * kNumXcd));
  const size_t lds = static_cast<size_t>(waves) * 256 * 16;
  hipLaunchKernelGGL((quantize_rows4_f6_kernel<NJ, G>), grid, dim3(64 * waves), lds, st, x, M, K, rows_padded, ksteps,
                     out, s);
  return hipGetLastError();
}

template <int NJ, int G>
hipError_t launch_qf6(const uint16_t* x, int64_t M, int64_t K, int64_t ksteps, uint8_t* out, float* s, int threads,
                      hipStream_t st) {
  const int64_t rows_padded = (M + 31) / 32 * 32;
  const int64_t groups_of_8_bands = (rows_padded / 32 + kNumXcd - 1) / kNumXcd;
  const dim3 grid(static_cast<unsigned>(groups_of_8_bands * 32 * kNumXcd));
  const size_t lds = static_cast<size_t>(threads / 64) * 256 * 16;
  hipLaunchKernelGGL((quantize_rows_f6_kernel<NJ, G>), grid, dim3(threads), lds, st, x, M, K, rows_padded, ksteps, out, s);
  return hipGetLastError();
}

}  // namespace

int64_t f6_ksteps(int64_t K) { return (K + 127) / 128 * 2; }

int64_t f6_operand_bytes(int64_t rows, int64_t K) { return (rows + 31) / 32 * f6_ksteps(K) * kFragBytes; }

// Tile height of the GEMM in bands of 32 rows (7 or 8).  Every tile costs its
// height in MFMA work plus about one band's worth of fixed work (the weight
// fragments, the epilogue); the blocks of an XCD take its tiles in rounds.
// The height with the cheapest rounds wins, the taller one on ties: at
// 9216 x 3072 on 256 CUs, 224-row tiles give 504 tiles in two rounds where
// 256-row tiles give 432, which also take two rounds.
int f6_tile_bands(int64_t M, int64_t N, int64_t slots) {
  const int64_t tiles_n = (N + kFBN - 1) / kFBN;
  const int64_t per_xcd_slots = std::max<int64_t>(1, slots / kNumXcd);
  int best = 8;
  int64_t best_cost = -1;
  for (int b = 8; b >= 7; --b) {
    const int64_t tiles = (M + 32 * b - 1) / (32 * b) * tiles_n;
    const int64_t per_xcd = (tiles + kNumXcd - 1) / kNumXcd;
    const int64_t rounds = (per_xcd + per_xcd_slots - 1) / per_xcd_slots;
    const int64_t cost = rounds * (b + 1);
    if (best_cost < 0 || cost < best_cost) best = b, best_cost = cost;
  }
  return best;
}

// Block shape of the GEMM.  One 8-wave block per CU on 224- or 256-row tiles
// re-reads the operands least, and wins when 256-row tiles cover M exactly
// or K is long.  Otherwise two 4-wave blocks per CU on 128-row tiles win:
// 224-row tiles save less than their missing band (the wave that holds three
// bands waits on the one beside it that holds four), and with short K a
// tile's epilogue is a large share of its time, which the other block's
// MFMAs fill.  Measured over M 1024..9216, K 2048..12288, N 3072..12288.
int f6_block_waves(int64_t M, int64_t N, int64_t K, int64_t slots) {
  return K > kShortK || f6_tile_bands(M, N, slots) == 8 ? 8 : 4;
}

template <int G>
hipError_t launch_quantize_f6(const uint16_t* x, int64_t M, int64_t K, uint8_t* out, float* scale, hipStream_t st) {
  const int64_t ksteps = f6_ksteps(K);
  const int64_t groups = 2 * ksteps;
  if (groups <= 512) {
    // four rows per block: up to 8 waves of 16 group slots, NJ <= 4 sets each
    const int64_t waves = std::min<int64_t>(8, (groups + 15) / 16);
    const int64_t nj = (groups + 16 * waves - 1) / (16 * waves);
    const int w = static_cast<int>(waves);
    if (nj <= 1) return launch_q4f6<1, G>(x, M, K, ksteps, out, scale, w, st);
    if (nj <= 2) return launch_q4f6<2, G>(x, M, K, ksteps, out, scale, w, st);
    if (nj <= 3) return launch_q4f6<3, G>(x, M, K, ksteps, out, scale, w, st);
    return launch_q4f6<4, G>(x, M, K, ksteps, out, scale, w, st);
  }
  // longer rows: one row per block, up to 512 threads each holding NJ groups
  const int64_t threads = 512;
  const int64_t nj = (groups + threads - 1) / threads;
  const int th = static_cast<int>(threads);
  if (nj <= 2) return launch_qf6<2, G>(x, M, K, ksteps, out, scale, th, st);
  return launch_qf6<4, G>(x, M, K, ksteps, out, scale, th, st);
}

hipError_t launch_quantize_rows_f6(const uint16_t* x, int64_t M, int64_t K, uint8_t* out, float* scale,
                                   hipStream_t st) {
  return launch_quantize_f6<0>(x, M, K, out, scale, st);
}

hipError_t launch_quantize_rows_f6_batch(int count, const uint16_t* const* x, const int64_t* M, const int64_t* K,
                                         uint8_t* const* out, float* const* scale, hipStream_t st) {
  // Inputs whose rows fit the four-rows-per-block kernel (at most 512 groups)
  // share one launch: its waves are the most any of them needs, and NJ the
  // most sets of groups any of them needs at that wave count.  Longer rows get
  // a launch of their own, on the same stream.
  Q4Batch b{};
  int waves = 1;
  for (int i = 0; i < count; ++i) {
    const int64_t groups = 2 * f6_ksteps(K[i]);
    if (groups <= 512) waves = static_cast<int>(std::max<int64_t>(waves, std::min<int64_t>(8, (groups + 15) / 16)));
  }
  int NJ = 1;
  int64_t first = 0;
  for (int i = 0; i < count; ++i) {
    const int64_t ksteps = f6_ksteps(K[i]);
    const int64_t groups = 2 * ksteps;
    if (groups > 512) {
      const hipError_t e = launch_quantize_f6<0>(x[i], M[i], K[i], out[i], scale[i], st);
      if (e != hipSuccess) return e;
      continue;
    }
    Q4Input& q = b.in[b.count++];
    q.x = x[i];
    q.out = out[i];
    q.scale = scale[i];
    q.M = M[i];
    q.K = K[i];
    q.rows_padded = (M[i] + 31) / 32 * 32;
    q.ksteps = ksteps;
    q.first = first;
    q.nj = static_cast<int>((groups + 16 * waves - 1) / (16 * waves));
    NJ = std::max(NJ, q.nj);
    first += (q.rows_padded / 32 + kNumXcd - 1) / kNumXcd * 8 * kNumXcd;  // as launch_q4f6's grid
  }
  if (b.count == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>(first));
  const size_t lds = static_cast<size_t>(waves) * 256 * 16;
#define JQ_Q4B(NN) hipLaunchKernelGGL((quantize_rows4_f6_batch_kernel<NN>), grid, dim3(64 * waves), lds, st, b)
  if (NJ <= 1) JQ_Q4B(1);
  else if (NJ <= 2) JQ_Q4B(2);
  else if (NJ <= 3) JQ_Q4B(3);
  else JQ_Q4B(4);
#undef JQ_Q4B
  return hipGetLastError();
}

hipError_t launch_quantize_groups_f6(const uint16_t* x, int64_t M, int64_t K, int G, uint8_t* out, float* scale,
                                     hipStream_t st) {
  return G == 64 ? launch_quantize_f6<64>(x, M, K, out, scale, st) : launch_quantize_f6<128>(x, M, K, out, scale, st);
}

hipError_t launch_w4a4g_f6_gemm(Epilogue epi, const uint8_t* xf6, const float* sx, int64_t M, int64_t K, int G,
                                const uint8_t* wf6, const float* sw, int64_t N, const uint16_t* bias, void* out,
                                hipStream_t st) {
  const int ksteps = static_cast<int>(f6_ksteps(K));
  const int tiles_m = static_cast<int>((M + 127) / 128), tiles_n = static_cast<int>((N + 127) / 128);
  const int64_t tiles = static_cast<int64_t>(tiles_m) * tiles_n;
  const unsigned blocks = static_cast<unsigned>((tiles + kNumXcd - 1) / kNumXcd * kNumXcd);
  const int mbands = static_cast<int>((M + 31) / 32), nbands = static_cast<int>((N + 31) / 32);
  const int KG = static_cast<int>(K / G);
  const int Mi = static_cast<int>(M), Ni = static_cast<int>(N);
#define JQ_F6G(GG, E, B)                                                                                       \
  hipLaunchKernelGGL((w4a4g_f6_gemm_kernel<GG, E, B>), dim3(blocks), dim3(256), 0, st, xf6, sx, Mi, mbands, wf6, \
                     sw, Ni, nbands, ksteps, KG, bias, out, tiles_m, tiles_n)
  if (G == 64) {
    if (epi == Epilogue::kF32) JQ_F6G(64, Epilogue::kF32, false);
    else if (bias != nullptr) JQ_F6G(64, Epilogue::kBf16, true);
    else JQ_F6G(64, Epilogue::kBf16, false);
  } else {
    if (epi == Epilogue::kF32) JQ_F6G(128, Epilogue::kF32, false);
    else if (bias != nullptr) JQ_F6G(128, Epilogue::kBf16, true);
    else JQ_F6G(128, Epilogue::kBf16, false);
  }
#undef JQ_F6G
  return hipGetLastError();
}

hipError_t launch_int4_to_f6(const uint8_t* q, int64_t rows, int64_t K, uint8_t* out, bool weight_layout,
                             bool ternary, hipStream_t st) {
  const int64_t ksteps = f6_ksteps(K);
  const int64_t rows_padded = (rows + 31) / 32 * 32;
  const int64_t total = rows_padded * 2 * ksteps;
  const dim3 grid(static_cast<unsigned>((total + 255) / 256));
#define JQ_CVT(W, T) hipLaunchKernelGGL((int4_to_f6_kernel<W, T>), grid, dim3(256), 0, st, q, rows, rows_padded, K, ksteps, out)
  if (ternary) {
    if (weight_layout) JQ_CVT(true, true);
    else JQ_CVT(false, true);
  } else {
    if (weight_layout) JQ_CVT(true, false);
    else JQ_CVT(false, false);
  }
#undef JQ_CVT
  return hipGetLastError();
}

hipError_t launch_w4a4_f6_gemm(Epilogue epi, const uint8_t* xf6, const float* sx, int64_t M, int64_t K,
                               const uint8_t* wf6, const float* sw, int64_t N, const uint16_t* bias, void* out,
                               hipStream_t st) {
  // Block slots: one 8-wave block or two 4-wave blocks per CU (a block's
  // registers fill half or all of the CU); each block walks its tiles in turn.
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const int ksteps = static_cast<int>(f6_ksteps(K));
  const int64_t slots = std::max<int64_t>(kNumXcd, cus / kNumXcd * kNumXcd);
  const int waves = f6_block_waves(M, N, K, slots);
  const int tile_bands = waves == 4 ? 4 : f6_tile_bands(M, N, slots);
  const int tiles_m = static_cast<int>((M + 32 * tile_bands - 1) / (32 * tile_bands));
  const int tiles_n = static_cast<int>((N + kFBN - 1) / kFBN);
  const int64_t T = static_cast<int64_t>(tiles_m) * tiles_n;
  const int64_t per_xcd = (T + kNumXcd - 1) / kNumXcd;
  const int64_t block_slots = (8 / waves) * slots;
  const int blocks =
      static_cast<int>(ksteps / 2 < 3 ? per_xcd * kNumXcd : std::min<int64_t>(per_xcd * kNumXcd, block_slots));
  const int mbands = static_cast<int>((M + 31) / 32);
  const int nbands = static_cast<int>((N + 31) / 32);
  const int Mi = static_cast<int>(M), Ni = static_cast<int>(N);
#define JQ_F6(W, E, B, BT)                                                                                   \
  hipLaunchKernelGGL((w4a4_f6_gemm_kernel<W, E, B, BT>), dim3(blocks), dim3(64 * W), 0, st, xf6, sx, Mi, mbands, \
                     wf6, sw, Ni, nbands, ksteps, bias, out, tile_bands, tiles_m, tiles_n, blocks)
#define JQ_F6_EPI(W)                                                      \
  if (epi == Epilogue::kInt32) JQ_F6(W, Epilogue::kInt32, false, false);  \
  else if (bias != nullptr && (N & 1)) JQ_F6(W, Epilogue::kBf16, true, true); \
  else if (bias != nullptr) JQ_F6(W, Epilogue::kBf16, true, false);      \
  else JQ_F6(W, Epilogue::kBf16, false, false);
  if (waves == 4) {
    JQ_F6_EPI(4)
  } else {
    JQ_F6_EPI(8)
  }
#undef JQ_F6_EPI
#undef JQ_F6
  return hipGetLastError();
}


// ---------------------------------------------------------------------------
// Library-held scratch of the allocation-free entry point
// (jq_w4a4_f6_linear_noalloc): the BF6 activation operand and the scales of
// one call, JQ_NOALLOC_SCRATCH_BYTES at most.  Each device the library runs
// on holds its own copy until the process ends.  In host code the name is
// only a handle for hipGetSymbolAddress; kernels get the device address it
// returns, as they get a workspace.

static __device__ __align__(256) uint8_t scratch[JQ_NOALLOC_SCRATCH_BYTES];

hipError_t noalloc_scratch(void** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    // once per device, with that device current
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

}  // namespace jq
