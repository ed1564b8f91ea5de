// Packed-int4 x packed-int4 GEMM with int32 accumulation and a fused
// dequantising epilogue, hand-written for gfx950 (CDNA4) int8 MFMA.
//
// Operation (Sec. 3.1 low-bit operator; appendix FAQ Q7 low-bit matrix
// multiplication):  acc[m,n] = sum_k qx[m,k] * qw[n,k]  on int4 codes, then
//   y[m,n] = bf16_rne(((fp32(acc) * sx[m]) * sw[n]) + bias[n])
// with every fp32 operation rounded on its own (built with -ffp-contract=off).
//
// Structure.
//  * Block tile 128 (m) x 256 (n), four waves of 64 x 128 outputs each (a
//    4 x 8 grid of 16 x 16 MFMA tiles, 128 int32 accumulators per lane).  A
//    block needs 64 KiB of LDS and at most 256 registers per lane, so two
//    blocks share a CU and each SIMD runs two waves from different blocks:
//    while one block waits at its barrier or on LDS, the other issues MFMAs.
//    Where 128-row tiles would leave the last round of blocks mostly empty
//    (FLUX MLP-down: 864 tiles over 512 slots), the launcher takes 112-row
//    tiles instead (seven fragments of 16 rows; 996 tiles, two full rounds).
//  * gfx950 has no int4 MFMA, so codes are widened to int8 for
//    v_mfma_i32_16x16x64_i8.  Widening is VALU work, and VALU instructions
//    between MFMAs slow the matrix pipe of the SIMD (measured with two waves
//    per SIMD: 1.5 and 2.25 VALU per MFMA cost 16% and 34% of the MFMA rate).
//    The activation tile is therefore widened once per block: it is loaded
//    into registers, widened, and written to LDS as int8, and the waves read
//    ready-to-use operands.  The weight tile (twice as many rows) stays packed
//    in LDS and each wave widens its own fragments.  That is ~1.7 VALU per
//    MFMA instead of 2.25, within the LDS budget of two blocks per CU.
//  * Widening without sign extension: hi = p & 0xF0F0F0F0 and
//    lo = (p << 4) & 0xF0F0F0F0 hold 16 * code as int8.  A packed dword of
//    codes k0..k7 becomes [k0 k2 k4 k6] and [k1 k3 k5 k7]; both operands are
//    widened in the same order, so every MFMA sees the same k permutation on
//    A and B and the sum is unchanged.  The accumulator holds 256 * acc
//    exactly (|256 * acc| <= 2^30 for K <= 65536); the epilogue shifts back.
//  * K is consumed 128 codes (64 packed bytes per row) per stage, two stages
//    alternating.  The weight tile moves from global memory straight into LDS
//    with buffer_load_dwordx4 ... lds (no staging registers, no LDS write
//    instructions), one stage ahead.  Weight LDS rows are 64 bytes: 16-byte
//    chunk c of row r sits at slot c ^ ((r >> 1) & 3), realised by choosing,
//    for each lane, the global chunk that belongs in its (lane-ordered) DMA
//    slot.  Activation LDS rows are 128 bytes of int8: chunk c of row r sits
//    at c ^ (r & 7).  Either way a ds_read_b128 of one chunk per lane spreads
//    8 consecutive lanes over 8 rows and all banks.
//  * Lane group g (lanes 16g..16g+15) takes, in MFMA half-stage h, codes
//    32g + 16h .. 32g + 16h + 15 of its row: bytes 8h..8h+7 of packed weight
//    chunk g, and int8 activation chunk 2g + h.
//  * Per stage: read this stage's fragments, start the weight DMA and the
//    activation loads of the next stage, 64 MFMAs (each weight fragment is
//    widened just before its four MFMAs), wait, widen and write the next
//    activation tile, barrier.  The loop body is one stage over a
//    parity-selected LDS buffer (no unrolling), which keeps the register
//    allocation free of rotating copies.
//  * The weight tile is the MFMA A operand and the activation tile the B
//    operand, so the result is y^T: each lane ends up with 4 consecutive
//    output columns n of one row m, stored as one 8-byte bf16 write.
//  * Blocks are dispatched round-robin over the 8 XCDs; each XCD is given a
//    contiguous range of tiles in a grouped (GROUP_M m-tiles per n sweep)
//    order, so tiles that share operand rows run under the same L2.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <initializer_list>

#include "gemm_common.h"
#include "jq_internal.h"

namespace jq {

namespace {

using namespace gemm_detail;

typedef unsigned v4u32 __attribute__((ext_vector_type(4)));
typedef unsigned v2u32 __attribute__((ext_vector_type(2)));

constexpr int kBN = 256;       // weight rows per block
constexpr int kWN = 64;        // per-wave tile: all activation rows of the block, a quarter of the weight rows
constexpr int kFN = kWN / 16;
constexpr int kXLoads = 2;     // 16-byte activation loads per thread per stage (rows r and r + 64)

static_assert(128 * kChunks / kThreads == kXLoads, "activation staging assumes at most two loads per thread");

// Weight formats.  kInt4: codes -8..7, two per byte (the W4A4 layer).
// kTernary: codes -1..1, four per byte as 2-bit fields (the W1.58A4 layer).
// Per stage (128 codes of K) a weight row holds kWChunks 16-byte chunks; one
// DMA instruction fills kDmaRows tile rows; kShift undoes the operand
// scaling (activations enter the MFMA as 16 * code, int4 weights as 16 * code,
// ternary weights as 64 * code).
template <WeightFormat WF>
struct WTraits {
  static constexpr bool kTern = WF == WeightFormat::kTernary;
  static constexpr int kWChunks = kTern ? 2 : 4;
  static constexpr int kStageBytes = 16 * kWChunks;
  static constexpr int kDmaRows = 64 / kWChunks;
  static constexpr int kDma = kWN / kDmaRows;          // weight DMA instructions per wave per stage
  static constexpr int kShift = kTern ? 10 : 8;
  static constexpr int kUnpackValu = kTern ? 7 : 6;    // VALU instructions per widened weight fragment
};

// Ternary weight rows are 32 bytes (two chunks); rows 8..15 of every 16 swap
// their chunks, so the 32 lanes of a ds_read_b64 half cover all 64 banks.
__device__ __forceinline__ int wt_slot(int row, int c) { return row * 2 + (c ^ ((row >> 3) & 1)); }

// Widen 16 ternary codes (one packed dword, code i in bits 2i .. 2i+1) to
// int8 64 * code: dword d, byte b of the result holds code 4b + d.  Shifting
// a 2-bit field to the top of its byte sign-extends it for free.
__device__ __forceinline__ v4i unpack_tern(uint32_t p) {
  v4i r;
  r[0] = static_cast<int>((p << 6) & 0xC0C0C0C0u);
  r[1] = static_cast<int>((p << 4) & 0xC0C0C0C0u);
  r[2] = static_cast<int>((p << 2) & 0xC0C0C0C0u);
  r[3] = static_cast<int>(p & 0xC0C0C0C0u);
  return r;
}

// Widen 16 int4 activation codes (p0: codes 0..7, p1: codes 8..15) into the
// order unpack_tern produces: dword d, byte b = 16 * code 4b + d.
__device__ __forceinline__ v4i unpack8_tern_order(uint32_t p0, uint32_t p1) {
  const v4i e = unpack8(p0, p1);  // e[0] = codes 0 2 4 6, e[1] = 1 3 5 7, e[2] = 8 10 12 14, e[3] = 9 11 13 15
  v4i r;
  // v_perm_b32: selector byte values 0..3 pick the second operand's bytes, 4..7 the first's.
  r[0] = static_cast<int>(__builtin_amdgcn_perm(static_cast<uint32_t>(e[2]), static_cast<uint32_t>(e[0]), 0x06040200u));
  r[1] = static_cast<int>(__builtin_amdgcn_perm(static_cast<uint32_t>(e[3]), static_cast<uint32_t>(e[1]), 0x06040200u));
  r[2] = static_cast<int>(__builtin_amdgcn_perm(static_cast<uint32_t>(e[2]), static_cast<uint32_t>(e[0]), 0x07050301u));
  r[3] = static_cast<int>(__builtin_amdgcn_perm(static_cast<uint32_t>(e[3]), static_cast<uint32_t>(e[1]), 0x07050301u));
  return r;
}

// BM: activation rows per block tile, 128 or 112 (seven 16-row fragments,
// for shapes whose 128-row tiles leave the last round of blocks mostly
// empty; the launcher picks it).
template <WeightFormat WF, Epilogue EPI, bool HAS_BIAS, bool KTAIL, int BM>
__global__ __launch_bounds__(kThreads, 2) void w4a4_gemm_kernel(
    const uint8_t* __restrict__ qx, const float* __restrict__ sx, int M, int K,
    const uint8_t* __restrict__ qw, const float* __restrict__ sw, int N,
    const uint16_t* __restrict__ bias, void* __restrict__ out, int tiles_m, int tiles_n) {
  using WT = WTraits<WF>;
  static_assert(BM == 128 || BM == 112, "tile heights of 7 or 8 fragments");
  constexpr int kBM = BM, kWM = BM, kFM = BM / 16;
  constexpr int kXSlots = kBM * kXChunks;  // 16-byte slots of the int8 activation tile
  constexpr int kStageSlots = kXSlots + kBN * WT::kWChunks, kWDma = WT::kDma;
  // Two stage buffers, each the int8 activation tile followed by the packed
  // weight tile; the bf16 epilogue reuses them to stage the output tile.
  constexpr int kOutSlots = kThreads / 64 * kWM * kWN * 2 / 16;
  __shared__ uint4 lds[2 * kStageSlots > kOutSlots ? 2 * kStageSlots : kOutSlots];

  TileCoord tc;
  if (!tile_of_block(blockIdx.x, tiles_m, tiles_n, &tc)) return;
  const int m0 = tc.tm * kBM;
  const int n0 = tc.tn * kBN;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform, held in an SGPR
  const int wn = wave;  // waves split the weight rows; each covers every activation row
  const int li = lane & 15, lg = lane >> 4;

  const int64_t row_bytes = K / 2;                       // packed activation row
  const int64_t wrow_bytes = WT::kTern ? K / 4 : K / 2;  // packed weight row
  const int ksteps = static_cast<int>((row_bytes + kBKB - 1) / kBKB);

  // Buffer descriptors over the two packed operands (sizes < 2^31, checked by
  // the host), so every per-lane address is a 32-bit offset.
  const __amdgpu_buffer_rsrc_t rsx =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(qx), 0, static_cast<int>(M * row_bytes), kBufferFlags);
  const __amdgpu_buffer_rsrc_t rsw =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(qw), 0, static_cast<int>(N * wrow_bytes), kBufferFlags);

  // Weight DMA: one instruction fills kDmaRows tile rows R .. in lane order
  // (int4: 16 rows of 4 slots, lane l -> row R + (l >> 2), swizzled chunk
  // l & 3, so it fetches global chunk (l & 3) ^ ((l >> 3) & 3); ternary: 32
  // rows of 2 slots, lane l -> row R + (l >> 1), global chunk
  // (l & 1) ^ ((l >> 4) & 1)).
  const int dma_chunk = WT::kTern ? ((lane & 1) ^ ((lane >> 4) & 1)) : ((lane & 3) ^ ((lane >> 3) & 3));
  uint32_t ow[kWDma];
#pragma unroll
  for (int j = 0; j < kWDma; ++j) {
    const int r = WT::kDmaRows * (kWDma * wave + j) + (WT::kTern ? (lane >> 1) : (lane >> 2));
    ow[j] = static_cast<uint32_t>(min(n0 + r, N - 1)) * static_cast<uint32_t>(wrow_bytes) + 16 * dma_chunk;
  }
  // Activation loads: thread loads packed chunk (tid & 3) of tile rows
  // (tid >> 2) + 64 i; it widens chunk c into int8 chunks 2c and 2c + 1.
  // With 112-row tiles the last wave (rows 112..127) has no second load.
  const int xl_chunk = tid & 3;
  const int xl_row = tid >> 2;
  const bool x2 = xl_row + 64 < kBM;  // wave-uniform
  uint32_t ox[kXLoads];
#pragma unroll
  for (int i = 0; i < kXLoads; ++i)
    ox[i] = static_cast<uint32_t>(min(m0 + xl_row + 64 * i, M - 1)) * static_cast<uint32_t>(row_bytes) +
            16 * xl_chunk;

  uint4 gx[kXLoads];
  auto issue = [&](uint4* buf, int ks) {
    const int kb = ks * kBKB;
    const int kbw = ks * WT::kStageBytes;
    // K % 128 == 64: in the last stage the upper half of every row (codes
    // 64 .. 127) lies past the row end.  The weight DMA then fetches an
    // in-bounds chunk instead; the activation codes there are zeroed, so
    // those products vanish.
    const uint32_t back = (KTAIL && kbw + 16 * dma_chunk >= wrow_bytes) ? WT::kStageBytes / 2 : 0u;
#pragma unroll
    for (int j = 0; j < kWDma; ++j) dma16(rsw, buf + kXSlots + 64 * (kWDma * wave + j), ow[j] - back, kbw);
    // Same for the activation chunks past the row end: read an in-bounds
    // chunk (never past the end of the operand), then zero the codes.
    const uint32_t xback = (KTAIL && kb + 16 * xl_chunk >= row_bytes) ? 32u : 0u;
#pragma unroll
    for (int i = 0; i < kXLoads; ++i)
      if (i == 0 || x2)
        gx[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rsx, ox[i] - xback, kb, 0));
    if (KTAIL && kb + 16 * xl_chunk >= row_bytes) {
#pragma unroll
      for (int i = 0; i < kXLoads; ++i) gx[i] = make_uint4(0, 0, 0, 0);
    }
  };
  auto store_x = [&](uint4* buf) {
#pragma unroll
    for (int i = 0; i < kXLoads; ++i) {
      const int row = xl_row + 64 * i;
      if (i == 1 && !x2) break;
      if constexpr (WT::kTern) {
        buf[x_slot(row, 2 * xl_chunk)] = __builtin_bit_cast(uint4, unpack8_tern_order(gx[i].x, gx[i].y));
        buf[x_slot(row, 2 * xl_chunk + 1)] = __builtin_bit_cast(uint4, unpack8_tern_order(gx[i].z, gx[i].w));
      } else {
        buf[x_slot(row, 2 * xl_chunk)] = __builtin_bit_cast(uint4, unpack8(gx[i].x, gx[i].y));
        buf[x_slot(row, 2 * xl_chunk + 1)] = __builtin_bit_cast(uint4, unpack8(gx[i].z, gx[i].w));
      }
    }
  };

  v4i acc[kFN][kFM];
#pragma unroll
  for (int a = 0; a < kFN; ++a)
#pragma unroll
    for (int b = 0; b < kFM; ++b) acc[a][b] = v4i{0, 0, 0, 0};

  // One stage: read fragments from `cur`, start the loads of stage ks + 1
  // into `nxt`, run both MFMA half-stages, wait, write the widened activation
  // tile of stage ks + 1, barrier.
  auto stage = [&](const uint4* cur, uint4* nxt, int ks) {
    // Lane group lg covers codes 32 lg .. 32 lg + 31 of the stage: 16 packed
    // bytes of an int4 row, 8 of a ternary row.
    uint4 pw[kFN];
#pragma unroll
    for (int f = 0; f < kFN; ++f) {
      const int row = kWN * wn + 16 * f + li;
      if constexpr (WT::kTern) {
        const uint2 v = reinterpret_cast<const uint2*>(cur + kXSlots)[2 * wt_slot(row, lg >> 1) + (lg & 1)];
        pw[f] = make_uint4(v.x, v.y, 0, 0);
      } else {
        pw[f] = cur[kXSlots + w_slot(row, lg)];
      }
    }
    v4i bx0[kFM], bx1[kFM];
#pragma unroll
    for (int f = 0; f < kFM; ++f) bx0[f] = __builtin_bit_cast(v4i, cur[x_slot(16 * f + li, 2 * lg)]);
#pragma unroll
    for (int f = 0; f < kFM; ++f) bx1[f] = __builtin_bit_cast(v4i, cur[x_slot(16 * f + li, 2 * lg + 1)]);
    const bool more = ks + 1 < ksteps;
    if (more) issue(nxt, ks + 1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int fn = 0; fn < kFN; ++fn) {
      const v4i aw = WT::kTern ? unpack_tern(pw[fn].x) : unpack8(pw[fn].x, pw[fn].y);
#pragma unroll
      for (int fm = 0; fm < kFM; ++fm)
        acc[fn][fm] = __builtin_amdgcn_mfma_i32_16x16x64_i8(aw, bx0[fm], acc[fn][fm], 0, 0, 0);
    }
    // Widen each weight fragment just before its row of MFMAs.
#pragma unroll
    for (int fn = 0; fn < kFN; ++fn) {
      __builtin_amdgcn_sched_group_barrier(0x002, WT::kUnpackValu, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, kFM, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int fn = 0; fn < kFN; ++fn) {
      const v4i aw = WT::kTern ? unpack_tern(pw[fn].y) : unpack8(pw[fn].z, pw[fn].w);
#pragma unroll
      for (int fm = 0; fm < kFM; ++fm)
        acc[fn][fm] = __builtin_amdgcn_mfma_i32_16x16x64_i8(aw, bx1[fm], acc[fn][fm], 0, 0, 0);
    }
    // Widen each weight fragment just before its four MFMAs.
#pragma unroll
    for (int fn = 0; fn < kFN; ++fn) {
      __builtin_amdgcn_sched_group_barrier(0x002, WT::kUnpackValu, 1);
      __builtin_amdgcn_sched_group_barrier(0x008, 4, 1);
    }
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(kWaitVm0);
    if (more) store_x(nxt);
    __syncthreads();
  };

  issue(lds, 0);
  __builtin_amdgcn_s_waitcnt(kWaitVm0);
  store_x(lds);
  __syncthreads();
  for (int ks = 0; ks < ksteps; ++ks) {
    const int cur = (ks & 1) * kStageSlots;
    stage(lds + cur, lds + (kStageSlots - cur), ks);
  }

  // Epilogue.  Lane holds, for tile (fn, fm), rows n = nb + 4 lg + r (r = 0..3)
  // of column m = mb + li of y^T.
  const int mb = m0 + li;
  const int nb = n0 + kWN * wn + 4 * lg;
  const bool full = (m0 + kBM <= M) && (n0 + kBN <= N) && (N % 4 == 0);

  if constexpr (EPI == Epilogue::kInt32) {
    int32_t* o = static_cast<int32_t*>(out);
#pragma unroll
    for (int fn = 0; fn < kFN; ++fn) {
      const int n = nb + 16 * fn;
#pragma unroll
      for (int fm = 0; fm < kFM; ++fm) {
        const int m = mb + 16 * fm;
        const v4i a = acc[fn][fm];
        const int v0 = a[0] >> WT::kShift, v1 = a[1] >> WT::kShift, v2 = a[2] >> WT::kShift, v3 = a[3] >> WT::kShift;
        int32_t* p = o + static_cast<int64_t>(m) * N + n;
        if (full) {
          *reinterpret_cast<int4*>(p) = make_int4(v0, v1, v2, v3);
        } else if (m < M) {
          if (n + 0 < N) p[0] = v0;
          if (n + 1 < N) p[1] = v1;
          if (n + 2 < N) p[2] = v2;
          if (n + 3 < N) p[3] = v3;
        }
      }
    }
  } else {
    uint16_t* o = static_cast<uint16_t*>(out);
    // The stage buffers are free once every wave is done with the last
    // stage; each wave then stages its outputs in 16 KiB of them.
    __syncthreads();
    v4u32* stg = reinterpret_cast<v4u32*>(lds);
    v2u32* stg2 = reinterpret_cast<v2u32*>(lds);
    const int sbase = wave * (kWM * kWN * 2 / 16);  // in 16-byte units
    float sxv[kFM];
#pragma unroll
    for (int fm = 0; fm < kFM; ++fm) sxv[fm] = sx[min(mb + 16 * fm, M - 1)];
#pragma unroll
    for (int fn = 0; fn < kFN; ++fn) {
      const int n = nb + 16 * fn;
      float swv[4], bv[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int nn = min(n + r, N - 1);
        swv[r] = sw[nn];
        bv[r] = HAS_BIAS ? __uint_as_float(static_cast<uint32_t>(bias[nn]) << 16) : 0.0f;
      }
#pragma unroll
      for (int fm = 0; fm < kFM; ++fm) {
        const v4i a = acc[fn][fm];
        uint16_t h[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float f = static_cast<float>(a[r] >> WT::kShift);
          f = f * sxv[fm];
          f = f * swv[r];
          if (HAS_BIAS) f = f + bv[r];
          h[r] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
        }
        // staged in LDS: the wave's 128 rows x 64 columns, 128 bytes a row,
        // 16-byte chunk c of row rr at chunk c ^ (rr & 7)
        const int rr = 16 * fm + li, col = 16 * fn + 4 * lg;
        stg2[2 * (sbase + 8 * rr + ((col >> 3) ^ (rr & 7))) + ((col & 7) >> 2)] =
            v2u32{h[0] | (static_cast<uint32_t>(h[1]) << 16), h[2] | (static_cast<uint32_t>(h[3]) << 16)};
      }
    }
    __builtin_amdgcn_wave_barrier();
    // whole 128-byte rows to memory, eight rows per instruction (in a ragged
    // tile, element by element where a row runs past M or N)
    const bool vec = full && (N % 8 == 0);
#pragma unroll
    for (int it = 0; it < kWM / 8; ++it) {
      const int rr = 8 * it + (lane >> 3), c = lane & 7;
      const v4u32 v = stg[sbase + 8 * rr + (c ^ (rr & 7))];
      const int m = m0 + rr;
      const int n = n0 + kWN * wn + 8 * c;
      uint16_t* p = o + static_cast<int64_t>(m) * N + n;
      if (m >= M) {
      } else if (vec) {
        __builtin_nontemporal_store(v, reinterpret_cast<v4u32*>(p));
      } else {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (n + e < N) p[e] = static_cast<uint16_t>(w[e >> 1] >> (16 * (e & 1)));
      }
    }
  }
}

}  // namespace

// Tile height of the GEMM, 128 or 112 activation rows, for an M x N output
// with `slots` block slots (two per CU).  The blocks of an XCD take its share
// of the tiles in rounds of its slots.  A round costs one tile time when more
// than half of the XCD's slots hold a block, about 0.6 of one when at most
// half do (a lone block has its CU's matrix pipes to itself), nothing when
// empty; a 112-row tile takes about 0.93 of a 128-row one.  The cheaper
// estimate wins, 128 on ties.  (Measured: FLUX MLP-down 9216 x 12288 -> 3072
// and the DiT projections gain 5-8% from 112-row tiles; the 8B dLLM linears,
// whose 128-row tiles fill whole rounds, and FLUX MLP-up, whose last round
// is three-eighths full, lose.)
int gemm_tile_rows(int64_t M, int64_t N, int64_t slots) {
  const int64_t tiles_n = (N + kBN - 1) / kBN;
  const int64_t xcd_slots = std::max<int64_t>(1, slots / kNumXcd);
  int best = 128;
  int64_t best_cost = -1;
  for (const int bm : {128, 112}) {
    const int64_t per_xcd = ((M + bm - 1) / bm * tiles_n + kNumXcd - 1) / kNumXcd;
    const int64_t rest = per_xcd % xcd_slots;
    const int64_t tenths = 10 * (per_xcd / xcd_slots) + (rest == 0 ? 0 : 2 * rest <= xcd_slots ? 6 : 10);
    const int64_t cost = tenths * (bm == 128 ? 100 : 93);
    if (best_cost < 0 || cost < best_cost) best = bm, best_cost = cost;
  }
  return best;
}

hipError_t launch_w4a4_gemm(Epilogue epi, const uint8_t* qx, const float* sx, int64_t M, int64_t K,
                            const uint8_t* qw, const float* sw, int64_t N, const uint16_t* bias,
                            void* out, hipStream_t st, WeightFormat wf) {
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const int bm = gemm_tile_rows(M, N, 2 * std::max<int64_t>(kNumXcd, cus / kNumXcd * kNumXcd));
  const int tiles_m = static_cast<int>((M + bm - 1) / bm);
  const int tiles_n = static_cast<int>((N + kBN - 1) / kBN);
  const int64_t T = static_cast<int64_t>(tiles_m) * tiles_n;
  const int64_t per_xcd = (T + kNumXcd - 1) / kNumXcd;
  const dim3 grid(static_cast<unsigned>(per_xcd * kNumXcd));
  const dim3 block(kThreads);
  const int Mi = static_cast<int>(M), Ki = static_cast<int>(K), Ni = static_cast<int>(N);
  const bool tail = (K % 128) != 0;
#define JQ_LAUNCH(W, E, B, T)                                                                                \
  do {                                                                                                       \
    if (bm == 112)                                                                                           \
      hipLaunchKernelGGL((w4a4_gemm_kernel<W, E, B, T, 112>), grid, block, 0, st, qx, sx, Mi, Ki, qw, sw, Ni, \
                         bias, out, tiles_m, tiles_n);                                                       \
    else                                                                                                     \
      hipLaunchKernelGGL((w4a4_gemm_kernel<W, E, B, T, 128>), grid, block, 0, st, qx, sx, Mi, Ki, qw, sw, Ni, \
                         bias, out, tiles_m, tiles_n);                                                       \
  } while (0)
#define JQ_DISPATCH(W)                                                                    \
  if (epi == Epilogue::kInt32) {                                                          \
    if (tail) JQ_LAUNCH(W, Epilogue::kInt32, false, true);                                \
    else JQ_LAUNCH(W, Epilogue::kInt32, false, false);                                    \
  } else if (bias != nullptr) {                                                           \
    if (tail) JQ_LAUNCH(W, Epilogue::kBf16, true, true);                                  \
    else JQ_LAUNCH(W, Epilogue::kBf16, true, false);                                      \
  } else {                                                                                \
    if (tail) JQ_LAUNCH(W, Epilogue::kBf16, false, true);                                 \
    else JQ_LAUNCH(W, Epilogue::kBf16, false, false);                                     \
  }
  if (wf == WeightFormat::kTernary) {
    JQ_DISPATCH(WeightFormat::kTernary)
  } else {
    JQ_DISPATCH(WeightFormat::kInt4)
  }
#undef JQ_DISPATCH
#undef JQ_LAUNCH
  return hipGetLastError();
}

}  // namespace jq
