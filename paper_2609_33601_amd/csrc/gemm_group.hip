// Group-wise W4A4 GEMM for gfx950: int4 x int4 codes with one scale per G
// consecutive k (G = 64 or 128) on both operands, accumulated exactly per
// group in int32 and summed over groups in fp32.
//
// Operation (the group64 / group128 INT4 rows of the appendix experimental-
// details tables; the operator stays plain, Sec. 3.1 and FAQ Q7):
//   acc_g[m,n] = sum_{k in group g} qx[m,k] * qw[n,k]                  (exact)
//   S[m,n]     = 0;  S = fl32(S + fl32(fl32(f32(acc_g) * sx[m,g]) * sw[n,g])) for g in k order
//   y[m,n]     = bf16_rne(fl32(S + bias[n]))         (or S itself, for checking)
// Scales are fp32 [rows, K/G] row-major; every fp32 operation is rounded on
// its own (built with -ffp-contract=off).
//
// Structure (shared pieces in gemm_common.h):
//  * Block tile 128 (m) x 128 (n), four waves of 128 x 32 outputs (an 8 x 2
//    grid of 16 x 16 MFMA tiles, 64 outputs per lane).  Each lane keeps an
//    int32 group accumulator and the running fp32 sum for its 64 outputs, so
//    a block needs ~240 registers and 52 KiB of LDS: two blocks per CU.
//  * Stages of 128 codes as in the per-token kernel: the packed weight tile
//    and the group scales of the stage arrive by buffer-to-LDS DMA (16-byte
//    and 4-byte lanes), the activation tile is widened once per block into
//    int8 LDS rows.  A stage is one group (G = 128) or two (G = 64, one per
//    MFMA half-stage).
//  * A group's first MFMA takes a zero accumulator input, so starting a group
//    costs nothing.  After its MFMAs each lane folds the group into its sums:
//    shift out the operand scaling (the MFMA accumulates 256 * acc), convert,
//    two multiplies and an add per output.  Those five VALU instructions per
//    output and group, not the matrix pipe, bound this kernel.
//  * For K % 128 == 64 (only possible with G = 64) the last stage has one
//    group: its second half-stage is skipped entirely.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gemm_common.h"
#include "jq_internal.h"

namespace jq {

namespace {

using namespace gemm_detail;

constexpr int kBM = 128;                         // activation rows per block
constexpr int kBN = 128;                         // weight rows per block
constexpr int kWN = kBN / 4;                     // weight rows per wave
constexpr int kFM = kBM / 16, kFN = kWN / 16;    // 8 x 2 MFMA tiles per wave
constexpr int kXSlots = kBM * kXChunks;          // int8 activation tile, 16-byte slots
constexpr int kWSlots = kBN * kChunks;           // packed weight tile, 16-byte slots
constexpr int kXLoads = kBM * kChunks / kThreads;
constexpr int kWDma = kWN / 16;                  // weight DMA instructions per wave per stage

static_assert(kXLoads == 2 && kWDma == 2, "staging below assumes two loads and two DMAs per wave");

template <int G>
struct GTraits {
  static constexpr int kGroups = 128 / G;                       // groups per stage
  static constexpr int kScaleFloats = 2 * kGroups * 128;        // sx[kGroups][128] then sw[kGroups][128]
  static constexpr int kStageSlots = kXSlots + kWSlots + kScaleFloats / 4;
  static constexpr int kScaleDma = kGroups;                     // 4-byte-lane DMA instructions per wave
};

template <int G, Epilogue EPI, bool HAS_BIAS, bool KTAIL>
__global__ __launch_bounds__(kThreads, 2) void w4a4g_gemm_kernel(
    const uint8_t* __restrict__ qx, const float* __restrict__ sx, int M, int K,
    const uint8_t* __restrict__ qw, const float* __restrict__ sw, int N,
    const uint16_t* __restrict__ bias, void* __restrict__ out, int tiles_m, int tiles_n) {
  using GT = GTraits<G>;
  constexpr int kStageSlots = GT::kStageSlots;
  __shared__ uint4 lds[2 * kStageSlots];

  TileCoord tc;
  if (!tile_of_block(blockIdx.x, tiles_m, tiles_n, &tc)) return;
  const int m0 = tc.tm * kBM;
  const int n0 = tc.tn * kBN;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave;
  const int li = lane & 15, lg = lane >> 4;

  const int64_t row_bytes = K / 2;
  const int ksteps = static_cast<int>((row_bytes + kBKB - 1) / kBKB);
  const int groups_row = K / G;

  const __amdgpu_buffer_rsrc_t rsx =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(qx), 0, static_cast<int>(M * row_bytes), kBufferFlags);
  const __amdgpu_buffer_rsrc_t rsw =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(qw), 0, static_cast<int>(N * row_bytes), kBufferFlags);
  const __amdgpu_buffer_rsrc_t rssx = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(sx), 0, static_cast<int>(static_cast<int64_t>(M) * groups_row * 4), kBufferFlags);
  const __amdgpu_buffer_rsrc_t rssw = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(sw), 0, static_cast<int>(static_cast<int64_t>(N) * groups_row * 4), kBufferFlags);

  // Weight DMA: wave w fills its own 32 rows, 16 per instruction, lane l ->
  // row R + (l >> 2), swizzled chunk l & 3 (global chunk (l & 3) ^ ((l >> 3) & 3)).
  const int dma_chunk = (lane & 3) ^ ((lane >> 3) & 3);
  uint32_t ow[kWDma];
#pragma unroll
  for (int j = 0; j < kWDma; ++j) {
    const int r = 16 * (kWDma * wave + j) + (lane >> 2);
    ow[j] = static_cast<uint32_t>(min(n0 + r, N - 1)) * static_cast<uint32_t>(row_bytes) + 16 * dma_chunk;
  }
  // Scale DMA: 4 * kGroups instructions of 64 rows per stage (activation
  // scales rows 0..63 and 64..127, then weight scales, per group), dealt to
  // the waves: wave w issues instructions w, w + 4, ...  Lane l loads the
  // scale of row 64 * half + l.
  uint32_t os[GT::kScaleDma];
  int sdst[GT::kScaleDma];
  bool s_is_w[GT::kScaleDma];
#pragma unroll
  for (int j = 0; j < GT::kScaleDma; ++j) {
    const int u = wave + 4 * j;
    const int mat = u / (2 * GT::kGroups);      // 0: activation scales, 1: weight scales
    const int jg = (u >> 1) % GT::kGroups;      // group within the stage
    const int half = u & 1;
    const int r = 64 * half + lane;
    const int row = mat ? min(n0 + r, N - 1) : min(m0 + r, M - 1);
    os[j] = static_cast<uint32_t>(row) * static_cast<uint32_t>(groups_row) * 4u + 4u * jg;
    sdst[j] = (mat * GT::kGroups + jg) * 128 + 64 * half;
    s_is_w[j] = mat != 0;
  }
  // Activation loads as in the per-token kernel.
  const int xl_chunk = tid & 3;
  const int xl_row = tid >> 2;
  uint32_t ox[kXLoads];
#pragma unroll
  for (int i = 0; i < kXLoads; ++i)
    ox[i] = static_cast<uint32_t>(min(m0 + xl_row + 64 * i, M - 1)) * static_cast<uint32_t>(row_bytes) +
            16 * xl_chunk;

  uint4 gx[kXLoads];
  auto issue = [&](uint4* buf, int ks) {
    const int kb = ks * kBKB;
    const uint32_t back = (KTAIL && kb + 16 * dma_chunk >= row_bytes) ? 32u : 0u;
#pragma unroll
    for (int j = 0; j < kWDma; ++j) dma16(rsw, buf + kXSlots + 64 * (kWDma * wave + j), ow[j] - back, kb);
    float* sbuf = reinterpret_cast<float*>(buf + kXSlots + kWSlots);
    const int sk = ks * GT::kGroups * 4;
#pragma unroll
    for (int j = 0; j < GT::kScaleDma; ++j) dma4(s_is_w[j] ? rssw : rssx, sbuf + sdst[j], os[j], sk);
    const uint32_t xback = (KTAIL && kb + 16 * xl_chunk >= row_bytes) ? 32u : 0u;
#pragma unroll
    for (int i = 0; i < kXLoads; ++i)
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
      buf[x_slot(row, 2 * xl_chunk)] = __builtin_bit_cast(uint4, unpack8(gx[i].x, gx[i].y));
      buf[x_slot(row, 2 * xl_chunk + 1)] = __builtin_bit_cast(uint4, unpack8(gx[i].z, gx[i].w));
    }
  };

  v4i acc[kFN][kFM];
  float sum[kFN][kFM][4];
#pragma unroll
  for (int a = 0; a < kFN; ++a)
#pragma unroll
    for (int b = 0; b < kFM; ++b) {
      acc[a][b] = v4i{0, 0, 0, 0};
#pragma unroll
      for (int r = 0; r < 4; ++r) sum[a][b][r] = 0.0f;
    }

  // Fold the finished group jg of the stage in `buf` into the fp32 sums.
  auto fold = [&](const uint4* buf, int jg) {
    const float* sxl = reinterpret_cast<const float*>(buf + kXSlots + kWSlots) + jg * 128;
    const float* swl = reinterpret_cast<const float*>(buf + kXSlots + kWSlots) + (GT::kGroups + jg) * 128;
    float sxv[kFM];
#pragma unroll
    for (int fm = 0; fm < kFM; ++fm) sxv[fm] = sxl[16 * fm + li];
    float4 swv[kFN];
#pragma unroll
    for (int fn = 0; fn < kFN; ++fn) swv[fn] = *reinterpret_cast<const float4*>(swl + kWN * wn + 16 * fn + 4 * lg);
#pragma unroll
    for (int fn = 0; fn < kFN; ++fn) {
      const float w4[4] = {swv[fn].x, swv[fn].y, swv[fn].z, swv[fn].w};
#pragma unroll
      for (int fm = 0; fm < kFM; ++fm)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float t = static_cast<float>(acc[fn][fm][r] >> 8);
          t = t * sxv[fm];
          t = t * w4[r];
          sum[fn][fm][r] = sum[fn][fm][r] + t;
        }
    }
  };

  // One half-stage of MFMAs on 8 packed weight bytes per lane and fragment;
  // `fresh` starts a new group (zero accumulator input).
  auto half_mfma = [&](const uint2* pw, const v4i* bx, bool fresh) {
#pragma unroll
    for (int fn = 0; fn < kFN; ++fn) {
      const v4i aw = unpack8(pw[fn].x, pw[fn].y);
#pragma unroll
      for (int fm = 0; fm < kFM; ++fm)
        acc[fn][fm] = __builtin_amdgcn_mfma_i32_16x16x64_i8(aw, bx[fm], fresh ? v4i{0, 0, 0, 0} : acc[fn][fm], 0, 0, 0);
    }
  };

  // Which codes a lane feeds to the MFMAs.  G = 128: in half-stage h lane
  // group lg takes codes 32 lg + 16 h .. + 15 (one 16-byte weight read
  // serves both halves), and the whole stage is one group.  G = 64: each
  // half-stage must be one group, so half h takes codes 64 h + 16 lg .. + 15,
  // i.e. packed weight bytes 32 h + 8 lg .. + 7 and int8 activation chunk
  // 4 h + lg.
  auto stage = [&](const uint4* cur, uint4* nxt, int ks) {
    uint2 pw0[kFN], pw1[kFN];
    v4i bx0[kFM], bx1[kFM];
    const uint2* w2 = reinterpret_cast<const uint2*>(cur + kXSlots);
#pragma unroll
    for (int f = 0; f < kFN; ++f) {
      const int row = kWN * wn + 16 * f + li;
      if constexpr (G == 64) {
        pw0[f] = w2[2 * w_slot(row, lg >> 1) + (lg & 1)];
        pw1[f] = w2[2 * w_slot(row, 2 + (lg >> 1)) + (lg & 1)];
      } else {
        const uint4 v = cur[kXSlots + w_slot(row, lg)];
        pw0[f] = make_uint2(v.x, v.y);
        pw1[f] = make_uint2(v.z, v.w);
      }
    }
    const int c0 = G == 64 ? lg : 2 * lg;
    const int c1 = G == 64 ? 4 + lg : 2 * lg + 1;
#pragma unroll
    for (int f = 0; f < kFM; ++f) bx0[f] = __builtin_bit_cast(v4i, cur[x_slot(16 * f + li, c0)]);
#pragma unroll
    for (int f = 0; f < kFM; ++f) bx1[f] = __builtin_bit_cast(v4i, cur[x_slot(16 * f + li, c1)]);
    const bool more = ks + 1 < ksteps;
    if (more) issue(nxt, ks + 1);
    half_mfma(pw0, bx0, true);
    const bool second = !(KTAIL && ks + 1 == ksteps);  // K % 128 == 64: the last stage has one group
    if constexpr (G == 64) {
      fold(cur, 0);
      if (second) {
        half_mfma(pw1, bx1, true);
        fold(cur, 1);
      }
    } else {
      half_mfma(pw1, bx1, false);
      fold(cur, 0);
    }
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

  // Epilogue.  Lane holds, for tile (fn, fm), outputs n = nb + 16 fn + r
  // (r = 0..3) of row m = mb + 16 fm.
  const int mb = m0 + li;
  const int nb = n0 + kWN * wn + 4 * lg;
  const bool full = (m0 + kBM <= M) && (n0 + kBN <= N) && (N % 4 == 0);
#pragma unroll
  for (int fn = 0; fn < kFN; ++fn) {
    const int n = nb + 16 * fn;
    float bv[4];
#pragma unroll
    for (int r = 0; r < 4; ++r)
      bv[r] = HAS_BIAS ? __uint_as_float(static_cast<uint32_t>(bias[min(n + r, N - 1)]) << 16) : 0.0f;
#pragma unroll
    for (int fm = 0; fm < kFM; ++fm) {
      const int m = mb + 16 * fm;
      if constexpr (EPI == Epilogue::kF32) {
        float* p = static_cast<float*>(out) + static_cast<int64_t>(m) * N + n;
        if (full) {
          *reinterpret_cast<float4*>(p) = make_float4(sum[fn][fm][0], sum[fn][fm][1], sum[fn][fm][2], sum[fn][fm][3]);
        } else if (m < M) {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (n + r < N) p[r] = sum[fn][fm][r];
        }
      } else {
        uint16_t h[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float f = sum[fn][fm][r];
          if (HAS_BIAS) f = f + bv[r];
          h[r] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
        }
        uint16_t* p = static_cast<uint16_t*>(out) + static_cast<int64_t>(m) * N + n;
        if (full) {
          *reinterpret_cast<uint2*>(p) = make_uint2(h[0] | (static_cast<uint32_t>(h[1]) << 16),
                                                    h[2] | (static_cast<uint32_t>(h[3]) << 16));
        } else if (m < M) {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (n + r < N) p[r] = h[r];
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_w4a4g_gemm(Epilogue epi, const uint8_t* qx, const float* sx, int64_t M, int64_t K, int G,
                             const uint8_t* qw, const float* sw, int64_t N, const uint16_t* bias, void* out,
                             hipStream_t st) {
  const int tiles_m = static_cast<int>((M + kBM - 1) / kBM);
  const int tiles_n = static_cast<int>((N + kBN - 1) / kBN);
  const int64_t T = static_cast<int64_t>(tiles_m) * tiles_n;
  const int64_t per_xcd = (T + kNumXcd - 1) / kNumXcd;
  const dim3 grid(static_cast<unsigned>(per_xcd * kNumXcd));
  const dim3 block(kThreads);
  const int Mi = static_cast<int>(M), Ki = static_cast<int>(K), Ni = static_cast<int>(N);
  const bool tail = (K % 128) != 0;
#define JQ_LAUNCH(GS, E, B, T)                                                                         \
  hipLaunchKernelGGL((w4a4g_gemm_kernel<GS, E, B, T>), grid, block, 0, st, qx, sx, Mi, Ki, qw, sw, Ni, \
                     bias, out, tiles_m, tiles_n)
  if (G == 128) {
    // K % 128 == 0 whenever G == 128.
    if (epi == Epilogue::kF32) JQ_LAUNCH(128, Epilogue::kF32, false, false);
    else if (bias != nullptr) JQ_LAUNCH(128, Epilogue::kBf16, true, false);
    else JQ_LAUNCH(128, Epilogue::kBf16, false, false);
  } else if (tail) {
    if (epi == Epilogue::kF32) JQ_LAUNCH(64, Epilogue::kF32, false, true);
    else if (bias != nullptr) JQ_LAUNCH(64, Epilogue::kBf16, true, true);
    else JQ_LAUNCH(64, Epilogue::kBf16, false, true);
  } else {
    if (epi == Epilogue::kF32) JQ_LAUNCH(64, Epilogue::kF32, false, false);
    else if (bias != nullptr) JQ_LAUNCH(64, Epilogue::kBf16, true, false);
    else JQ_LAUNCH(64, Epilogue::kBf16, false, false);
  }
#undef JQ_LAUNCH
  return hipGetLastError();
}

}  // namespace jq
