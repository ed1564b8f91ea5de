// Packed-int4 x packed-int4 GEMM with int32 accumulation and a fused
// dequantising epilogue, hand-written for gfx950 (CDNA4) int8 MFMA.
//
// Operation (Sec. 3.1 low-bit operator; appendix FAQ Q7 low-bit matrix
// multiplication):  acc[m,n] = sum_k qx[m,k] * qw[n,k]  on int4 codes, then
//   y[m,n] = bf16_rne(((fp32(acc) * sx[m]) * sw[n]) + bias[n])
// with every fp32 operation rounded on its own (built with -ffp-contract=off).
//
// Structure.
//  * Block tile 256 (m) x 256 (n); four waves, each owning 128 x 128 outputs
//    as an 8 x 8 grid of 16 x 16 MFMA tiles (256 int32 accumulators per lane).
//  * K is consumed 128 codes (64 packed bytes per row) per stage.  Packed
//    tiles are loaded from global memory with 16-byte loads into registers one
//    stage ahead, then written to a double-buffered LDS tile (2 x 32 KiB).
//    LDS rows are 64 bytes; the 16-byte chunk c of row r is stored at
//    c ^ ((r >> 1) & 3) so that the 16 rows a lane group reads land on
//    different banks.
//  * Each MFMA v_mfma_i32_16x16x64_i8 consumes, per lane, 8 packed bytes of
//    one row of each operand.  They are unpacked in registers without any
//    sign extension: hi = p & 0xF0F0F0F0 and lo = (p << 4) & 0xF0F0F0F0 hold
//    16 * code as int8.  Both operands are unpacked the same way, so the k
//    order inside an MFMA is the same permutation for both and the sum is
//    unchanged; the accumulator holds 256 * acc exactly (|256 * acc| <= 2^30
//    for K <= 65536) and the epilogue shifts it back with >> 8.
//  * The weight tile is the MFMA A operand and the activation tile the B
//    operand, so the result is y^T: each lane ends up with 4 consecutive
//    output columns n of one row m, stored as one 8-byte bf16 write.
//  * Blocks are dispatched round-robin over the 8 XCDs; each XCD is given a
//    contiguous range of tiles in a grouped (GROUP_M m-tiles per n sweep)
//    order, so tiles that share operand rows run under the same L2.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "jq_internal.h"

namespace jq {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int kBM = 256;       // activation rows per block
constexpr int kBN = 256;       // weight rows per block
constexpr int kBKB = 64;       // packed bytes of K per stage (128 codes)
constexpr int kChunks = kBKB / 16;  // 16-byte chunks per row per stage
constexpr int kThreads = 256;
constexpr int kWM = 128, kWN = 128;  // per-wave tile
constexpr int kFM = kWM / 16, kFN = kWN / 16;
constexpr int kGroupM = 4;
constexpr int kNumXcd = 8;

static_assert(kChunks == 4, "swizzle below assumes 4 chunks per LDS row");

__device__ __forceinline__ int swz(int row, int chunk) { return row * kChunks + (chunk ^ ((row >> 1) & 3)); }

__device__ __forceinline__ v4i unpack8(uint32_t p0, uint32_t p1) {
  v4i r;
  r[0] = static_cast<int>((p0 << 4) & 0xF0F0F0F0u);
  r[1] = static_cast<int>(p0 & 0xF0F0F0F0u);
  r[2] = static_cast<int>((p1 << 4) & 0xF0F0F0F0u);
  r[3] = static_cast<int>(p1 & 0xF0F0F0F0u);
  return r;
}

struct TileCoord {
  int tm, tn;
};

__device__ __forceinline__ bool tile_of_block(int bid, int tiles_m, int tiles_n, TileCoord* tc) {
  const int T = tiles_m * tiles_n;
  const int per_xcd = (T + kNumXcd - 1) / kNumXcd;
  const int t = (bid % kNumXcd) * per_xcd + bid / kNumXcd;
  if (t >= T) return false;
  const int band = kGroupM * tiles_n;
  const int group = t / band;
  const int first_m = group * kGroupM;
  const int gm = min(tiles_m - first_m, kGroupM);
  const int r = t - group * band;
  tc->tm = first_m + r % gm;
  tc->tn = r / gm;
  return true;
}

template <Epilogue EPI, bool HAS_BIAS>
__global__ __launch_bounds__(kThreads, 1) void w4a4_gemm_kernel(
    const uint8_t* __restrict__ qx, const float* __restrict__ sx, int M, int K,
    const uint8_t* __restrict__ qw, const float* __restrict__ sw, int N,
    const uint16_t* __restrict__ bias, void* __restrict__ out, int tiles_m, int tiles_n) {
  __shared__ uint4 lds_x[2][kBM * kChunks];
  __shared__ uint4 lds_w[2][kBN * kChunks];

  TileCoord tc;
  if (!tile_of_block(blockIdx.x, tiles_m, tiles_n, &tc)) return;
  const int m0 = tc.tm * kBM;
  const int n0 = tc.tn * kBN;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int li = lane & 15, lg = lane >> 4;

  const int64_t row_bytes = K / 2;
  const int ksteps = static_cast<int>((row_bytes + kBKB - 1) / kBKB);

  // Global -> register staging: thread loads chunk (tid & 3) of rows (tid >> 2) + 64 i.
  const int ld_chunk = tid & 3;
  const int ld_row = tid >> 2;
  const uint8_t* gx[4];
  const uint8_t* gw[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int rx = min(m0 + ld_row + 64 * i, M - 1);
    const int rw = min(n0 + ld_row + 64 * i, N - 1);
    gx[i] = qx + static_cast<int64_t>(rx) * row_bytes + ld_chunk * 16;
    gw[i] = qw + static_cast<int64_t>(rw) * row_bytes + ld_chunk * 16;
  }
  uint4 stx[4], stw[4];

  auto load_stage = [&](int ks) {
    const int64_t kb = static_cast<int64_t>(ks) * kBKB;
    const bool ok = kb + ld_chunk * 16 < row_bytes;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      stx[i] = ok ? *reinterpret_cast<const uint4*>(gx[i] + kb) : make_uint4(0, 0, 0, 0);
      stw[i] = ok ? *reinterpret_cast<const uint4*>(gw[i] + kb) : make_uint4(0, 0, 0, 0);
    }
  };
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      lds_x[buf][swz(ld_row + 64 * i, ld_chunk)] = stx[i];
      lds_w[buf][swz(ld_row + 64 * i, ld_chunk)] = stw[i];
    }
  };

  v4i acc[kFN][kFM];
#pragma unroll
  for (int a = 0; a < kFN; ++a)
#pragma unroll
    for (int b = 0; b < kFM; ++b) acc[a][b] = v4i{0, 0, 0, 0};

  load_stage(0);
  store_stage(0);
  __syncthreads();

  for (int ks = 0; ks < ksteps; ++ks) {
    const int buf = ks & 1;
    if (ks + 1 < ksteps) load_stage(ks + 1);

    // This lane's 16 packed bytes (chunk lg) of each fragment row; the first 8
    // bytes feed the first MFMA k-step of the stage, the last 8 the second.
    uint4 pw[kFN], px[kFM];
#pragma unroll
    for (int f = 0; f < kFN; ++f) pw[f] = lds_w[buf][swz(kWN * wn + 16 * f + li, lg)];
#pragma unroll
    for (int f = 0; f < kFM; ++f) px[f] = lds_x[buf][swz(kWM * wm + 16 * f + li, lg)];

#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      v4i bx[kFM];
#pragma unroll
      for (int f = 0; f < kFM; ++f) bx[f] = kk == 0 ? unpack8(px[f].x, px[f].y) : unpack8(px[f].z, px[f].w);
#pragma unroll
      for (int fn = 0; fn < kFN; ++fn) {
        const v4i aw = kk == 0 ? unpack8(pw[fn].x, pw[fn].y) : unpack8(pw[fn].z, pw[fn].w);
#pragma unroll
        for (int fm = 0; fm < kFM; ++fm)
          acc[fn][fm] = __builtin_amdgcn_mfma_i32_16x16x64_i8(aw, bx[fm], acc[fn][fm], 0, 0, 0);
      }
    }

    if (ks + 1 < ksteps) store_stage(buf ^ 1);
    __syncthreads();
  }

  // Epilogue.  Lane holds, for tile (fn, fm), rows n = nb + 4 lg + r (r = 0..3)
  // of column m = mb + li of y^T.
  const int mb = m0 + kWM * wm + li;
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
        const int v0 = a[0] >> 8, v1 = a[1] >> 8, v2 = a[2] >> 8, v3 = a[3] >> 8;
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
        const int m = mb + 16 * fm;
        const v4i a = acc[fn][fm];
        uint16_t h[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float f = static_cast<float>(a[r] >> 8);
          f = f * sxv[fm];
          f = f * swv[r];
          if (HAS_BIAS) f = f + bv[r];
          h[r] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
        }
        uint16_t* p = o + static_cast<int64_t>(m) * N + n;
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

hipError_t launch_w4a4_gemm(Epilogue epi, const uint8_t* qx, const float* sx, int64_t M, int64_t K,
                            const uint8_t* qw, const float* sw, int64_t N, const uint16_t* bias,
                            void* out, hipStream_t st) {
  const int tiles_m = static_cast<int>((M + kBM - 1) / kBM);
  const int tiles_n = static_cast<int>((N + kBN - 1) / kBN);
  const int64_t T = static_cast<int64_t>(tiles_m) * tiles_n;
  const int64_t per_xcd = (T + kNumXcd - 1) / kNumXcd;
  const dim3 grid(static_cast<unsigned>(per_xcd * kNumXcd));
  const dim3 block(kThreads);
  const int Mi = static_cast<int>(M), Ki = static_cast<int>(K), Ni = static_cast<int>(N);
  if (epi == Epilogue::kInt32) {
    hipLaunchKernelGGL((w4a4_gemm_kernel<Epilogue::kInt32, false>), grid, block, 0, st, qx, sx, Mi,
                       Ki, qw, sw, Ni, bias, out, tiles_m, tiles_n);
  } else if (bias != nullptr) {
    hipLaunchKernelGGL((w4a4_gemm_kernel<Epilogue::kBf16, true>), grid, block, 0, st, qx, sx, Mi,
                       Ki, qw, sw, Ni, bias, out, tiles_m, tiles_n);
  } else {
    hipLaunchKernelGGL((w4a4_gemm_kernel<Epilogue::kBf16, false>), grid, block, 0, st, qx, sx, Mi,
                       Ki, qw, sw, Ni, bias, out, tiles_m, tiles_n);
  }
  return hipGetLastError();
}

}  // namespace jq
