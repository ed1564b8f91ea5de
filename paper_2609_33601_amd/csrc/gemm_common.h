// Building blocks shared by the packed low-bit GEMM kernels for gfx950:
// stage geometry, LDS swizzles, int4 widening, buffer-to-LDS DMA and the
// XCD-aware tile order.  Device code only; included by the GEMM sources.
#ifndef JQ_GEMM_COMMON_H
#define JQ_GEMM_COMMON_H

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace jq {
namespace gemm_detail {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int kBKB = 64;                      // packed activation bytes of K per stage (128 codes)
constexpr int kChunks = kBKB / 16;            // 16-byte packed chunks per activation row per stage
constexpr int kXChunks = 2 * kChunks;         // 16-byte int8 chunks per widened activation row per stage
constexpr int kThreads = 256;                 // four waves per block
constexpr int kGroupM = 8;                    // m-tiles per n sweep in the tile order
constexpr int kNumXcd = 8;                    // MI355X accelerator complex dies
constexpr int kBufferFlags = 0x00020000;      // buffer descriptor word 3 for raw byte-addressed loads
constexpr int kWaitVm0 = (0x7 << 4) | (0xF << 8);  // s_waitcnt vmcnt(0), other counters untouched

static_assert(kChunks == 4 && kXChunks == 8, "swizzles below assume 4 packed / 8 int8 chunks per LDS row");

// LDS slots (16-byte units): chunk c of a packed int4 row r (64 bytes per
// stage), and int8 chunk c of a widened activation row r (128 bytes).  The
// XOR swizzles spread the 16 rows read by one ds_read_b128 over all banks.
__device__ __forceinline__ int w_slot(int row, int c) { return row * kChunks + (c ^ ((row >> 1) & 3)); }
__device__ __forceinline__ int x_slot(int row, int c) { return row * kXChunks + (c ^ (row & 7)); }

// Widen 16 int4 codes (p0: codes 0..7, p1: codes 8..15, even k in the low
// nibble) to int8 16 * code without sign extension: hi = p & 0xF0F0F0F0 and
// lo = (p << 4) & 0xF0F0F0F0.  Result dwords: codes 0 2 4 6 | 1 3 5 7 |
// 8 10 12 14 | 9 11 13 15.
__device__ __forceinline__ v4i unpack8(uint32_t p0, uint32_t p1) {
  v4i r;
  r[0] = static_cast<int>((p0 << 4) & 0xF0F0F0F0u);
  r[1] = static_cast<int>(p0 & 0xF0F0F0F0u);
  r[2] = static_cast<int>((p1 << 4) & 0xF0F0F0F0u);
  r[3] = static_cast<int>(p1 & 0xF0F0F0F0u);
  return r;
}

// 16 (or 4) bytes per lane from a buffer straight into LDS: lane i writes
// dst + 16 i (dst + 4 i), with no registers involved (buffer_load ... lds).
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rs, uint4* dst, uint32_t voffset, int soffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t*)dst, 16, voffset, soffset, 0, 0);
}
__device__ __forceinline__ void dma4(__amdgpu_buffer_rsrc_t rs, float* dst, uint32_t voffset, int soffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t*)dst, 4, voffset, soffset, 0, 0);
}

struct TileCoord {
  int tm, tn;
};

// Blocks are dealt round-robin to the XCDs; XCD x takes the contiguous tile
// range [x * per_xcd, (x + 1) * per_xcd) in a grouped order (kGroupM m-tiles
// per n sweep), so tiles that share operand rows run under the same L2.
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

}  // namespace gemm_detail
}  // namespace jq

#endif  // JQ_GEMM_COMMON_H
