// LDS tiles of the attention kernels (forward and backward) on gfx950: 64
// rows of HD bf16, row-major, each row's 16-byte chunks XOR-swizzled by the
// row index (chunk c of row r is stored at c ^ (r & kSwz)), so that the
// 16-byte fragment reads of 16 consecutive rows and the transpose loads both
// spread over the banks. The tiles are filled by buffer DMA (global -> LDS
// without registers) by the four waves of a workgroup.
#pragma once

#include <hip/hip_runtime.h>

#include "dsf_device.h"

namespace dsf {

constexpr int kAttnTileRows = 64;

template <int HD>
struct AttnTile {
  static constexpr int kRowBytes = HD * 2;
  static constexpr int kNch = HD / 8;                          // 16-byte chunks per row
  static constexpr int kSwz = kNch - 1;                        // chunk c of row r is stored at c ^ (r & kSwz)
  static constexpr int kTileBytes = kAttnTileRows * kRowBytes;  // one tile
  static constexpr int kDmaPerWave = kTileBytes / 1024 / 4;    // 1 KB per wave-wide DMA, 4 waves
  static_assert(kDmaPerWave >= 1 && (kNch & (kNch - 1)) == 0, "head dim");
};

// DMA of rows r0 .. r0 + 63 of a bf16 matrix (row stride `stride` elements,
// HD elements per row used) into the tile at `lds`. The buffer resource ends
// after row n - 1, so rows >= n land as zeros. Lane `lane` of this wave's
// e-th DMA fills 16 bytes at tile byte 1024 (wave kDmaPerWave + e) + 16 lane:
// row r, chunk position c, which holds the row's global chunk c ^ (r & kSwz).
template <int HD>
__device__ __forceinline__ void attn_tile_dma(const uint16_t* src, int64_t stride, int r0, int n, char* lds,
                                              int wave, int lane) {
  using A = AttnTile<HD>;
  const int rows = n - r0;
  int64_t bytes = rows > 0 ? (int64_t(rows - 1) * stride + HD) * 2 : 0;
  if (bytes > 0x7fffffff) bytes = 0x7fffffff;  // the tile's rows lie far below the clamp
  const auto rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(src + int64_t(r0) * stride), (short)0,
                                                      int(bytes), 0x00020000);
#pragma unroll
  for (int e = 0; e < A::kDmaPerWave; ++e) {
    const int byte = 1024 * (wave * A::kDmaPerWave + e) + 16 * lane;
    const int r = byte / A::kRowBytes, c = (byte % A::kRowBytes) / 16;
    const uint32_t voff = uint32_t(int64_t(r) * stride * 2 + ((c ^ (r & A::kSwz)) * 16));
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rsrc, (__attribute__((address_space(3))) void*)(lds + 1024 * (wave * A::kDmaPerWave + e)), 16, int(voff), 0,
        0, 0);
  }
}

// 8 bf16 of tile row `row`, logical chunk `ch` (elements 8 ch .. 8 ch + 7).
template <int HD>
__device__ __forceinline__ bf16x8 attn_row_frag(const char* tile, int row, int ch) {
  using A = AttnTile<HD>;
  return *reinterpret_cast<const bf16x8*>(tile + row * A::kRowBytes + ((ch ^ (row & A::kSwz)) * 16));
}

// The four LDS transpose loads of one 16-column block of a tile's transpose
// (rows 0-15, 16-31, 32-47, 48-63 at byte stride 16 rows) and the wait for
// them, as one inline-assembly statement: the compiler, which cannot see
// whether such a load overlaps an LDS DMA in flight, would otherwise wait for
// every DMA before it; the callers have made the tile's own DMA visible (the
// wave's wait and a barrier), and the DMA in flight writes another stage.
template <int HD>
__device__ __forceinline__ void lds_read_tr4(uint32_t addr, u32x2 (&v)[4]) {
  asm volatile(
      "ds_read_b64_tr_b16 %0, %4\n\t"
      "ds_read_b64_tr_b16 %1, %4 offset:%5\n\t"
      "ds_read_b64_tr_b16 %2, %4 offset:%6\n\t"
      "ds_read_b64_tr_b16 %3, %4 offset:%7\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3])
      : "v"(addr), "n"(16 * HD * 2), "n"(32 * HD * 2), "n"(48 * HD * 2)
      : "memory");
}

// Transposed fragments of a tile: with the transpose load, lane 16 G + 4 a + b
// receives element b of the 8-byte rows addressed by lanes 16 G + a + 4 j
// (j = 0..3). Addressing row 4 G + j at columns 16 blk + 4 a .. + 3, lane
// (r16, grp) of the MFMA A operand gets T[16 blk + r16][32 s + 4 grp + j]
// (j = 0..3) and T[16 blk + r16][32 s + 16 + 4 grp + j] for s = 0, 1, where
// T[c][r] = tile[r][c]: the k-slot order in which a lane holds the
// probabilities after the score MFMA.
template <int HD>
struct AttnTrans {
  using A = AttnTile<HD>;
  int base;  // lane-constant byte offset within the tile
  int u;     // lane-constant part of the swizzled chunk index
  __device__ __forceinline__ explicit AttnTrans(int lane) {
    const int tg = lane >> 4, ta = lane & 3, tj = (lane >> 2) & 3;
    const int vrow = 4 * tg + tj;
    base = vrow * A::kRowBytes + (ta & 1) * 8;
    u = (ta >> 1) ^ (vrow & A::kSwz);
  }
  // LDS byte address of the first of the four loads of column block blk
  __device__ __forceinline__ uint32_t addr(const char* tile, int blk) const {
    return uint32_t(size_t((__attribute__((address_space(3))) const char*)(tile))) + uint32_t(base) +
           uint32_t(((2 * blk) ^ u) * 16);
  }
  // the two MFMA A operands (s = 0, 1) of column block blk
  __device__ __forceinline__ void read(const char* tile, int blk, bf16x8 (&out)[2]) const {
    u32x2 v[4];
    lds_read_tr4<HD>(addr(tile, blk), v);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const u32x4 raw = {v[2 * s][0], v[2 * s][1], v[2 * s + 1][0], v[2 * s + 1][1]};
      out[s] = __builtin_bit_cast(bf16x8, raw);
    }
  }
};

}  // namespace dsf
