// LDS tile helpers shared by the attention kernels (internal to liblt).
#pragma once

#include "common.hpp"

namespace lt {

// Row-layout tile [rows][D] (features contiguous), 2D bytes per row; the
// 16-byte chunk c of row r sits at chunk c ^ gsw(r).  For 256-byte rows gsw
// spreads sixteen consecutive rows over sixteen chunk positions (row reads:
// 16 lanes x 16 B per LDS cycle) and four consecutive rows over four 64-byte
// windows (transpose reads).
template <int D, int NW>
struct RowTile {
  static constexpr int CPR = D / 8;       // 16-byte chunks per row
  static constexpr int ROWB = 2 * D;
  __device__ static __forceinline__ int gsw(int r) { return ((r & 15) ^ ((r & 3) << 2)) & (CPR - 1); }
  __device__ static __forceinline__ int addr(int r, int c) { return r * ROWB + ((c ^ gsw(r)) << 4); }

  // Direct loads of ROWS rows starting at global row pointer g (row stride
  // `stride` elements, `valid` rows readable, the rest read as zero), into
  // the tile at lds, by this wave's share of the 1 KiB blocks.
  template <int ROWS>
  __device__ static __forceinline__ void dma(char* lds, const lt_half* g, int64_t stride, int valid,
                                             int wave, int lane) {
    constexpr int RPI = 64 / CPR;                 // rows per 1 KiB load
    constexpr int NINST = ROWS / RPI;
    static_assert(NINST % NW == 0, "tile must split across waves");
    const int nv = valid < ROWS ? valid : ROWS;
    const uint32_t nrec = nv > 0 ? (uint32_t)((int64_t)nv * stride * 2) : 0u;
#pragma unroll
    for (int t = 0; t < NINST / NW; ++t) {
      const int n = wave * (NINST / NW) + t;
      const int r = n * RPI + lane / CPR;
      const int c = (lane % CPR) ^ gsw(r);
      lds_dma16_opaque(g, nrec, lds + n * 1024, (uint32_t)((r * stride + c * 8) * 2));
    }
  }

  // A/B operand with rows rb + lane%32 and features kk*16 + 8*(lane/32) + 0..7.
  __device__ static __forceinline__ half8 row_frag(const char* lds, int rb, int kk, int lane) {
    return as_half8(*reinterpret_cast<const u32x4*>(lds + addr(rb + (lane & 31), kk * 2 + (lane >> 5))));
  }

  // Transposed operand (rows of the tile are the reduction index): lane gets
  // features fb + lane%32 at tile rows
  //   canonical : kb + 8*(lane/32) + j                    (j = 0..7)
  //   acc order : kb + 8*(j/4) + 4*(lane/32) + (j%4)       (MFMA accumulator rows)
  template <bool ACC_ORDER>
  __device__ static __forceinline__ half8 tr_frag(const char* lds, int kb, int fb, int lane) {
    const int f = fb + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
    const int c = f >> 3;
    const int inoff = (f & 7) * 2;
    v4s part[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int k = ACC_ORDER ? kb + 8 * h + 4 * (lane >> 5) + ((lane & 15) >> 2)
                              : kb + 8 * (lane >> 5) + 4 * h + ((lane & 15) >> 2);
      part[h] = lds_read_tr16(lds + addr(k, c) + inoff);
    }
    return as_half8(pack_v4s_pair(part[0], part[1]));
  }
};

// (b, h) of a query-head workgroup from bh = blockIdx.x % (B * Hq).  The
// hardware deals consecutive workgroups to the 8 XCDs in turn, so bh's
// residue mod 8 picks the XCD (B * Hq is then a multiple of 8).  With
// grouped queries and B * Hkv a multiple of 8, the Hq / Hkv query heads of
// one kv head get bh values equal mod 8: they run on one XCD and read their
// shared K / V tiles through one L2.  Otherwise heads follow bh in order.
__device__ __forceinline__ void query_head(int bh, int B, int Hq, int Hkv, int& b, int& h) {
  if (Hq != Hkv && (B * Hkv) % 8 == 0) {
    const int bkv = bh % (B * Hkv);
    const int j = bh / (B * Hkv);
    b = bkv / Hkv;
    h = (bkv % Hkv) * (Hq / Hkv) + j;
  } else {
    b = bh / Hq;
    h = bh % Hq;
  }
}

}  // namespace lt
