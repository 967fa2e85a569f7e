// FP16 GEMM update C = alpha * op(A) op(B) + beta * C for gfx950.
//
// Sec. 4.1 of the paper describes the GEMM primitive (C tile loaded as the
// accumulation buffer) that serves the QKV / output / FFN projections in
// forward, data-gradient and weight-gradient form.  The MT-3000 dataflow
// (DDR -> GSM -> SM / AM staging, VLIW micro-kernel) is replaced here by the
// CDNA4 form of the same idea:
//   * a workgroup owns a BM x BN output tile held in MFMA accumulators;
//   * K is walked in BK = 64 slices, double-buffered in LDS, with the next
//     slice's global loads in flight while the current one feeds MFMA
//     (the overlap of operand preparation with MACs that the paper's
//     micro-kernel pipeline achieves);
//   * both operands are kept K-contiguous in LDS whatever their layout in
//     HBM: an operand whose HBM layout is M- or N-contiguous (dgrad B,
//     wgrad A and B) is transposed in registers (8x8 half blocks) between
//     the coalesced 16-byte global load and the LDS store, so one MFMA inner
//     loop serves every (transA, transB);
//   * LDS rows are 128 bytes with the 16-byte chunk index XOR-swizzled by the
//     row, which keeps the 16-byte MFMA operand reads conflict-free;
//   * output tiles are ordered so that consecutive tiles of one XCD share A
//     rows (grouped ordering) and each XCD gets a contiguous range of tiles.
#include "common.hpp"
#include "kernels.hpp"

namespace lt {
namespace {

constexpr int BK = 64;            // K slice per LDS stage (halves)
constexpr int ROWB = BK * 2;      // bytes per LDS row
constexpr int CHUNKS = BK / 8;    // 16-byte chunks per LDS row

__device__ __forceinline__ int swz(int row, int chunk) {   // chunk position in LDS row
  return chunk ^ (row & 7);
}

// Global -> register staging of one operand tile (R rows x BK), "rows" being
// M for A and N for B.  KCONTIG: the operand is stored with K contiguous
// (row r of the tile is a K-run at base + r*ld); otherwise it is stored with
// the row index contiguous (K-run r at base + k*ld + r).
template <int R, int NT, bool KCONTIG>
struct TileLoader {
  // K-contiguous: 16-byte chunks, R*BK/8 per tile.  Row-contiguous: 8x8
  // blocks (8 k-runs of 8 rows), (R/8)*(BK/8) per tile; threads beyond the
  // block count idle during staging.
  static constexpr int TOTAL = KCONTIG ? R * CHUNKS : (R / 8) * (BK / 8);
  static constexpr int PER = (TOTAL + NT - 1) / NT;
  static constexpr int NREG = KCONTIG ? PER : PER * 8;
  static_assert(!KCONTIG || TOTAL % NT == 0, "chunk count must divide evenly");
  u32x4 reg[NREG];

  __device__ __forceinline__ void load(const lt_half* __restrict__ base, int64_t ld,
                                       int64_t row0, int64_t rows, int64_t k0, int64_t K,
                                       int tid) {
    if constexpr (KCONTIG) {
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int id = tid + i * NT;
        const int r = id / CHUNKS;
        const int c = id % CHUNKS;
        const int64_t gr = row0 + r;
        const int64_t gk = k0 + c * 8;
        if (gr < rows && gk < K)
          reg[i] = ld16(base + gr * ld + gk);
        else
          reg[i] = u32x4{0, 0, 0, 0};
      }
    } else {
#pragma unroll
      for (int bi = 0; bi < PER; ++bi) {
        const int blk = tid + bi * NT;
        const int rb = blk % (R / 8);
        const int kb = blk / (R / 8);
        const int64_t gr = row0 + rb * 8;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int64_t gk = k0 + kb * 8 + j;
          if (blk < TOTAL && gr < rows && gk < K)
            reg[bi * 8 + j] = ld16(base + gk * ld + gr);
          else
            reg[bi * 8 + j] = u32x4{0, 0, 0, 0};
        }
      }
    }
  }

  __device__ __forceinline__ void store(char* lds, int tid) {
    if constexpr (KCONTIG) {
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int id = tid + i * NT;
        const int r = id / CHUNKS;
        const int c = id % CHUNKS;
        *reinterpret_cast<u32x4*>(lds + r * ROWB + swz(r, c) * 16) = reg[i];
      }
    } else {
#pragma unroll
      for (int bi = 0; bi < PER; ++bi) {
        const int blk = tid + bi * NT;
        if (blk >= TOTAL) break;
        const int rb = blk % (R / 8);
        const int kb = blk / (R / 8);
        u32x4 t[8];
        transpose8x8(&reg[bi * 8], t);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int r = rb * 8 + j;
          *reinterpret_cast<u32x4*>(lds + r * ROWB + swz(r, kb) * 16) = t[j];
        }
      }
    }
  }
};

// BM x BN tile, WGM x WGN waves, each wave (BM/WGM) x (BN/WGN).
template <int BM, int BN, int WGM, int WGN, bool TA, bool TB>
__global__ void __launch_bounds__(WGM * WGN * kWave)
gemm_f16_kernel(int64_t M, int64_t N, int64_t K, float alpha,
                const lt_half* __restrict__ A, int64_t lda,
                const lt_half* __restrict__ B, int64_t ldb, float beta,
                const lt_half* R, int64_t ldr, lt_half* C, int64_t ldc, int tiles_m,
                int tiles_n) {
  constexpr int NT = WGM * WGN * kWave;
  constexpr int WTM = BM / WGM;      // wave tile rows (M)
  constexpr int WTN = BN / WGN;      // wave tile cols (N)
  constexpr int TM = WTM / 32;       // 32x32 MFMA blocks per wave along M
  constexpr int TN = WTN / 32;
  constexpr int A_BYTES = BM * ROWB;
  constexpr int B_BYTES = BN * ROWB;
  __shared__ __attribute__((aligned(16))) char smem[2 * (A_BYTES + B_BYTES)];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WGN;
  const int wn = wave % WGN;

  // ---- tile ordering: contiguous range per XCD, then grouped along M ----
  int pid = blockIdx.x;
  const int nwg = gridDim.x;
  if ((nwg & 7) == 0) {
    const int per = nwg >> 3;
    pid = (pid & 7) * per + (pid >> 3);
  }
  constexpr int GROUP_M = 8;
  const int group_size = GROUP_M * tiles_n;
  const int group = pid / group_size;
  const int first_m = group * GROUP_M;
  const int gm = min(tiles_m - first_m, GROUP_M);
  const int in_group = pid % group_size;
  const int tile_m = first_m + in_group % gm;
  const int tile_n = in_group / gm;
  const int64_t m0 = (int64_t)tile_m * BM;
  const int64_t n0 = (int64_t)tile_n * BN;

  TileLoader<BM, NT, !TA> la;
  TileLoader<BN, NT, TB> lb;

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int nk = (int)((K + BK - 1) / BK);
  if (nk > 0) {
    la.load(A, lda, m0, M, 0, K, tid);
    lb.load(B, ldb, n0, N, 0, K, tid);
    la.store(smem, tid);
    lb.store(smem + A_BYTES, tid);
    __syncthreads();
  }

  const int lrow = lane & 31;
  const int lhalf = lane >> 5;

  for (int kt = 0; kt < nk; ++kt) {
    const int stage = kt & 1;
    char* sa = smem + stage * (A_BYTES + B_BYTES);
    char* sb = sa + A_BYTES;
    const bool more = kt + 1 < nk;
    if (more) {
      la.load(A, lda, m0, M, (int64_t)(kt + 1) * BK, K, tid);
      lb.load(B, ldb, n0, N, (int64_t)(kt + 1) * BK, K, tid);
    }
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int chunk = kk * 2 + lhalf;
      half8 af[TM], bf[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = wm * WTM + i * 32 + lrow;
        af[i] = as_half8(*reinterpret_cast<const u32x4*>(sa + r * ROWB + swz(r, chunk) * 16));
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int r = wn * WTN + j * 32 + lrow;
        bf[j] = as_half8(*reinterpret_cast<const u32x4*>(sb + r * ROWB + swz(r, chunk) * 16));
      }
      // D[n][m] = sum_k B^T[n][k] A^T[k][m]: lane holds column m, 4-runs of n.
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32(bf[j], af[i], acc[i][j]);
    }
    if (more) {
      char* na = smem + (stage ^ 1) * (A_BYTES + B_BYTES);
      la.store(na, tid);
      lb.store(na + A_BYTES, tid);
    }
    __syncthreads();
  }

  // ---- epilogue: C[m][n..n+3] = alpha * acc + beta * R[m][n..n+3] ----
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int64_t m = m0 + wm * WTM + i * 32 + lrow;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t n = n0 + wn * WTN + j * 32 + q * 8 + lhalf * 4;
        if (n >= N) continue;
        lt_half* p = C + m * ldc + n;
        const lt_half* pr = R + m * ldr + n;
        float v0 = alpha * acc[i][j][4 * q + 0];
        float v1 = alpha * acc[i][j][4 * q + 1];
        float v2 = alpha * acc[i][j][4 * q + 2];
        float v3 = alpha * acc[i][j][4 * q + 3];
        if (beta != 0.f) {
          const half4 c = *reinterpret_cast<const half4*>(pr);
          v0 += beta * (float)c[0];
          v1 += beta * (float)c[1];
          v2 += beta * (float)c[2];
          v3 += beta * (float)c[3];
        }
        half4 o;
        o[0] = (_Float16)v0; o[1] = (_Float16)v1; o[2] = (_Float16)v2; o[3] = (_Float16)v3;
        *reinterpret_cast<half4*>(p) = o;
      }
    }
  }
}

template <int BM, int BN, int WGM, int WGN, bool TA, bool TB>
hipError_t launch(const GemmArgs& g, hipStream_t s) {
  const int tiles_m = (int)((g.M + BM - 1) / BM);
  const int tiles_n = (int)((g.N + BN - 1) / BN);
  const int grid = tiles_m * tiles_n;
  hipLaunchKernelGGL((gemm_f16_kernel<BM, BN, WGM, WGN, TA, TB>), dim3(grid),
                     dim3(WGM * WGN * kWave), 0, s, g.M, g.N, g.K, g.alpha, g.A,
                     g.lda, g.B, g.ldb, g.beta, g.R, g.ldr, g.C, g.ldc, tiles_m, tiles_n);
  return hipGetLastError();
}

template <bool TA, bool TB>
hipError_t dispatch_tile(const GemmArgs& g, hipStream_t s) {
  // 256x256 tiles fill the chip once there are >= ~1 tile per CU; smaller
  // problems use 128x128 tiles so that more workgroups exist.
  const int64_t big_tiles = ((g.M + 255) / 256) * ((g.N + 255) / 256);
  if (big_tiles >= 192) return launch<256, 256, 2, 2, TA, TB>(g, s);
  return launch<128, 128, 2, 2, TA, TB>(g, s);
}

}  // namespace

hipError_t gemm_f16_launch(const GemmArgs& g, hipStream_t s) {
  if (g.transA) {
    return g.transB ? dispatch_tile<true, true>(g, s) : dispatch_tile<true, false>(g, s);
  }
  return g.transB ? dispatch_tile<false, true>(g, s) : dispatch_tile<false, false>(g, s);
}

}  // namespace lt
