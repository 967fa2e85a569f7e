// FP16 GEMM update C = alpha * op(A) op(B) + beta * R for gfx950.
//
// Sec. 4.1 of the paper describes the GEMM primitive (output tile loaded as
// the accumulation buffer) that serves the QKV / output / FFN projections in
// forward, data-gradient and weight-gradient form.  The MT-3000 dataflow
// (DDR -> GSM -> SM / AM staging, VLIW micro-kernel) is replaced here by the
// CDNA4 form of the same idea:
//   * a workgroup owns a BM x BN output tile held in MFMA accumulators
//     (16x16x32 FP16 MFMA, FP32 accumulate).  256x256 tiles of the forward
//     and data-gradient layouts use 4 waves, one per SIMD, each a 128x128
//     wave tile with its accumulators in AGPRs; their main loop is a fixed
//     sequence of asm statements (fragment reads a whole k-step ahead, MFMAs,
//     direct loads, counter waits), so that one wave keeps its matrix unit
//     fed without a second wave to cover its waits.  Every layout and the
//     split-K partial tiles use it; the half-size tail tiles and the
//     ragged-K form use 8 waves, two per SIMD, whose compiler-scheduled loop
//     relies on the other wave to cover LDS and barrier waits;
//   * K is walked in 64-wide slices, double-buffered in LDS.  Operands move
//     HBM -> LDS with direct buffer loads (16 B per lane, no register
//     staging), issued one slice ahead so that they overlap the current
//     slice's MFMA work -- the overlap of operand preparation with MACs that
//     the paper's micro-kernel pipeline provides.  In 8-wave tiles only one
//     wave per SIMD issues them ("loader waves"), with uniform (scalar)
//     addressing;
//   * each operand keeps its HBM orientation in LDS.  A K-contiguous operand
//     (forward A and B, dgrad A) is stored row-major; an M/N-contiguous one
//     (dgrad B, wgrad A and B) is stored k-major and read with the gfx950
//     LDS transpose read (ds_read_b64_tr_b16), so every (transA, transB)
//     runs the same MFMA loop at the same speed;
//   * LDS positions are XOR-swizzled so that both the direct loads and the
//     MFMA operand reads are free of bank conflicts (16 lanes x 16 B per LDS
//     cycle);
//   * tiles are ordered so that each XCD gets a contiguous range of tiles,
//     grouped eight tile-rows at a time for L2 reuse of A and B.
//   Buffer loads return zeros out of range, which provides the M, N and K
//   tails without branches.
//   A last wave of 256x256 tiles at most half full runs either as half-size
//   tiles (256x128 / 128x256) or, when the caller provides an FP32 workspace,
//   as 256x256 tiles whose K is split over several workgroups (epilogue 3
//   stores their partial sums; splitk_reduce_kernel adds them in a fixed
//   order and applies alpha, beta * R and the bias).  With a workspace, a
//   launch of less than about one wave of 256x256 tiles is split the same
//   way as a whole when the split gives twice the workgroups of 128x128 tiles
//   or keeps a long K loop per split; else it runs as 128x128 tiles.
#include <type_traits>
#include <utility>

#include "common.hpp"
#include "kernels.hpp"

namespace lt {
namespace {

// One operand tile: R rows (M for A, N for B) x BK.
//   KC  (K-contiguous in HBM): LDS row-major, CPR = BK/8 16-byte chunks per
//       row; chunk c of row r sits at position c ^ swz(r), which places the
//       16 consecutive rows read by one LDS cycle (16 lanes x 16 B) in 16
//       different bank groups.
//   !KC (row index contiguous in HBM): LDS k-major, 2R bytes per k-row;
//       16-byte chunk c (rows 8c..8c+7) of k-row k sits at position
//       kpos(c, k) = ((c >> 2) ^ (k & 3)) * 4 + ((c & 3) ^ 2 * ((k >> 3) & 1)):
//       the transpose reads of one MFMA operand (4 k-rows x 32 bytes per
//       16-lane group, groups 8 k-rows apart) then hit every bank once.
// Both are filled by direct global -> LDS loads issued as opaque
// instructions, so the caller orders them with explicit vmcnt waits.
template <int R, int BK, bool KC, int NT, bool PAIRED = false, int PB = 32>
struct Operand {
  static constexpr int BYTES = R * BK * 2;
  static constexpr int NINST = BYTES / 1024;        // 1 KiB direct loads per slice
  static constexpr int PERW = NINST / (NT / 64);     // ... per wave
  static_assert(NINST % (NT / 64) == 0, "slice must split across waves");
  static constexpr int CPR = BK / 8;                 // KC: 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;               // KC: rows per direct load
  static constexpr int KR_PER = 1024 / (2 * R);      // !KC: k-rows per direct load
  static constexpr int LPR = 64 / KR_PER;            // !KC: lanes per k-row
  static_assert(CPR >= 4 && CPR <= 16, "KC layout needs 32 <= BK <= 128");

  __device__ static __forceinline__ int swz(int r) { return (r / (16 / CPR)) & (CPR - 1); }
  // !KC chunk position; an involution in c for fixed k
  __device__ static __forceinline__ int kpos(int c, int k) {
    return (((c >> 2) ^ (k & 3)) << 2) | ((c & 3) ^ (((k >> 3) & 1) << 1));
  }

  uint32_t voff[PERW];
  const lt_half* base;
  int64_t ld, row0;
  uint32_t nrec;

  // PAIRED (K-contiguous only): tile row r = 32*blk + w reads matrix row
  // row0 + 32*(blk/2) + w, plus pair_off for odd blk: alternating 32-row
  // blocks of two row ranges (gate and up rows of a fused projection);
  // `rows` bounds the index inside each range.
  __device__ __forceinline__ void init(const lt_half* b, int64_t ld_, int64_t row0_, int64_t rows,
                                       int wave, int lane, int64_t pair_off = 0) {
    base = b;
    ld = ld_;
    row0 = row0_;
    if constexpr (PAIRED) {
      static_assert(KC, "paired rows are K-contiguous");
      nrec = 0x7fffffff;
#pragma unroll
      for (int t = 0; t < PERW; ++t) {
        const int r = (wave * PERW + t) * RPI + lane / CPR;
        const int64_t idx = row0 + PB * (r / (2 * PB)) + (r % PB);
        const int64_t abs_row = idx + ((r / PB) & 1 ? pair_off : 0);
        const int c = (lane % CPR) ^ swz(r);
        voff[t] = idx < rows ? (uint32_t)((abs_row * ld + c * 8) * 2) : kOOB;
      }
    } else if constexpr (KC) {
      // rows past the matrix fall outside the buffer and read as zero
      const int64_t nvalid = rows - row0 < R ? rows - row0 : R;
      nrec = (uint32_t)(nvalid * ld * 2);
#pragma unroll
      for (int t = 0; t < PERW; ++t) {
        const int r = (wave * PERW + t) * RPI + lane / CPR;
        const int c = (lane % CPR) ^ swz(r);
        voff[t] = (uint32_t)((r * ld + c * 8) * 2);
      }
    } else {
      nrec = 0x7fffffff;
#pragma unroll
      for (int t = 0; t < PERW; ++t) {
        const int k = (wave * PERW + t) * KR_PER + lane / LPR;
        const int c = kpos(lane % LPR, k);             // chunk that lands at position lane % LPR
        voff[t] = row0 + c * 8 < rows ? (uint32_t)((k * ld + c * 8) * 2) : kOOB;
      }
    }
  }

  // Direct loads of the slice starting at k0 into the LDS tile at `lds`;
  // kvalid < BK only for the last slice of a ragged K.
  __device__ __forceinline__ void load(char* lds, int64_t k0, int kvalid, int wave, int lane) const {
    if constexpr (KC) {
      // descriptor based at column k0 of row row0: the range shrinks by the
      // same 2*k0 bytes, so rows past the matrix still read as zero (paired
      // rows carry absolute offsets and explicit out-of-range offsets)
      const lt_half* b = PAIRED ? base + k0 : base + row0 * ld + k0;
      const uint32_t n = PAIRED ? nrec : nrec - (uint32_t)(k0 * 2);
      if (kvalid >= BK) {
#pragma unroll
        for (int t = 0; t < PERW; ++t) {
          const int i = wave * PERW + t;
          lds_dma16_opaque(b, n, lds + i * 1024, voff[t]);
        }
      } else {
#pragma unroll
        for (int t = 0; t < PERW; ++t) {
          const int i = wave * PERW + t;
          const int r = i * RPI + lane / CPR;
          const uint32_t off = ((lane % CPR) ^ swz(r)) * 8 >= kvalid ? kOOB : voff[t];
          lds_dma16_opaque(b, n, lds + i * 1024, off);
        }
      }
    } else {
      const lt_half* b = base + k0 * ld + row0;
      if (kvalid >= BK) {
#pragma unroll
        for (int t = 0; t < PERW; ++t) {
          const int i = wave * PERW + t;
          lds_dma16_opaque(b, nrec, lds + i * 1024, voff[t]);
        }
      } else {
#pragma unroll
        for (int t = 0; t < PERW; ++t) {
          const int i = wave * PERW + t;
          const uint32_t off = i * KR_PER + lane / LPR >= kvalid ? kOOB : voff[t];
          lds_dma16_opaque(b, nrec, lds + i * 1024, off);
        }
      }
    }
  }

  // buffer descriptor of the full K-contiguous slice at k0 (uniform)
  __device__ __forceinline__ u32x4 desc(int64_t k0) const {
    const uint64_t b = (uint64_t)(!KC ? base + k0 * ld + row0 : PAIRED ? base + k0 : base + row0 * ld + k0);
    u32x4 r;
    r[0] = __builtin_amdgcn_readfirstlane((uint32_t)b);
    r[1] = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32) & 0xffffu);
    r[2] = __builtin_amdgcn_readfirstlane(!KC || PAIRED ? nrec : nrec - (uint32_t)(k0 * 2));
    r[3] = 0x00020000u;
    return r;
  }

  // one direct load (index t of this wave's PERW) of the K-contiguous slice
  // at k0 with kv = clamp(K - k0, 0, BK) valid columns; kv = 0 fills the
  // tile with zeros and touches no memory (empty range)
  __device__ __forceinline__ void load1(char* lds, int64_t k0, int kv, int t, int wave,
                                        int lane) const {
    const int i = wave * PERW + t;
    if constexpr (KC) {
      const lt_half* b = PAIRED ? base + (kv > 0 ? k0 : 0) : base + row0 * ld + (kv > 0 ? k0 : 0);
      const uint32_t n = kv > 0 ? (PAIRED ? nrec : nrec - (uint32_t)(k0 * 2)) : 0u;
      const int r = i * RPI + lane / CPR;
      const uint32_t off = ((lane % CPR) ^ swz(r)) * 8 >= kv ? kOOB : voff[t];
      lds_dma16_opaque(b, n, lds + i * 1024, off);
    } else {
      const lt_half* b = base + (kv > 0 ? k0 * ld : 0) + row0;
      const uint32_t n = kv > 0 ? nrec : 0u;
      const uint32_t off = i * KR_PER + lane / LPR >= kv ? kOOB : voff[t];
      lds_dma16_opaque(b, n, lds + i * 1024, off);
    }
  }

  // K % 8 != 0 (K-contiguous tiles only; the k-major layout loads whole
  // k-rows, so its rows past K are already zero): the chunk of each row that
  // straddles K was loaded whole and holds the row's next elements in memory
  // (padding up to the leading dimension) past K.  Threads t < R of the
  // workgroup zero elements kvalid % 8 .. 7 of row t's chunk kvalid / 8 in
  // the LDS tile.  Called between the barrier after which the slice is
  // resident and a barrier before its first fragment read.
  __device__ __forceinline__ void zero_k_tail(char* lds, int kvalid, int t) const {
    static_assert(KC, "k-major tiles need no fix-up");
    if (t < 0 || t >= R) return;
    const int e0 = kvalid & 7;
    char* q = lds + t * (CPR * 16) + (((kvalid >> 3) ^ swz(t)) << 4);
    u32x4 v = *reinterpret_cast<const u32x4*>(q);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      // 16-bit elements 2w and 2w + 1 of the chunk
      const uint32_t keep = (2 * w < e0 ? 0x0000ffffu : 0u) | (2 * w + 1 < e0 ? 0xffff0000u : 0u);
      v[w] &= keep;
    }
    *reinterpret_cast<u32x4*>(q) = v;
  }

  // MFMA operand (16x16x32): rows rb..rb+15 (lane row = lane % 16),
  // reduction indices kk*32 + 8*(lane/16) + 0..7.
  __device__ __forceinline__ half8 frag(const char* lds, int rb, int kk, int lane) const {
    if constexpr (KC) {
      const int r = rb + (lane & 15);
      const int c = kk * 4 + (lane >> 4);
      return as_half8(*reinterpret_cast<const u32x4*>(lds + r * (CPR * 16) + ((c ^ swz(r)) << 4)));
    } else {
      // Two transpose reads (h = 0, 1).  Within 16-lane group G = L/16, lane
      // s = L%16 reads the 4 rows at m = rb + 4*(s%4) of k-row
      // kk*32 + 8G + 4h + s/4, and receives row rb + s of k-rows
      // kk*32 + 8G + 4h + 0..3.
      const int m = rb + 4 * (lane & 3);
      const int c = m >> 3;
      const int inoff = (m & 7) * 2;
      v4s part[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int k = kk * 32 + 8 * (lane >> 4) + 4 * h + ((lane & 15) >> 2);
        part[h] = lds_read_tr16(lds + k * (2 * R) + kpos(c, k) * 16 + inoff);
      }
      return as_half8(pack_v4s_pair(part[0], part[1]));
    }
  }
};

// s_waitcnt vmcnt(n * PER), n clamped to [0, MAXN]: wait until at most n
// slices of direct loads (PER instructions each) are still in flight.
template <int PER, int MAXN>
__device__ __forceinline__ void wait_slices(int n) {
  if constexpr (MAXN > 0) {
    if (n >= MAXN) {
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(MAXN * PER) : "memory");
      return;
    }
    wait_slices<PER, MAXN - 1>(n);
  } else {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }
}

// ---- building blocks of the 4-wave main loop ----
// The loop is written as asm statements that the compiler keeps in program
// order (volatile asm).  Two rules make that safe with the compiler still
// allocating the registers:
//   * a fragment read issued by asm is, to the compiler, complete at once; its
//     registers must not be read, copied or reused before the explicit
//     lgkmcnt wait.  Every fragment is consumed only by MFMA asm after that
//     wait (xfence re-defines the two halves of a transposed fragment after
//     the wait, so that joining them happens there), and the fragments read
//     for a step that never runs are kept allocated until the final wait
//     (xkeep);
//   * MFMAs issued by asm are not seen by the compiler's hazard checks: the
//     wait states before any other instruction reads an accumulator are in
//     one statement that takes every accumulator as an operand.
template <int... I, class F>
__device__ __forceinline__ void sfor_impl(std::integer_sequence<int, I...>, F&& f) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void sfor(F&& f) {
  sfor_impl(std::make_integer_sequence<int, N>{}, f);
}
// direct 16-byte-per-lane load into LDS at m0 = mbase + OFF (uniform)
template <int OFF>
__device__ __forceinline__ void dma16_at(uint32_t mbase, uint32_t voff, u32x4 desc) {
  asm volatile("s_add_u32 m0, %0, %3\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(mbase), "v"(voff), "s"(desc), "n"(OFF)
               : "memory");
}
// LDS transpose read of one half of a k-major fragment
template <int OFF>
__device__ __forceinline__ void xrd_tr(u32x2& d, uint32_t a) {
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(d) : "v"(a), "n"(OFF));
}
// the two halves are (re)defined here: nothing that joins them moves above
__device__ __forceinline__ void xfence(u32x2& a, u32x2& b) {
  asm volatile("" : "+v"(a), "+v"(b));
}
// keep a value's registers allocated up to this point
__device__ __forceinline__ void xkeep(const half8& a) { asm volatile("" ::"v"(a)); }
__device__ __forceinline__ void xkeep(const u32x2& a, const u32x2& b) { asm volatile("" ::"v"(a), "v"(b)); }
// read q of a 4-wave step: fragments in the order B0, A0, B1..B7, A1..A7,
// ra (rb) reads per A (B) fragment; op 0 = A, 1 = B
struct X4Rd {
  int op, f, h;
};
constexpr X4Rd x4_read(int q, int ra, int rb) {
  for (int e = 0; e < 16; ++e) {
    const int op = e == 0 ? 1 : e == 1 ? 0 : e <= 8 ? 1 : 0;
    const int f = e <= 1 ? 0 : e <= 8 ? e - 1 : e - 8;
    const int n = op ? rb : ra;
    if (q < n) return X4Rd{op, f, q};
    q -= n;
  }
  return X4Rd{-1, 0, 0};
}
// reads issued after MFMA idx of a step: [x4_q0(idx), x4_q0(idx + 1))
constexpr int x4_q0(int idx, int nrd) {
  const int q = idx < 2 ? 0 : ((idx - 2) * nrd + 47) / 48;
  return q < nrd ? q : nrd;
}
// LDS read of a K-contiguous fragment
template <int OFF>
__device__ __forceinline__ void xrd(half8& d, uint32_t a) {
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(d) : "v"(a), "n"(OFF));
}
// c += a b (16x16x32), c in AGPRs
__device__ __forceinline__ void xmma(f32x4& c, const half8& a, const half8& b) {
  asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
}

__device__ __forceinline__ float sigmoid_f(float x) { return 1.f / (1.f + __expf(-x)); }

template <int BM, int BN, int WGM, int WGN, int BK, int NS, bool TA, bool TB, int EPI,
          bool RK = false>
__global__ void __launch_bounds__(WGM * WGN * kWave)
gemm_f16_kernel(int64_t M, int64_t N, int64_t K, float alpha,
                const lt_half* __restrict__ A, int64_t lda,
                const lt_half* __restrict__ B, int64_t ldb, float beta,
                const lt_half* R, int64_t ldr, lt_half* C, int64_t ldc, int tiles_m,
                int tiles_n, int group_m, lt_half* X1, int64_t ldx1, int64_t Fb, int64_t P,
                const lt_half* bias) {
  constexpr int NT = WGM * WGN * kWave;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;   // wave tile
  constexpr int TM = WTM / 16, TN = WTN / 16;     // 16x16 MFMA blocks per wave
  static_assert(EPI != 1 || TB, "paired gate/up tiles: K-contiguous weights");
  // Loader waves: in an 8-wave tile only waves 0-3 (one per SIMD) issue the
  // direct loads, twice as many each; the other four waves only compute.
  // Fewer waves feeding the shared load queues measured 4-13% faster in
  // every layout.
  constexpr int NWAVE = NT / kWave;
  constexpr int LOADERS = NWAVE >= 8 ? 4 : NWAVE;
  constexpr bool SPLIT_ISSUE = LOADERS < NWAVE;
  using OA = Operand<BM, BK, !TA, LOADERS * kWave>;
  // EPI 1: a wave's columns are WTN/2 gate rows and the same WTN/2 up rows
  using OB = Operand<BN, BK, TB, LOADERS * kWave, EPI == 1, WTN / 2>;
  constexpr int STAGE = OA::BYTES + OB::BYTES;
  constexpr int PER_SLICE = OA::PERW + OB::PERW;  // direct loads per wave per slice
  static_assert(NS >= 2 && (NS - 1) * PER_SLICE <= 63, "vmcnt range");
  __shared__ __attribute__((aligned(1024))) char smem[NS * STAGE];

  if constexpr (EPI == 3) {
    // split-K unit blockIdx.y of gridDim.y: slices [y*kc, (y+1)*kc) of the
    // reduction, as a product of its own over the offset operands
    const int64_t kc = ((K + BK - 1) / BK + gridDim.y - 1) / gridDim.y;
    const int64_t k0 = (int64_t)blockIdx.y * kc * BK;
    A += TA ? k0 * lda : k0;
    B += TB ? k0 : k0 * ldb;
    K = K - k0 < kc * BK ? K - k0 : kc * BK;
  }
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar addressing
  const int wm = wave / WGN;
  const int wn = wave % WGN;

  // ---- tile ordering: contiguous range per XCD (consecutive workgroups go
  // to the 8 XCDs in turn), then column-major within groups of group_m
  // tile rows, so that the tiles resident on one XCD share A and B panels ----
  int pid = blockIdx.x;
  const int nwg = gridDim.x;
  if ((nwg & 7) == 0) {
    const int per = nwg >> 3;
    pid = (pid & 7) * per + (pid >> 3);
  }
  const int group_size = group_m * tiles_n;
  const int first_m = (pid / group_size) * group_m;
  const int gm = min(tiles_m - first_m, group_m);
  const int in_group = pid % group_size;
  const int64_t m0 = (int64_t)(first_m + in_group % gm) * BM;
  // EPI 1: a tile covers BN/2 gate columns and the same BN/2 up columns
  const int64_t n0 = (int64_t)(in_group / gm) * (EPI == 1 ? BN / 2 : BN);

  OA oa;
  OB ob;
  const bool loader = wave < LOADERS;
  if (loader) oa.init(A, lda, m0, M, wave, lane);
  if constexpr (EPI == 1)
    { if (loader) ob.init(B, ldb, n0, Fb, wave, lane, P); }
  else
    { if (loader) ob.init(B, ldb, n0, N, wave, lane); }

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[i][j][r] = 0.f;

  const int nk = (int)((K + BK - 1) / BK);
  auto kvalid = [&](int kt) {
    const int64_t rem = K - (int64_t)kt * BK;
    return rem >= BK ? BK : (int)rem;
  };
  auto stage_of = [&](int kt) { return smem + (kt % NS) * STAGE; };
  auto issue = [&](int kt) {
    if (!loader) return;
    char* st = stage_of(kt);
    oa.load(st, (int64_t)kt * BK, kvalid(kt), wave, lane);
    ob.load(st + OA::BYTES, (int64_t)kt * BK, kvalid(kt), wave, lane);
  };
  // RK (ragged K, not a multiple of 8; plain epilogue only): the last
  // slice's K-contiguous tiles are cleared past K, between two barriers.  A
  // separate instantiation, so that no branch sits at the slice barrier of
  // the other kernels (their first MFMAs after it are scheduled across it).
  static_assert(!RK || EPI == 0, "ragged K: plain epilogue");
  constexpr bool KFIX = RK && (!TA || TB);
  static_assert(!KFIX || (TA ? 0 : BM) + (TB ? BN : 0) <= NT, "one thread per tile row");
  auto fix_k_tail = [&](int kt) {
    if constexpr (KFIX) {
      char* st = stage_of(kt);
      const int kv = kvalid(kt);
      if constexpr (!TA) oa.zero_k_tail(st, kv, tid);
      if constexpr (TB) ob.zero_k_tail(st + OA::BYTES, kv, TA ? tid : tid - BM);
      __syncthreads();
    }
  };
  constexpr bool ragged_k = KFIX;

  constexpr bool X4 = NT == 256 && BM == 256 && BN == 256 && EPI <= 3 && !RK && BK == 64 && NS == 2;
  if constexpr (X4) {
    // One wave per SIMD, 128x128 wave tiles, accumulators in AGPRs.  Every
    // fragment read, MFMA and counter wait of the loop is an ordered asm
    // statement: a step's MFMAs run on one register set while the reads of
    // the next step fill the other, all issued in the step's first 48 MFMAs;
    // after the slice barrier the 16 direct loads of slice kt+2 are spread
    // over the step's MFMAs.
    static_assert(TM == 8 && TN == 8 && STAGE == 65536 && OA::BYTES == 32768, "X4 shape");
    constexpr bool AK = !TA, BKC = TB;           // K-contiguous operands (row reads)
    constexpr int XRA = AK ? 1 : 2, XRB = BKC ? 1 : 2;
    constexpr int NRD = 8 * (XRA + XRB);        // LDS reads per step
    half8 xa[2][8], xb[2][8];                  // fragments of K-contiguous operands
    u32x2 ta[2][8][2], tb[2][8][2];            // ... of k-major ones (two transpose reads)
    const uint32_t sbase = (uint32_t)(uintptr_t)smem;
    // K-contiguous: fragment f of k-step kk at r[stage][kk] + 2048 f
    auto lterm = [&](int kk) {
      const int r = lane & 15;
      const int c = kk * 4 + (lane >> 4);
      return (uint32_t)(r * 128 + ((c ^ (r >> 1)) << 4));
    };
    // k-major: read h of fragment f, k-step kk at z[stage][f] + 16384 kk + 2048 h
    // (the fragment's XOR-swizzled position differs per lane only in address
    // bits 5..7, which no other term touches)
    auto yterm = [&](int wx) {
      const int kl = (lane >> 2) & 3, g1 = (lane >> 4) & 1;
      return (uint32_t)(((8 * (lane >> 4) + kl) * 512 + 256 * wx + 16 * ((lane & 3) >> 1) + 8 * (lane & 1)) |
                        (kl << 6) | (g1 << 5));
    };
    uint32_t ra[2][2], rb[2][2], za[2][8], zb[2][8];
#pragma unroll
    for (int p = 0; p < 2; ++p) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        ra[p][kk] = sbase + p * STAGE + wm * 16384 + lterm(kk);
        rb[p][kk] = sbase + p * STAGE + OA::BYTES + wn * 16384 + lterm(kk);
      }
#pragma unroll
      for (int f = 0; f < 8; ++f) {
        const uint32_t cf = ((f >> 1) << 6) | ((f & 1) << 5);
        za[p][f] = (sbase + p * STAGE + yterm(wm)) ^ cf;
        zb[p][f] = (sbase + p * STAGE + OA::BYTES + yterm(wn)) ^ cf;
      }
    }
    // read q of the step into set D, from stage P, k-step KK
    auto xread = [&](auto Q_, auto D_, auto P_, auto KK_) __attribute__((always_inline)) {
      constexpr X4Rd r = x4_read(decltype(Q_)::value, XRA, XRB);
      constexpr int D = decltype(D_)::value, P = decltype(P_)::value, KK = decltype(KK_)::value;
      if constexpr (r.op == 0) {
        if constexpr (AK) xrd<r.f * 2048>(xa[D][r.f], ra[P][KK]);
        else xrd_tr<KK * 16384 + r.h * 2048>(ta[D][r.f][r.h], za[P][r.f]);
      } else {
        if constexpr (BKC) xrd<r.f * 2048>(xb[D][r.f], rb[P][KK]);
        else xrd_tr<KK * 16384 + r.h * 2048>(tb[D][r.f][r.h], zb[P][r.f]);
      }
    };
    // set S resident: wait for its reads; the k-major halves are joined
    // only after the wait
    auto xwait = [&](auto S_) __attribute__((always_inline)) {
      constexpr int S = decltype(S_)::value;
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
      for (int f = 0; f < 8; ++f) {
        if constexpr (!AK) xfence(ta[S][f][0], ta[S][f][1]);
        if constexpr (!BKC) xfence(tb[S][f][0], tb[S][f][1]);
      }
    };
    auto fragA = [&](auto S_, int i) __attribute__((always_inline)) {
      constexpr int S = decltype(S_)::value;
      if constexpr (AK) return xa[S][i];
      else return __builtin_bit_cast(half8, __builtin_shufflevector(ta[S][i][0], ta[S][i][1], 0, 1, 2, 3));
    };
    auto fragB = [&](auto S_, int j) __attribute__((always_inline)) {
      constexpr int S = decltype(S_)::value;
      if constexpr (BKC) return xb[S][j];
      else return __builtin_bit_cast(half8, __builtin_shufflevector(tb[S][j][0], tb[S][j][1], 0, 1, 2, 3));
    };
    using Z0 = std::integral_constant<int, 0>;
    using Z1 = std::integral_constant<int, 1>;
    // prologue: slices 0 and 1 in flight, slice 0 resident, its first
    // k-step's fragments into set 0
    auto kv_of = [&](int kt) {
      const int64_t rem = K - (int64_t)kt * BK;
      return rem >= BK ? BK : rem > 0 ? (int)rem : 0;
    };
#pragma unroll
    for (int sl = 0; sl < NS; ++sl)
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        oa.load1(smem + sl * STAGE, (int64_t)sl * BK, kv_of(sl), t, wave, lane);
        ob.load1(smem + sl * STAGE + OA::BYTES, (int64_t)sl * BK, kv_of(sl), t, wave, lane);
      }
    asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
    __syncthreads();
    sfor<NRD>([&](auto Q) __attribute__((always_inline)) { xread(Q, Z0{}, Z0{}, Z0{}); });
    const uint32_t mbase = __builtin_amdgcn_readfirstlane(sbase + wave * 8 * 1024);
    // One 32-wide k-step on set S; the next step's fragments come from
    // stage P, k-step KK.  LD: 0 no loads, 1 loads of any slice at lk0 (lkv
    // valid columns, masked) into the stage at lst, 2 loads of a full slice
    // through the descriptors dA, dB into stage LP.
    auto xstep = [&](auto S_, auto P_, auto KK_, auto LD_, char* lst, int64_t lk0, int lkv,
                     auto LP_, u32x4 dA, u32x4 dB) __attribute__((always_inline)) {
      constexpr int S = decltype(S_)::value;
      constexpr int LD = decltype(LD_)::value;
      constexpr int LP = decltype(LP_)::value;
      xwait(S_);
      sfor<64>([&](auto IDX) __attribute__((always_inline)) {
        constexpr int idx = decltype(IDX)::value;
        constexpr int i = idx / 8, j = idx % 8;
        xmma(acc[i][j], fragB(S_, j), fragA(S_, i));
        // the slice barrier after the second step's first two MFMAs (they
        // run on registers and cover the barrier's skew): slice kt+1
        // resident for every wave, and nobody reads slice kt's stage any more
        if constexpr (S == 1 && idx == 1) {
          asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
          __syncthreads();
        }
        constexpr int q0 = x4_q0(idx, NRD), q1 = x4_q0(idx + 1, NRD);
        static_assert(q1 - q0 <= 2, "at most two reads per MFMA");
        sfor<2>([&](auto R_) __attribute__((always_inline)) {
          constexpr int q = q0 + decltype(R_)::value;
          if constexpr (q < q1) xread(std::integral_constant<int, q>{}, std::integral_constant<int, S ^ 1>{}, P_, KK_);
        });
        if constexpr (LD == 1 && idx % 4 == 1) {
          constexpr int t = idx / 4;
          if constexpr (t < 8) oa.load1(lst, lk0, lkv, t, wave, lane);
          else ob.load1(lst + OA::BYTES, lk0, lkv, t - 8, wave, lane);
        }
        if constexpr (LD == 2 && idx % 4 == 1) {
          constexpr int t = idx / 4;
          if constexpr (t < 8) dma16_at<LP * STAGE + t * 1024>(mbase, oa.voff[t], dA);
          else dma16_at<LP * STAGE + OA::BYTES + (t - 8) * 1024>(mbase, ob.voff[t - 8], dB);
        }
      });
    };
    using NO = std::integral_constant<int, 0>;
    using YS = std::integral_constant<int, 1>;
    using FS = std::integral_constant<int, 2>;
    const u32x4 dz = {0, 0, 0, 0};
    // Slices are taken in pairs (stage 0, stage 1).  For an odd slice count
    // the last pair's second slice lies past K: its stage was filled with
    // zeros, so its products add exact zeros (an accumulator that starts at
    // +0 never holds -0), and the loop body has no branch.
    auto xslice = [&](int kt, auto P_, auto FAST_) __attribute__((always_inline)) {
      constexpr int P = decltype(P_)::value;
      constexpr bool FAST = decltype(FAST_)::value;
      xstep(Z0{}, P_, Z1{}, NO{}, nullptr, 0, 0, P_, dz, dz);
      const int64_t lk0 = (int64_t)(kt + 2) * BK;
      if constexpr (FAST)
        xstep(Z1{}, std::integral_constant<int, P ^ 1>{}, Z0{}, FS{}, nullptr, 0, 0, P_,
              oa.desc(lk0), ob.desc(lk0));
      else
        xstep(Z1{}, std::integral_constant<int, P ^ 1>{}, Z0{}, YS{}, smem + P * STAGE, lk0,
              kv_of(kt + 2), P_, dz, dz);
    };
    // pairs whose loads (slices kt+2, kt+3) are whole slices inside K take
    // the unmasked loads
    const int nkf = (int)(K / BK);
    int kt = 0;
    for (; kt + 3 < nkf; kt += 2) {
      xslice(kt, Z0{}, std::true_type{});
      xslice(kt + 1, Z1{}, std::true_type{});
    }
    for (; kt < nk; kt += 2) {
      xslice(kt, Z0{}, std::false_type{});
      xslice(kt + 1, Z1{}, std::false_type{});
    }
    // The last step read the fragments of a step that never runs: their
    // registers stay allocated until those reads have landed, so that no
    // epilogue value is placed where a late LDS result would overwrite it.
    // The MFMAs are opaque to the compiler's hazard checks: the wait states
    // before the accumulators may be read sit in one statement that takes
    // every accumulator, so no spill or copy of one can be placed between
    // the last MFMA and the wait.
#define X4_ROW(i) "+a"(acc[i][0]), "+a"(acc[i][1]), "+a"(acc[i][2]), "+a"(acc[i][3]), \
                  "+a"(acc[i][4]), "+a"(acc[i][5]), "+a"(acc[i][6]), "+a"(acc[i][7])
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n\t"
                 "s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7"
                 : X4_ROW(0), X4_ROW(1), X4_ROW(2), X4_ROW(3), X4_ROW(4), X4_ROW(5), X4_ROW(6), X4_ROW(7)
                 :
                 : "memory");
#undef X4_ROW
#pragma unroll
    for (int f = 0; f < 8; ++f) {
      if constexpr (AK) xkeep(xa[0][f]);
      else xkeep(ta[0][f][0], ta[0][f][1]);
      if constexpr (BKC) xkeep(xb[0][f]);
      else xkeep(tb[0][f][0], tb[0][f][1]);
    }
  } else {
  // Fragments: A in place (each re-read right after its last use), B
  // double-buffered (used by every A row of a step).
  half8 fa[TM], fb[2][TN];

  // ---- prologue: slices 0 .. NS-1 in flight, wait for slice 0 ----
#pragma unroll
  for (int s = 0; s < NS; ++s)
    if (s < nk) issue(s);
  wait_slices<PER_SLICE, NS - 1>(min(NS - 1, nk - 1));
  __syncthreads();
  if (ragged_k && nk == 1) fix_k_tail(0);

  // One MFMA step on (fa, fb[S]).  With LD, the fragments of the next step
  // (32-wide k-step kk of stage st) are read meanwhile: after the MFMAs of A
  // row i come the reads of fa[i] and, for the first TN rows, of fb[S^1][i],
  // so every read overlaps the MFMAs that follow it.  S and LD are
  // compile-time constants so that the fragment arrays stay in registers.
  constexpr int KS = BK / 32;
  static_assert(KS % 2 == 0, "B fragments alternate buffers within a slice");
  constexpr int RA = TA ? 2 : 1;   // LDS reads per A fragment (transpose reads: 2)
  constexpr int RB = TB ? 1 : 2;   // ... per B fragment
  // B fragments read after A row i: fb[j] for j % TM == i (BPI of them while
  // i < NBI; one for each of the first TN rows when TN <= TM).
  static_assert(TN <= TM || TN % TM == 0, "B fragments must spread over the A rows");
  constexpr int BPI = TN <= TM ? 1 : TN / TM;
  constexpr int NBI = TN <= TM ? TN : TM;
  // First fragments, read in the order the steps read theirs (after A row i:
  // the B fragments of row i, then A fragment i).  The LDS counter waits at
  // the top of the slice loop then hold for the entry from here as well as
  // for the loop's back edge; with all B fragments read last, the waits the
  // compiler derived for the merged entry stalled each slice's first MFMAs
  // on the reads of the previous step's last rows.
  if (nk > 0) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      if (i < NBI) {
#pragma unroll
        for (int q = 0; q < BPI; ++q)
          fb[0][i + q * TM] = ob.frag(smem + OA::BYTES, wn * WTN + (i + q * TM) * 16, 0, lane);
      }
      fa[i] = oa.frag(smem, wm * WTM + i * 16, 0, lane);
    }
  }
  auto step = [&](auto S_, auto LD_, const char* st, int kk, auto&& after_first_row) {
    constexpr int S = decltype(S_)::value;
    constexpr bool LD = decltype(LD_)::value;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = mfma16(fb[S][j], fa[i], acc[i][j]);
      if (i == 0) after_first_row(std::integral_constant<int, 0>{});
      if (i == TM / 2) after_first_row(std::integral_constant<int, 1>{});
      if constexpr (LD) {
        if (i < NBI) {
#pragma unroll
          for (int q = 0; q < BPI; ++q) {
            const int j = i + q * TM;
            fb[S ^ 1][j] = ob.frag(st + OA::BYTES, wn * WTN + j * 16, kk, lane);
          }
        }
        fa[i] = oa.frag(st, wm * WTM + i * 16, kk, lane);
      }
    }
    if constexpr (LD) {
#pragma unroll
      for (int i = 0; i < NBI; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, TN, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, BPI * RB + RA, 0);
      }
#pragma unroll
      for (int i = NBI; i < TM; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, TN, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, RA, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  using C0 = std::integral_constant<int, 0>;
  using C1 = std::integral_constant<int, 1>;
  using YES = std::integral_constant<bool, true>;

  // Per slice kt: step 0, then the barrier after which slice kt+1 is
  // resident and nobody reads slice kt's stage any more.  Step 1 runs on
  // registers while reading slice kt+1's first fragments; after its first
  // MFMAs are queued, the loads of slice kt+NS go into the freed stage,
  // almost a full slice ahead of their wait.
  for (int kt = 0; kt < nk; ++kt) {
    static_assert(KS == 2, "one step before and one after the slice barrier");
    step(C0{}, YES{}, stage_of(kt), 1, [](auto) {});
    // slices after kt+1 that are already issued may stay in flight
    wait_slices<PER_SLICE, NS - 2>(min(kt + NS - 1, nk - 1) - (kt + 1));
    __syncthreads();
    if (ragged_k && kt + 2 == nk) fix_k_tail(kt + 1);
    // (after the last slice these reads of a stale stage are unused; reading
    // unconditionally keeps one copy of the fragments live across the loop)
    step(C1{}, YES{}, stage_of(kt + 1), 0, [&](auto part) {
      constexpr int PART = decltype(part)::value;
      if (!loader || kt + NS >= nk) return;
      if constexpr (!SPLIT_ISSUE) {
        if constexpr (PART == 0) issue(kt + NS);
      } else {
        // loader waves: A's loads after the first A row, B's after row TM/2
        char* st = stage_of(kt + NS);
        if constexpr (PART == 0)
          oa.load(st, (int64_t)(kt + NS) * BK, kvalid(kt + NS), wave, lane);
        else
          ob.load(st + OA::BYTES, (int64_t)(kt + NS) * BK, kvalid(kt + NS), wave, lane);
      }
    });
  }

  }  // !X4

  // ---- epilogue ----
  // lane holds column m = ... + lane % 16 and rows n = ... + 4*(lane/16) + 0..3
  if constexpr (EPI == 3) {
    // FP32 partial sums of this split, unscaled: W[split][m][n], ldc floats
    // per row (C is the workspace)
    float* W = reinterpret_cast<float*>(C) + (int64_t)blockIdx.y * M * ldc;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int64_t m = m0 + wm * WTM + i * 16 + (lane & 15);
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int64_t n = n0 + wn * WTN + j * 16 + 4 * (lane >> 4);
        if (m < M && n < N)
          *reinterpret_cast<float4*>(W + m * ldc + n) =
              make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
      }
    }
  } else if constexpr (EPI == 1) {
    // accumulator blocks j and j + TN/2 hold the gate and up columns of the
    // same n: GU[m][n] = G, GU[m][F + n] = U, A[m][n] = silu(G) U (from the
    // FP32 values, one rounding each)
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int64_t m = m0 + wm * WTM + i * 16 + (lane & 15);
      if (m >= M) continue;
#pragma unroll
      for (int j = 0; j < TN / 2; ++j) {
        const int64_t n = n0 + wn * (WTN / 2) + j * 16 + 4 * (lane >> 4);
        if (n >= Fb) continue;
        half4 g4, u4, a4;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float g = alpha * acc[i][j][e];
          const float u = alpha * acc[i][j + TN / 2][e];
          g4[e] = (_Float16)g;
          u4[e] = (_Float16)u;
          a4[e] = (_Float16)(g * sigmoid_f(g) * u);
        }
        *reinterpret_cast<half4*>(C + m * ldc + n) = g4;
        *reinterpret_cast<half4*>(C + m * ldc + P + n) = u4;
        *reinterpret_cast<half4*>(X1 + m * ldx1 + n) = a4;
      }
    }
  } else {
    // The rows of the wave tile are handled in NG groups: the loads of group
    // g (beta * R, or G and U for the SwiGLU gradient) are issued before the
    // stores of group g - 1, and group g's values are computed only after
    // those stores are in flight.  Loads and stores share one completion
    // counter, so a load consumed after a store is waited for together with
    // that store: in this order every group costs one overlapped memory
    // round trip instead of one per 16x16 block.  R may be C itself; groups
    // touch disjoint rows, so loading group g before storing group g - 1 is
    // safe.
    constexpr int NL = EPI == 2 ? 2 : 1;               // half4 per block and lane, in and out
    constexpr int NG = EPI == 2 ? (TM >= 4 ? 4 : TM) : (TM >= 2 ? 2 : 1);
    constexpr int IG = TM / NG;                        // accumulator rows per group
    static_assert(TM % NG == 0, "row groups");
    const bool reads = EPI == 2 || beta != 0.f;        // uniform over the grid
    const int64_t mb = m0 + wm * WTM + (lane & 15);
    const int64_t nb = n0 + wn * WTN + 4 * (lane >> 4);
    half4 in[IG][TN][NL];
    half4 out[IG][TN][NL];
    // bias (epilogue 0): the same 4 columns for every accumulator row
    const bool has_bias = EPI == 0 && bias != nullptr;   // uniform over the grid
    half4 bv[TN];
    if (has_bias) {
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int64_t n = nb + j * 16;
        if (n + 4 <= N) {
          bv[j] = *reinterpret_cast<const half4*>(bias + n);
        } else {
          // bias holds exactly N entries
#pragma unroll
          for (int e = 0; e < 4; ++e)
            bv[j][e] = n + e < N ? __builtin_bit_cast(_Float16, bias[n + e]) : (_Float16)0;
        }
      }
    }

    // loads are unconditional, from addresses clamped into the matrix
    // (values of out-of-range blocks are never stored): no branch between
    // the loads keeps the completion-counter waits exact
    auto load_group = [&](int g) {
#pragma unroll
      for (int ii = 0; ii < IG; ++ii) {
        const int64_t m = mb + (g * IG + ii) * 16;
        const int64_t mc = m < M ? m : M - 1;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          // a 4-column group that starts before N is read whole: rows are
          // readable up to N rounded up to 8 (leading dimensions are
          // multiples of 8)
          const int64_t n = nb + j * 16;
          const int64_t nc = n < N ? n : 0;
          if constexpr (EPI == 2) {
            in[ii][j][0] = *reinterpret_cast<const half4*>(X1 + mc * ldx1 + nc);
            in[ii][j][1] = *reinterpret_cast<const half4*>(X1 + mc * ldx1 + P + nc);
          } else {
            in[ii][j][0] = *reinterpret_cast<const half4*>(R + mc * ldr + nc);
          }
        }
      }
    };
    auto compute_group = [&](int g) {
#pragma unroll
      for (int ii = 0; ii < IG; ++ii)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int i = g * IG + ii;
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = alpha * acc[i][j][e];
          if constexpr (EPI == 2) {
            // v = dA; dG = dA U s (1 + G (1 - s)),  dU = dA silu(G),  s = sigmoid(G)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float gv = (float)in[ii][j][0][e], uv = (float)in[ii][j][1][e];
              const float sg = sigmoid_f(gv);
              out[ii][j][0][e] = (_Float16)(v[e] * uv * sg * (1.f + gv * (1.f - sg)));
              out[ii][j][1][e] = (_Float16)(v[e] * gv * sg);
            }
          } else {
            if (reads) {
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] += beta * (float)in[ii][j][0][e];
            }
            if (has_bias) {
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] += (float)bv[j][e];
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) out[ii][j][0][e] = (_Float16)v[e];
          }
        }
    };
    auto store_group = [&](int g) {
#pragma unroll
      for (int ii = 0; ii < IG; ++ii) {
        const int64_t m = mb + (g * IG + ii) * 16;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int64_t n = nb + j * 16;
          if (m < M && n < N) {
            if (EPI == 2 || n + 4 <= N) {
              *reinterpret_cast<half4*>(C + m * ldc + n) = out[ii][j][0];
              if constexpr (EPI == 2)
                *reinterpret_cast<half4*>(C + m * ldc + P + n) = out[ii][j][1];
            } else {
              // the last 1-3 columns of a ragged N (plain epilogue only),
              // taken from the packed bits (the element-indexed form of
              // these stores compiled to stores of element 0 only)
              const uint64_t bits = __builtin_bit_cast(uint64_t, out[ii][j][0]);
              C[m * ldc + n] = (lt_half)bits;
              if (n + 1 < N) C[m * ldc + n + 1] = (lt_half)(bits >> 16);
              if (n + 2 < N) C[m * ldc + n + 2] = (lt_half)(bits >> 32);
            }
          }
        }
      }
    };
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      if (reads) load_group(g);
      if (g > 0) store_group(g - 1);
      compute_group(g);
    }
    store_group(NG - 1);
  }
}

template <int BM, int BN, int WGM, int WGN, int BK, int NS, bool TA, bool TB, int EPI,
          bool RK = false>
hipError_t launch(const GemmArgs& g, hipStream_t s, int splits = 1) {
  const int tiles_m = (int)((g.M + BM - 1) / BM);
  const int tiles_n = EPI == 1 ? (int)((g.F + BN / 2 - 1) / (BN / 2)) : (int)((g.N + BN - 1) / BN);
  if constexpr (BM == 256 && BN == 256 && WGM == 2 && WGN == 4 && EPI <= 3 && !RK && BK == 64 && NS == 2) {
    hipLaunchKernelGGL((gemm_f16_kernel<256, 256, 2, 2, 64, 2, TA, TB, EPI, false>),
                       dim3(tiles_m * tiles_n, splits), dim3(4 * kWave), 0, s, g.M, g.N, g.K, g.alpha,
                       g.A, g.lda, g.B, g.ldb, g.beta, g.R, g.ldr, g.C, g.ldc, tiles_m, tiles_n, 8,
                       g.X1, g.ldx1, g.F, g.pair_off > 0 ? g.pair_off : g.F, g.bias);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((gemm_f16_kernel<BM, BN, WGM, WGN, BK, NS, TA, TB, EPI, RK>),
                     dim3(tiles_m * tiles_n, splits), dim3(WGM * WGN * kWave), 0, s, g.M, g.N, g.K, g.alpha,
                     g.A, g.lda, g.B, g.ldb, g.beta, g.R, g.ldr, g.C, g.ldc, tiles_m, tiles_n, 8,
                     g.X1, g.ldx1, g.F, g.pair_off > 0 ? g.pair_off : g.F, g.bias);
  return hipGetLastError();
}

// The same product restricted to output columns [n0, ...) (in units of
// output columns; for the gate/up epilogue, of gate columns).
template <bool TA, bool TB, int EPI>
GemmArgs column_part(const GemmArgs& g, int64_t n0) {
  GemmArgs t = g;
  if (EPI == 1) {
    t.pair_off = g.pair_off > 0 ? g.pair_off : g.F;
    t.B = g.B + n0 * g.ldb;        // gate rows n0..; up rows stay pair_off further
    t.F = g.F - n0;
    t.N = 2 * t.F;
    t.C = g.C + n0;
    t.X1 = g.X1 + n0;
  } else {
    t.B = TB ? g.B + n0 * g.ldb : g.B + n0;
    t.N = g.N - n0;
    t.C = g.C + n0;
    t.R = g.R + n0;
    if (g.bias) t.bias = g.bias + n0;
    if (EPI == 2) {
      t.pair_off = g.pair_off > 0 ? g.pair_off : g.F;
      t.X1 = g.X1 + n0;
    }
  }
  return t;
}

// ... restricted to output rows [m0, ...).
template <bool TA, bool TB, int EPI>
GemmArgs row_part(const GemmArgs& g, int64_t m0) {
  GemmArgs t = g;
  t.A = TA ? g.A + m0 : g.A + m0 * g.lda;
  t.M = g.M - m0;
  t.C = g.C + m0 * g.ldc;
  t.R = g.R + m0 * g.ldr;
  if (EPI != 0) t.X1 = g.X1 + m0 * g.ldx1;
  return t;
}

// C = alpha * sum_s W[s] + beta * R + bias over an Mt x Nt region, the
// splits summed in ascending order; eight columns per thread (Nt % 8 == 0).
__global__ void __launch_bounds__(256)
splitk_reduce_kernel(const float* __restrict__ W, int S, int64_t Mt, int64_t Nt, float alpha,
                     float beta, const lt_half* R, int64_t ldr, const lt_half* __restrict__ bias,
                     lt_half* C, int64_t ldc) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t n8 = Nt / 8;
  if (idx >= Mt * n8) return;
  const int64_t m = idx / n8, n = (idx % n8) * 8;
  float v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = 0.f;
  for (int sp = 0; sp < S; ++sp) {
    const float* w = W + ((int64_t)sp * Mt + m) * Nt + n;
    const float4 a = *reinterpret_cast<const float4*>(w);
    const float4 b = *reinterpret_cast<const float4*>(w + 4);
    v[0] += a.x; v[1] += a.y; v[2] += a.z; v[3] += a.w;
    v[4] += b.x; v[5] += b.y; v[6] += b.z; v[7] += b.w;
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] *= alpha;
  if (beta != 0.f) {
    const half8 r = as_half8(ld16(R + m * ldr + n));
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] += beta * (float)r[e];
  }
  if (bias) {
    const half8 bb = as_half8(ld16(bias + n));
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] += (float)bb[e];
  }
  half8 o;
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = (_Float16)v[e];
  *reinterpret_cast<half8*>(C + m * ldc + n) = o;
}

template <bool TA, bool TB, int EPI>
hipError_t dispatch_tile(const GemmArgs& g, hipStream_t s) {
  // 256x256 tiles once there are about as many tiles as CUs; smaller
  // problems use 128x128 tiles so that more workgroups exist.
  const int64_t unit_n = EPI == 1 ? 128 : 256;            // output columns per 256-wide tile
  const int64_t ncols = EPI == 1 ? g.F : g.N;
  const int64_t tm = (g.M + 255) / 256, tn = (ncols + unit_n - 1) / unit_n;
  const int64_t big_tiles = tm * tn;
  // A last wave at most half full runs as half-size tiles in one short round:
  // whole waves of 256x256 tiles first, then the remaining columns (or rows)
  // as 256x128 (or 128x256) tiles.
  constexpr int64_t kCUs = 256;
  const int64_t waves = big_tiles / kCUs, rem = big_tiles % kCUs;
  SplitTail st;
  if constexpr (EPI == 0) {
    // K not a multiple of 8 (no layer shape): one launch of the tiles with
    // the last slice's fix-up (256x256 from about one wave of them)
    if (g.K & 7) {
      if (big_tiles >= 192) return launch<256, 256, 2, 4, 64, 2, TA, TB, 0, true>(g, s);
      return launch<128, 128, 2, 2, 64, 2, TA, TB, 0, true>(g, s);
    }
    if (g.ws != nullptr && gemm_splitk_tail(g.M, g.N, g.K, &st) &&
        gemm_splitk_ws_bytes(g.M, g.N, g.K) <= g.ws_bytes) {
      // The last wave (or a launch of less than one wave) as split-K 256x256
      // tiles: whole waves first (full K), then the remaining tiles' K split
      // S ways (FP32 partials in the workspace), then the fixed-order sum
      // with alpha, beta * R and bias.
      GemmArgs head = g, tail;
      if (st.columns) {
        head.N = st.split_at;
        tail = column_part<TA, TB, 0>(g, st.split_at);
      } else {
        head.M = st.split_at;
        tail = row_part<TA, TB, 0>(g, st.split_at);
      }
      hipError_t e = hipSuccess;
      if (st.split_at > 0) e = launch<256, 256, 2, 4, 64, 2, TA, TB, 0>(head, s);
      if (e != hipSuccess) return e;
      GemmArgs part = tail;
      part.C = reinterpret_cast<lt_half*>(g.ws);
      part.ldc = st.Nt;
      part.beta = 0.f;
      part.bias = nullptr;
      e = launch<256, 256, 2, 4, 64, 2, TA, TB, 3>(part, s, st.S);
      if (e != hipSuccess) return e;
      const int64_t threads = st.Mt * (st.Nt / 8);
      hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0,
                         s, g.ws, st.S, st.Mt, st.Nt, g.alpha, g.beta, tail.R, tail.ldr, tail.bias,
                         tail.C, tail.ldc);
      return hipGetLastError();
    }
  }
  if (big_tiles < 192) return launch<128, 128, 2, 2, 64, 2, TA, TB, EPI>(g, s);
  if (waves >= 1 && rem > 0 && 2 * rem <= kCUs) {
    const int64_t full = waves * kCUs;
    if (full % tm == 0 && full / tm < tn) {
      const int64_t n_main = (full / tm) * unit_n;
      GemmArgs head = g;
      if (EPI == 1) {
        head.pair_off = g.pair_off > 0 ? g.pair_off : g.F;
        head.F = n_main;
        head.N = 2 * n_main;
      } else {
        head.N = n_main;
      }
      hipError_t e = launch<256, 256, 2, 4, 64, 2, TA, TB, EPI>(head, s);
      if (e != hipSuccess) return e;
      return launch<256, 128, 4, 2, 64, 2, TA, TB, EPI>(column_part<TA, TB, EPI>(g, n_main), s);
    }
    if (full % tn == 0 && full / tn < tm) {
      const int64_t m_main = (full / tn) * 256;
      GemmArgs head = g;
      head.M = m_main;
      hipError_t e = launch<256, 256, 2, 4, 64, 2, TA, TB, EPI>(head, s);
      if (e != hipSuccess) return e;
      return launch<128, 256, 2, 4, 64, 2, TA, TB, EPI>(row_part<TA, TB, EPI>(g, m_main), s);
    }
  }
  return launch<256, 256, 2, 4, 64, 2, TA, TB, EPI>(g, s);
}

}  // namespace

hipError_t gemm_f16_launch(const GemmArgs& g, hipStream_t s) {
  if (g.epi == 1) return dispatch_tile<false, true, 1>(g, s);     // X Wgu^T
  if (g.epi == 2) return dispatch_tile<false, false, 2>(g, s);    // dY Wd
  if (g.transA) {
    return g.transB ? dispatch_tile<true, true, 0>(g, s) : dispatch_tile<true, false, 0>(g, s);
  }
  return g.transB ? dispatch_tile<false, true, 0>(g, s) : dispatch_tile<false, false, 0>(g, s);
}

}  // namespace lt
