// Causal MHA / GQA attention backward (recomputed P), gfx950.
//
// Sec. 4.1 / Algorithm 1 of the paper: per key/value tile j and query tile i
//   GP = GO V^T,  GS = SoftmaxBackward(P, GP),  GV_j += P^T GO,
//   GQ_i += GS K,  GK_j += GS^T Q,
// with the partial GV / GK of the processing units reduced before write-back.
// Here P is rebuilt from the forward's row LSE, P = exp(scale q.k - LSE), and
// SoftmaxBackward is GS = P * (GP - D) with D_i = rowsum(GO_i * O_i).
//
// Three kernels (four with workspace shares), none with an atomic:
//   1. attn_bwd_rowterms: D_i = rowsum(dO_i * O_i) and the LSE in base 2 per
//                     query, for the dK/dV pass.  HBM-bound.
//   2. attn_bwd_dkdv: key-major.  One workgroup per (batch, kv head, 256-key
//                     tile); each of the 8 waves owns 32 keys and keeps their
//                     K fragments and the dK, dV accumulators in registers for
//                     the whole loop over the GQA group's query heads and the
//                     causal 64-query blocks (the paper's GSM reduction of
//                     GV / GK becomes register accumulation, and the GQA sum
//                     is the same loop).  V stays in LDS; Q, dO, LSE and D
//                     blocks stream HBM -> LDS by direct loads, double-buffered.
//                     S = Q K^T and dP = dO V^T put one key per lane, so P and
//                     dS feed the dV / dK MFMAs from registers; their Q^T /
//                     dO^T operands come from the same row-layout tiles through
//                     the LDS transpose read, in the accumulators' query order.
//                     Each wave also stores its FP16 dS, exactly as its
//                     registers hold it (one coalesced 2 KiB block per 32 keys
//                     x 32 queries), for the dQ pass.
//                     When 256-key tiles give too few workgroups (short
//                     sequences, few kv heads) the tiles hold 128 keys: waves
//                     w and w + 4 own the same keys, take the two 32-query
//                     halves of each block, and add their accumulators
//                     through LDS at the end.  Still too few: each key tile's
//                     (query head, query block) work is split over several
//                     workgroups, whose FP32 partial dK, dV go to the
//                     workspace and are summed in a fixed order by
//                     attn_bwd_dkdv_sum.
//   3. attn_bwd_dq  : GQ = GS K from the stored dS, query-major: one workgroup
//                     per (batch, head, 256 queries), each wave one 32-query
//                     group, streaming K slices (shared, LDS) and its own dS
//                     blocks (LDS, read transposed) by direct loads, two
//                     slices ahead of the one in use.  dQ is
//                     written once, in FP16.  One contraction, HBM-bound on
//                     the dS read.
// The pair (S, dP) is computed once per causal tile pair (five contractions
// with the recomputed S); the dS round trip through HBM replaces both the
// second S / dP recompute of a query-major dQ pass and dQ atomics.

#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "attn_tiles.hpp"

namespace lt {
namespace {

// Direct load of 16 bytes per lane into LDS, as lds_dma16_opaque, for data
// read once (non-temporal: the line is not kept in the caches for reuse, so
// it does not evict the operands that are).
__device__ __forceinline__ void lds_dma16_stream(const void* base, uint32_t nrec, void* lds,
                                                 uint32_t voff) {
  const uint64_t b = (uint64_t)base;
  u32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((uint32_t)b);
  r[1] = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32) & 0xffffu);
  r[2] = __builtin_amdgcn_readfirstlane(nrec);
  r[3] = 0x00020000u;
  const uint32_t m0v = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen nt lds"
               :
               : "s"(m0v), "v"(voff), "s"(r)
               : "memory");
}

constexpr int NWA = 8;         // dK/dV: waves per workgroup
constexpr int BKV = NWA * 32;  // dK/dV: keys per workgroup (32 per wave)
constexpr int BQA = 64;        // dK/dV: queries per block (two 32-query halves)
constexpr int NW = 8;          // recomputing dQ: waves per workgroup
constexpr int BQB = NW * 32;   // recomputing dQ: queries per workgroup (32 per wave)
constexpr int BKB = 128;       // recomputing dQ: keys per slice
constexpr int64_t kDqFillWgs = 512;   // recomputing dQ: 256-query workgroups needed to skip the split
constexpr float kLog2e = 1.4426950408889634f;

// ------------------------------------------------------------ kernel 0: saved P
// P = exp(scale q.k - LSE) of every (32-key group, 32-query group) block the
// mask keeps, written after the forward for the saved-P backward (Algorithm 1
// loads the forward's probability tiles instead of recomputing them).  Same
// lane layout and block order as the dS blocks, so the dK/dV pass loads each
// lane's P straight into registers.  Masked entries (key after query, key or
// query past S) are exactly 0.  One workgroup per (batch, query head,
// 256-key tile): 8 waves of 32 keys (K fragments in registers); 64-query Q
// blocks and their LSE rows stream through LDS by direct loads,
// double-buffered.
template <int D>
struct SavePSmem {
  using RT = RowTile<D, NWA>;
  static constexpr int TQ = BQA * RT::ROWB;
  static constexpr int ROW_OFF = 2 * TQ;             // LSE rows: 2 buffers x 256 B
  static constexpr int BYTES = ROW_OFF + 2 * 256;
};

template <int D>
__global__ void __launch_bounds__(NWA * 64, 2)
attn_save_p_kernel(const lt_half* __restrict__ Q, const lt_half* __restrict__ K, int64_t q_stride,
                   int64_t kv_stride, const float* __restrict__ LSE, lt_half* __restrict__ P,
                   int64_t nblk, int B, int S, int Hq, int Hkv, float scale, int causal) {
  using SM = SavePSmem<D>;
  using RT = RowTile<D, NWA>;
  constexpr int KK = D / 16;
  __shared__ __attribute__((aligned(1024))) char smem[SM::BYTES];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lrow = lane & 31;
  const int g = lane >> 5;
  const int jt = blockIdx.x / (B * Hq);            // ascending key tile = descending work
  int b, h;
  query_head(blockIdx.x % (B * Hq), B, Hq, Hkv, b, h);
  const int bh = b * Hq + h;
  const int kvh = h / (Hq / Hkv);
  const int kbase = jt * BKV;
  const int kw0 = kbase + wave * 32;
  const int mykey = kw0 + lrow;

  const lt_half* Kp = K + (int64_t)b * S * kv_stride + (int64_t)kvh * D;
  half8 kf[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk)
    kf[kk] = mykey < S ? as_half8(ld16(Kp + (int64_t)mykey * kv_stride + kk * 16 + g * 8))
                       : as_half8(u32x4{0, 0, 0, 0});

  const float c = scale * kLog2e;
  const int n_qb = (S + BQA - 1) / BQA;
  const int qb0 = causal ? kbase / BQA : 0;
  const int n_iter = n_qb - qb0;
  char* ph = reinterpret_cast<char*>(P) + (int64_t)bh * nblk * kDsBlockBytes + lane * 32;

  // Q rows and LSE entries past S read as zero (those queries are masked)
  // query blocks last to first (the key tiles of a head move in step, L2 reuse)
  auto stage = [&](int it, int buf) {
    const int qbase = (n_qb - 1 - it) * BQA;
    RT::template dma<BQA>(smem + buf * SM::TQ,
                          Q + ((int64_t)b * S + qbase) * q_stride + (int64_t)h * D, q_stride,
                          S - qbase, wave, lane);
    if (wave == 0) {
      const int nv = S - qbase < BQA ? S - qbase : BQA;
      lds_dma4_opaque(LSE + (int64_t)bh * S + qbase, (uint32_t)(nv * 4),
                      smem + SM::ROW_OFF + buf * 256, (uint32_t)(lane * 4));
    }
  };

  if (n_iter > 0) stage(0, 0);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) loaded_here(kf[kk]);

  for (int it = 0; it < n_iter; ++it) {
    const int cur = it & 1;
    const int qbase = (n_qb - 1 - it) * BQA;
    if (it + 1 < n_iter) stage(it + 1, cur ^ 1);
    const char* qs = smem + cur * SM::TQ;
    const float* lse_s = reinterpret_cast<const float*>(smem + SM::ROW_OFF + cur * 256);
#pragma unroll
    for (int hq = 0; hq < 2; ++hq) {
      const int qh = qbase + hq * 32;
      if ((!causal || kw0 <= qh + 31) && kw0 < S && qh < S) {   // wave-uniform
        //   S = Q K^T (lane owns key `mykey`, 16 query rows), P = exp2(s*scale*log2e - LSE*log2e)
        f32x16 sacc;
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[r] = 0.f;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) sacc = mfma32(RT::row_frag(qs, hq * 32, kk, lane), kf[kk], sacc);
        float p[16];
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
          const float4 l4 = *reinterpret_cast<const float4*>(lse_s + hq * 32 + 8 * rq + 4 * g);
          const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int r = 4 * rq + e;
            const int q = qh + 8 * rq + 4 * g + e;
            const float v = fast_exp2(fmaf(sacc[r], c, -lv[e] * kLog2e));
            p[r] = ((causal && q < mykey) || mykey >= S || q >= S) ? 0.f : v;
          }
        }
        const int qg = qh >> 5;
        const int kgi = kw0 >> 5;
        const int64_t blk = causal ? (int64_t)qg * (qg + 1) / 2 + kgi
                                   : (int64_t)qg * ((S + 31) >> 5) + kgi;
        char* dst = ph + blk * kDsBlockBytes;
        st16(dst, as_u32x4(pack8(p[0], p[1], p[2], p[3], p[4], p[5], p[6], p[7])));
        st16(dst + 16, as_u32x4(pack8(p[8], p[9], p[10], p[11], p[12], p[13], p[14], p[15])));
      }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  }
}

// ------------------------------------------------------------ kernel 2: dK/dV
template <int D>
struct DkdvSmem {
  using RT = RowTile<D, NWA>;
  static constexpr int TQ = BQA * RT::ROWB;             // one Q or dO block
  // Q and dO buffers first: every fragment read of them is a per-lane
  // register plus a constant below 64 KiB (the LDS instructions' offset field)
  static constexpr int Q_OFF = 0;                        // 2 buffers
  static constexpr int DO_OFF = Q_OFF + 2 * TQ;          // 2 buffers
  // base-2 LSE and D rows: 2 buffers x {LSE2, D} x 256 B (one 4-byte direct
  // load of 64 lanes each)
  static_assert(BQA == 64, "one 4-byte direct load per row vector");
  static constexpr int ROW_OFF = DO_OFF + 2 * TQ;
  static constexpr int V_OFF = ROW_OFF + 4 * 256;        // V tile [BKV][D]
  static_assert(DO_OFF + 2 * TQ <= 65536, "Q / dO offsets fit the offset field");
  static constexpr int BYTES = V_OFF + BKV * RT::ROWB;
};

// KSPLIT = 1: 8 key groups of 32 (256 keys), every wave walks both 32-query
// halves of each block.  KSPLIT = 2 (few workgroups): 4 key groups (128
// keys); waves w and w + 4 own the same keys, take one half each, and their
// FP32 accumulators are summed through LDS at the end (fixed order).
// SP (saved P): P is read from the forward's saved blocks (same layout as
// the dS blocks, written by attn_save_p) instead of recomputed, so there are
// no K fragments, no S products and no exponentials; V fragments are held in
// registers; no dS is stored (the dQ pass recomputes).
template <int D, int KSPLIT, bool SP>
__global__ void __launch_bounds__(NWA * 64, 1)
attn_bwd_dkdv_kernel(const lt_half* __restrict__ Q, const lt_half* __restrict__ K,
                     const lt_half* __restrict__ V, int64_t q_stride, int64_t kv_stride,
                     const lt_half* __restrict__ dO, int64_t o_stride, const float* __restrict__ lse2,
                     const float* __restrict__ delta, lt_half* __restrict__ dK,
                     lt_half* __restrict__ dV, int64_t dkv_stride, lt_half* __restrict__ ds_out,
                     const lt_half* __restrict__ psaved, int64_t nblk, float* __restrict__ part,
                     int nsplit, int B, int S, int Hq, int Hkv, float scale, int causal) {
  using SM = DkdvSmem<D>;
  using RT = RowTile<D, NWA>;
  constexpr int KK = D / 16;       // MFMA steps over the head dim
  constexpr int DB = D / 32;       // 32-feature blocks
  constexpr int NKG = NWA / KSPLIT;                // key groups of 32
  constexpr int BK = NKG * 32;                     // keys per workgroup
  static_assert(KSPLIT == 1 || KSPLIT == BQA / 32, "one 32-query half per wave of a pair");
  static_assert(KSPLIT == 1 || NKG * 2 * DB * 4 * 64 * 16 <= SM::BYTES, "reduction fits in LDS");
  __shared__ __attribute__((aligned(1024))) char smem[SM::BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar addressing
  const int lrow = lane & 31;
  const int g = lane >> 5;
  const int kg = wave % NKG;                       // key group
  const int kpart = wave / NKG;                    // query half taken (KSPLIT = 2)

  const int bkv = blockIdx.x % (B * Hkv);
  const int sp = (blockIdx.x / (B * Hkv)) % nsplit;   // which share of the query blocks
  const int jt = blockIdx.x / (B * Hkv * nsplit);     // ascending key tile = descending work
  const int b = bkv / Hkv;
  const int kvh = bkv % Hkv;
  const int G = Hq / Hkv;                             // query heads of the kv head
  const int h0 = kvh * G;
  const int kbase = jt * BK;
  const int kw0 = kbase + kg * 32;                 // this wave's first key
  const int mykey = kw0 + lrow;                    // key owned by this lane (S, dP columns)

  const lt_half* Kp = K + (int64_t)b * S * kv_stride + (int64_t)kvh * D;
  const lt_half* Vp = V + (int64_t)b * S * kv_stride + (int64_t)kvh * D;

  // ---- V tile -> LDS (B operand of dP = dO V^T); rows past S read as zero ----
  if constexpr (!SP)
    RT::template dma<BK>(smem + SM::V_OFF, Vp + (int64_t)kbase * kv_stride, kv_stride, S - kbase,
                         wave, lane);
  // ---- K fragments (B operand of S = Q K^T), or with saved P the V
  // fragments (B operand of dP = dO V^T) in registers instead of LDS ----
  half8 kf[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk)
    kf[kk] = mykey < S ? as_half8(ld16((SP ? Vp : Kp) + (int64_t)mykey * kv_stride + kk * 16 + g * 8))
                       : as_half8(u32x4{0, 0, 0, 0});

  // lane part of the row-fragment address of step kk (rows rb + lane % 32,
  // rb a multiple of 16, so the swizzle depends on the lane only)
  uint32_t rlane[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) rlane[kk] = (uint32_t)RT::addr(lane & 31, kk * 2 + (lane >> 5));
  const uint32_t vrow0 = __builtin_amdgcn_readfirstlane(SM::V_OFF + kg * 32 * RT::ROWB);

  f32x16 dkacc[DB], dvacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      dkacc[db][r] = 0.f;
      dvacc[db][r] = 0.f;
    }

  const float c = scale * kLog2e;
  const int n_qb = (S + BQA - 1) / BQA;
  const int qb0 = causal ? kbase / BQA : 0;
  const int per_head = n_qb - qb0;
  // The group's (query head, query block) pairs, head-major, are split into
  // nsplit contiguous shares; this workgroup takes share sp (possibly empty:
  // its partial sums are then zero).
  const int total = G * per_head;
  const int it0 = (int)((int64_t)sp * total / nsplit);
  const int n_iter = (int)((int64_t)(sp + 1) * total / nsplit) - it0;

  // Block `it` = (query head, 64 queries).  Q, dO (rows past S read as zero)
  // and the base-2 LSE and D entries (zero past S: with zero Q and dO rows
  // those queries contribute nothing) go to LDS by direct loads.
  // Within a head the query blocks run last to first: the key tiles of one
  // kv head (resident on one XCD, which the workgroup order gives them) then
  // start on the same block and move in step, so each Q / dO block comes from
  // memory once and from that XCD's L2 for the other tiles.
  auto block_of = [&](int i, int& h, int& qbase) {
    const int it = it0 + i;
    h = h0 + it / per_head;
    qbase = (n_qb - 1 - it % per_head) * BQA;
  };
  auto stage = [&](int it, int buf) {
    int h, qbase;
    block_of(it, h, qbase);
    RT::template dma<BQA>(smem + SM::Q_OFF + buf * SM::TQ,
                          Q + ((int64_t)b * S + qbase) * q_stride + (int64_t)h * D, q_stride,
                          S - qbase, wave, lane);
    RT::template dma<BQA>(smem + SM::DO_OFF + buf * SM::TQ,
                          dO + ((int64_t)b * S + qbase) * o_stride + (int64_t)h * D, o_stride,
                          S - qbase, wave, lane);
    if (wave < 2) {
      const float* rowp = (wave == 0 ? lse2 : delta) + ((int64_t)b * Hq + h) * S + qbase;
      const int nv = S - qbase < BQA ? S - qbase : BQA;
      lds_dma4_opaque(rowp, (uint32_t)(nv * 4), smem + SM::ROW_OFF + buf * 512 + wave * 256,
                      (uint32_t)(lane * 4));
    }
  };

  // Saved P: the P blocks of a block iteration's halves, loaded one
  // iteration ahead straight into registers (the lane layout the blocks
  // were written in); halves past S or wholly masked read as zero.
  constexpr int NH = BQA / 32 / KSPLIT;            // 32-query halves per wave and block
  half8 pcur[NH][2], pnxt[NH][2];
  auto load_p = [&](int it, half8 (&dst)[NH][2]) {
    int h, qbase;
    block_of(it, h, qbase);
#pragma unroll
    for (int ih = 0; ih < NH; ++ih) {
      const int hq = KSPLIT > 1 ? kpart : ih;
      const int qh = qbase + hq * 32;
      if ((!causal || kw0 <= qh + 31) && kw0 < S && qh < S) {
        const int qg = qh >> 5;
        const int kgi = kw0 >> 5;
        const int64_t blk = causal ? (int64_t)qg * (qg + 1) / 2 + kgi
                                   : (int64_t)qg * ((S + 31) >> 5) + kgi;
        const char* src = reinterpret_cast<const char*>(psaved) +
                          (((int64_t)b * Hq + h) * nblk + blk) * kDsBlockBytes + lane * 32;
        dst[ih][0] = as_half8(ld16(src));
        dst[ih][1] = as_half8(ld16(src + 16));
      } else {
        dst[ih][0] = as_half8(u32x4{0, 0, 0, 0});
        dst[ih][1] = as_half8(u32x4{0, 0, 0, 0});
      }
    }
  };

  if (n_iter > 0) stage(0, 0);
  if constexpr (SP) {
    if (n_iter > 0) load_p(0, pcur);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) loaded_here(kf[kk]);
  if constexpr (SP) {
#pragma unroll
    for (int ih = 0; ih < NH; ++ih) {
      loaded_here(pcur[ih][0]);
      loaded_here(pcur[ih][1]);
    }
  }

  // two block iterations per trip, so that the buffer index is a constant
  auto iteration = [&](int it, auto CUR_) {
    const int cur = CUR_;   // a constant in the unrolled main path
    int h, qbase;
    block_of(it, h, qbase);
    // that buffer was last read before the previous barrier
    if (it + 1 < n_iter) stage(it + 1, cur ^ 1);
    if constexpr (SP) {
      if (it + 1 < n_iter) load_p(it + 1, pnxt);
    }
    const char* qs = smem + SM::Q_OFF + cur * SM::TQ;
    const char* dos = smem + SM::DO_OFF + cur * SM::TQ;
    const float* lse_s = reinterpret_cast<const float*>(smem + SM::ROW_OFF + cur * 512);
    const float* del_s = reinterpret_cast<const float*>(smem + SM::ROW_OFF + cur * 512 + 256);

    auto half = [&](int ih) {
      const int hq = KSPLIT > 1 ? kpart : ih;
      // 32-query half hq of the block; causal: all of this wave's keys after
      // all of its queries -> P = 0
      const int qh = qbase + hq * 32;
      const bool active = (!causal || kw0 <= qh + 31) && kw0 < S;
      if (SP && active) {
        //   dP = dO V^T   (lane owns key `mykey`, 16 query rows; V fragments in registers)
        //   dS = P (dP - D) with the saved P,  dV^T += dO^T P,  dK^T += Q^T dS
        f32x16 pacc;
#pragma unroll
        for (int r = 0; r < 16; ++r) pacc[r] = 0.f;
        half8 fd = RT::row_frag(dos, hq * 32, 0, lane);
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
          half8 nd = fd;
          if (kk + 1 < KK) nd = RT::row_frag(dos, hq * 32, kk + 1, lane);
          pacc = mfma32(fd, kf[kk], pacc);
          fd = nd;
        }
        __builtin_amdgcn_s_setprio(0);
        const half8* pp = pcur[0];   // this half's P (the halves are shifted down below)
        float ds[16];
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
          const float4 d4 = *reinterpret_cast<const float4*>(del_s + hq * 32 + 8 * rq + 4 * g);
          const float dv[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int r = 4 * rq + e;
            ds[r] = (float)pp[r >> 3][r & 7] * (pacc[r] - dv[e]);
          }
        }
        half8 pds[2];
#pragma unroll
        for (int kc = 0; kc < 2; ++kc)
          pds[kc] = pack8(ds[8 * kc], ds[8 * kc + 1], ds[8 * kc + 2], ds[8 * kc + 3],
                          ds[8 * kc + 4], ds[8 * kc + 5], ds[8 * kc + 6], ds[8 * kc + 7]);
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int kc = 0; kc < 2; ++kc)
#pragma unroll
          for (int db = 0; db < DB; ++db) {
            dvacc[db] = mfma32(RT::template tr_frag<true>(dos, hq * 32 + kc * 16, db * 32, lane),
                               pp[kc], dvacc[db]);
            dkacc[db] = mfma32(RT::template tr_frag<true>(qs, hq * 32 + kc * 16, db * 32, lane),
                               pds[kc], dkacc[db]);
          }
        __builtin_amdgcn_s_setprio(0);
      }
      if constexpr (SP && NH > 1) {   // next half's P into pcur[0] (constant register indices)
#pragma unroll
        for (int j = 0; j + 1 < NH; ++j) {
          pcur[j][0] = pcur[j + 1][0];
          pcur[j][1] = pcur[j + 1][1];
        }
      }
      if (!SP && active) {
        //   S = Q K^T, dP = dO V^T   (lane owns key `mykey`, 16 query rows)
        //   P = exp2(s*scale*log2e - LSE2), dS = P (dP - D)
        //   dV^T += dO^T P,  dK^T += Q^T dS
        f32x16 sacc, pacc;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          sacc[r] = 0.f;
          pacc[r] = 0.f;
        }
        // fragments of step kk+1 are read before the MFMAs of step kk; the Q
        // and dO reads are a lane register plus a constant, the V read's address
        // is added right before it (kept there: holding eight V addresses
        // through the loop does not fit the register budget)
        auto rdq = [&](int kk) {
          return as_half8(*reinterpret_cast<const u32x4*>(smem + SM::Q_OFF + cur * SM::TQ +
                                                          hq * 32 * RT::ROWB + rlane[kk]));
        };
        auto rdo = [&](int kk) {
          return as_half8(*reinterpret_cast<const u32x4*>(smem + SM::DO_OFF + cur * SM::TQ +
                                                          hq * 32 * RT::ROWB + rlane[kk]));
        };
        auto rdv = [&](int kk) {
          uint32_t a;
          asm volatile("v_add_u32 %0, %1, %2" : "=v"(a) : "v"(rlane[kk]), "s"(vrow0));
          return as_half8(*reinterpret_cast<const u32x4*>(smem + a));
        };
        half8 fq = rdq(0);
        half8 fd = rdo(0);
        half8 fv = rdv(0);
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
          half8 nq = fq, nd = fd, nv = fv;
          if (kk + 1 < KK) {
            nq = rdq(kk + 1);
            nd = rdo(kk + 1);
            nv = rdv(kk + 1);
          }
          sacc = mfma32(fq, kf[kk], sacc);
          pacc = mfma32(fd, fv, pacc);
          if (kk + 1 < KK) {
            __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);   // the three reads
            __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);   // then the two MFMAs
          }
          fq = nq;
          fd = nd;
          fv = nv;
        }

        __builtin_amdgcn_s_setprio(0);
        float p[16], ds[16];
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
          const int ql0 = hq * 32 + 8 * rq + 4 * g;
          const float4 l4 = *reinterpret_cast<const float4*>(lse_s + ql0);
          const float4 d4 = *reinterpret_cast<const float4*>(del_s + ql0);
          const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
          const float dv[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int r = 4 * rq + e;
            p[r] = fast_exp2(fmaf(sacc[r], c, -lv[e]));
            ds[r] = pacc[r] - dv[e];
          }
        }
        if ((causal && kw0 + 31 > qh) || kw0 + 32 > S) {   // wave-uniform
          // key > query (causal) or key past S -> P = 0
          const int qlim = causal ? mykey : 0;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int q = qh + 8 * (r >> 2) + 4 * g + (r & 3);
            p[r] = ((q < qlim) | (mykey >= S)) ? 0.f : p[r];
          }
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) ds[r] *= p[r];
        half8 pp[2], pds[2];
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
          pp[kc] = pack8(p[8 * kc], p[8 * kc + 1], p[8 * kc + 2], p[8 * kc + 3], p[8 * kc + 4],
                         p[8 * kc + 5], p[8 * kc + 6], p[8 * kc + 7]);
          pds[kc] = pack8(ds[8 * kc], ds[8 * kc + 1], ds[8 * kc + 2], ds[8 * kc + 3],
                          ds[8 * kc + 4], ds[8 * kc + 5], ds[8 * kc + 6], ds[8 * kc + 7]);
        }
        // dS block (query group qh / 32, key group kw0 / 32) for the dQ pass, as
        // held here (lane-major, 32 bytes per lane).  The padded second half of
        // a last query block lies past the sequence and is not stored.
        if (qh < S) {
          const int qg = qh >> 5;
          const int kgi = kw0 >> 5;
          const int64_t blk = causal ? (int64_t)qg * (qg + 1) / 2 + kgi
                                     : (int64_t)qg * ((S + 31) >> 5) + kgi;
          char* dst = reinterpret_cast<char*>(ds_out) +
                      (((int64_t)b * Hq + h) * nblk + blk) * kDsBlockBytes + lane * 32;
          // written once, read once by the dQ pass: non-temporal, so that the
          // 2 KiB blocks (0.5 GB per call at S = 4096) do not evict the Q / dO
          // blocks and K / V tiles the key tiles share through L2
          __builtin_nontemporal_store(as_u32x4(pds[0]), reinterpret_cast<u32x4*>(dst));
          __builtin_nontemporal_store(as_u32x4(pds[1]), reinterpret_cast<u32x4*>(dst + 16));
        }
        __builtin_amdgcn_s_setprio(1);
        // steps (kc, db): the transposed dO and Q fragments of step s + 1 are
        // read before step s's two MFMAs, into the other of two register sets
        constexpr int NST = 2 * DB;
        half8 tdo[2], tq[2];
        auto rd_tr = [&](int st_, half8& a, half8& b) {
          const int kc = st_ / DB, db = st_ % DB;
          a = RT::template tr_frag<true>(dos, hq * 32 + kc * 16, db * 32, lane);
          b = RT::template tr_frag<true>(qs, hq * 32 + kc * 16, db * 32, lane);
        };
        rd_tr(0, tdo[0], tq[0]);
#pragma unroll
        for (int st_ = 0; st_ < NST; ++st_) {
          const int kc = st_ / DB, db = st_ % DB;
          if (st_ + 1 < NST) rd_tr(st_ + 1, tdo[(st_ + 1) & 1], tq[(st_ + 1) & 1]);
          dvacc[db] = mfma32(tdo[st_ & 1], pp[kc], dvacc[db]);
          dkacc[db] = mfma32(tq[st_ & 1], pds[kc], dkacc[db]);
          // the groups count from the top of the block: the first read group
          // holds steps 0 and 1 (two transposed reads per fragment)
          if (st_ + 1 < NST) {
            if (st_ == 0)
              __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
            else
              __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
          }
        }
        __builtin_amdgcn_s_setprio(0);
      }
    };
    if constexpr (KSPLIT == 1 && !SP) {
#pragma unroll
      for (int ih = 0; ih < BQA / 32; ++ih) half(ih);
    } else {
#pragma nounroll
      for (int ih = 0; ih < BQA / 32 / KSPLIT; ++ih) half(ih);
    }

    // next block resident for every wave; nobody reads this buffer any more
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if constexpr (SP) {
#pragma unroll
      for (int ih = 0; ih < NH; ++ih) {
        pcur[ih][0] = pnxt[ih][0];
        pcur[ih][1] = pnxt[ih][1];
      }
    }
  };
  if constexpr (KSPLIT == 1) {
    for (int it = 0; it < n_iter; it += 2) {
      iteration(it, std::integral_constant<int, 0>{});
      if (it + 1 < n_iter) iteration(it + 1, std::integral_constant<int, 1>{});
    }
  } else {
    for (int it = 0; it < n_iter; ++it) iteration(it, it & 1);
  }

  if constexpr (KSPLIT > 1) {
    // all of LDS is free after the loop's last barrier: the second wave of
    // each pair passes its dK, dV accumulators through it (lane-major float4,
    // conflict-free) to the first, which adds them
    float4* red = reinterpret_cast<float4*>(smem);
    auto slot = [&](int which, int db, int rq) { return ((kg * 2 + which) * DB + db) * 4 + rq; };
    if (kpart == 1) {
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
          red[slot(0, db, rq) * 64 + lane] =
              make_float4(dkacc[db][4 * rq], dkacc[db][4 * rq + 1], dkacc[db][4 * rq + 2],
                          dkacc[db][4 * rq + 3]);
          red[slot(1, db, rq) * 64 + lane] =
              make_float4(dvacc[db][4 * rq], dvacc[db][4 * rq + 1], dvacc[db][4 * rq + 2],
                          dvacc[db][4 * rq + 3]);
        }
    }
    __syncthreads();
    if (kpart != 0) return;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const float4 k = red[slot(0, db, rq) * 64 + lane];
        const float4 v = red[slot(1, db, rq) * 64 + lane];
        dkacc[db][4 * rq] += k.x;
        dkacc[db][4 * rq + 1] += k.y;
        dkacc[db][4 * rq + 2] += k.z;
        dkacc[db][4 * rq + 3] += k.w;
        dvacc[db][4 * rq] += v.x;
        dvacc[db][4 * rq + 1] += v.y;
        dvacc[db][4 * rq + 2] += v.z;
        dvacc[db][4 * rq + 3] += v.w;
      }
  }

  // ---- write dK = scale * acc, dV (or this split's FP32 partial sums) ----
  if (nsplit > 1) {
    if (mykey < S) {
      const int64_t rowsz = (int64_t)B * S * Hkv * D;
      float* pk = part + (int64_t)sp * rowsz + (((int64_t)b * S + mykey) * Hkv + kvh) * D;
      float* pv = pk + (int64_t)nsplit * rowsz;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
          const int d = db * 32 + 8 * rq + 4 * g;
          *reinterpret_cast<float4*>(pk + d) =
              make_float4(dkacc[db][4 * rq], dkacc[db][4 * rq + 1], dkacc[db][4 * rq + 2],
                          dkacc[db][4 * rq + 3]);
          *reinterpret_cast<float4*>(pv + d) =
              make_float4(dvacc[db][4 * rq], dvacc[db][4 * rq + 1], dvacc[db][4 * rq + 2],
                          dvacc[db][4 * rq + 3]);
        }
    }
  } else if (mykey < S) {
    lt_half* dkp = dK + ((int64_t)b * S + mykey) * dkv_stride + (int64_t)kvh * D;
    lt_half* dvp = dV + ((int64_t)b * S + mykey) * dkv_stride + (int64_t)kvh * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        half4 k4, v4;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          k4[e] = (_Float16)(dkacc[db][4 * rq + e] * scale);
          v4[e] = (_Float16)dvacc[db][4 * rq + e];
        }
        *reinterpret_cast<half4*>(dkp + db * 32 + 8 * rq + 4 * g) = k4;
        *reinterpret_cast<half4*>(dvp + db * 32 + 8 * rq + 4 * g) = v4;
      }
  }
}

// ------------------------------------------------------------ kernel 3: dQ from dS
constexpr int NWQ = 8;          // dQ: waves per workgroup, one 32-query group each
constexpr int BQQ = NWQ * 32;   // dQ: queries per workgroup
constexpr int BKQ = 64;         // dQ: keys per slice (two 32-key groups)
constexpr int NSQ = 3;          // dQ: LDS stages (two slices in flight while one is used)

template <int D>
struct DqSmem {
  using RT = RowTile<D, NWQ>;
  static constexpr int KT = BKQ * RT::ROWB;          // K slice [64][D]
  static constexpr int DSW = 2 * kDsBlockBytes;      // one wave's two dS blocks of a slice
  static constexpr int STAGE = KT + NWQ * DSW;
  static constexpr int BYTES = NSQ * STAGE;
  // direct loads per wave and stage: K rows, then always four 1 KiB dS loads
  // (blocks the mask drops load nothing: zero-length buffer), so that the
  // count behind each vmcnt wait is fixed
  static constexpr int LOADS = KT / 1024 / NWQ + 4;
};

// B operand dS^T of GQ^T = K^T dS^T from one dS block in LDS (lane-major,
// 32 bytes per lane of the dK/dV pass, see attn_bwd_ds_blocks): lane L gets
// stored query position L % 32 at keys kb + 8 (j / 4) + 4 (L / 32) + j % 4,
// j = 0..7 (the key order of RowTile::tr_frag<true>).  Each 16-lane group
// reads four consecutive 32-byte lanes; the two groups of one 32-lane read
// cycle are 1 KiB apart and share their banks (a two-way conflict).  The
// pass is bound by the dS stream: a 128-byte gap between the block halves,
// which removes the conflict, measured level.
__device__ __forceinline__ half8 ds_tr_frag(const char* blk, int kb, int lane) {
  v4s part[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int k = kb + 8 * h + 4 * (lane >> 5) + ((lane & 15) >> 2);
    part[h] = lds_read_tr16(blk + (k + 32 * ((lane >> 4) & 1)) * 32 + 8 * (lane & 3));
  }
  return as_half8(pack_v4s_pair(part[0], part[1]));
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

template <int D>
__global__ void __launch_bounds__(NWQ * 64, 1)
attn_bwd_dq_kernel(const lt_half* __restrict__ K, int64_t kv_stride, const lt_half* __restrict__ ds,
                   int64_t nblk, lt_half* __restrict__ dQ, int64_t dq_stride, int B, int S, int Hq,
                   int Hkv, float scale, int causal) {
  using SM = DqSmem<D>;
  using RT = RowTile<D, NWQ>;
  constexpr int DB = D / 32;
  static_assert(SM::BYTES <= 160 * 1024, "stages fit in LDS");
  __shared__ __attribute__((aligned(1024))) char smem[SM::BYTES];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n32 = (S + 31) / 32;
  const int n_qt = (S + BQQ - 1) / BQQ;
  const int qt = causal ? n_qt - 1 - (int)(blockIdx.x / (B * Hq)) : (int)(blockIdx.x / (B * Hq));
  int b, h;
  query_head(blockIdx.x % (B * Hq), B, Hq, Hkv, b, h);
  const int bh = b * Hq + h;
  const int kvh = h / (Hq / Hkv);
  const int qg = qt * NWQ + wave;                  // this wave's 32-query group
  // key groups this wave takes: 0 .. kg_end - 1 (those the mask keeps)
  const int kg_end = qg >= n32 ? 0 : (causal ? qg + 1 : n32);
  const int key_end = causal ? min(S, (qt + 1) * BQQ) : S;   // keys any wave needs
  const int n_ks = (key_end + BKQ - 1) / BKQ;

  const lt_half* Kp = K + (int64_t)b * S * kv_stride + (int64_t)kvh * D;
  // block (qg, 0); block (qg, kg) follows at kg * 2 KiB
  const char* dsq = reinterpret_cast<const char*>(ds) +
                    ((int64_t)bh * nblk + (causal ? (int64_t)qg * (qg + 1) / 2 : (int64_t)qg * n32)) *
                        kDsBlockBytes;

  f32x16 acc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[db][r] = 0.f;

  // slice ks -> stage ks % NSQ; K rows past S read as zero (their dS is zero)
  auto stage = [&](int ks) {
    char* st = smem + (ks % NSQ) * SM::STAGE;
    RT::template dma<BKQ>(st, Kp + (int64_t)ks * BKQ * kv_stride, kv_stride, S - ks * BKQ, wave,
                          lane);
    char* mine = st + SM::KT + wave * SM::DSW;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int kg = 2 * ks + c;
      const char* src = dsq + (int64_t)(kg < kg_end ? kg : 0) * kDsBlockBytes;
      const uint32_t nrec = kg < kg_end ? kDsBlockBytes : 0u;
      lds_dma16_stream(src, nrec, mine + c * kDsBlockBytes, (uint32_t)(lane * 16));
      lds_dma16_stream(src, nrec, mine + c * kDsBlockBytes + 1024, (uint32_t)(1024 + lane * 16));
    }
  };

  for (int ks = 0; ks < NSQ - 1 && ks < n_ks; ++ks) stage(ks);
  if (n_ks > 1) wait_vmcnt<SM::LOADS>(); else wait_vmcnt<0>();   // slice 0 resident
  __syncthreads();
  for (int ks = 0; ks < n_ks; ++ks) {
    // the stage of slice ks + 2 was last read before the previous barrier
    if (ks + NSQ - 1 < n_ks) stage(ks + NSQ - 1);
    const char* st = smem + (ks % NSQ) * SM::STAGE;
    const char* mine = st + SM::KT + wave * SM::DSW;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      if (2 * ks + c < kg_end) {
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
          //   dQ^T += K^T dS^T  (K^T read transposed, keys in accumulator order)
          const half8 bds = ds_tr_frag(mine + c * kDsBlockBytes, kc * 16, lane);
#pragma unroll
          for (int db = 0; db < DB; ++db)
            acc[db] = mfma32(RT::template tr_frag<true>(st, c * 32 + kc * 16, db * 32, lane), bds,
                             acc[db]);
        }
      }
    }
    // slice ks + 1 resident for every wave (slice ks + 2's loads may still be
    // in flight); nobody reads stage ks any more
    if (ks + NSQ - 1 < n_ks) wait_vmcnt<SM::LOADS>(); else wait_vmcnt<0>();
    __syncthreads();
  }

  // ---- dQ = scale * acc -> FP16; lane L holds stored query position L % 32 ----
  if (qg < n32) {
    const int pos = lane & 31;
    const int q = qg * 32 + 8 * ((pos & 15) >> 2) + 4 * (pos >> 4) + (pos & 3);
    const int g = lane >> 5;
    if (q < S) {
      lt_half* qp = dQ + ((int64_t)b * S + q) * dq_stride + (int64_t)h * D;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
          half4 o;
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = (_Float16)(acc[db][4 * rq + e] * scale);
          *reinterpret_cast<half4*>(qp + db * 32 + 8 * rq + 4 * g) = o;
        }
    }
  }
}

// ------------------------------------------------------------ saved P: dQ (and D)
// dQ with S and dP recomputed, query-major, for the saved-P backward (whose
// dK/dV pass stores no dS): D and the base-2 LSE are formed in its prologue and
// stored for the dK/dV pass, which runs second.
template <int D>
struct DqrSmem {
  using RT = RowTile<D, NW>;
  static constexpr int TILE = BKB * RT::ROWB;     // one K or V slice
  static constexpr int STAGE = 2 * TILE;          // K then V
};

// QSPLIT = 1: 8 query groups of 32 (256 queries), every wave walks every
// 32-key block.  QSPLIT = 2 (short sequences, for twice the workgroups): 4
// query groups (128 queries); waves w and w + 4 share a query group and take
// alternate 32-key blocks of each slice, and their FP32 accumulators are
// summed through LDS at the end (wave w + 4's into wave w's, fixed order).
template <int D, int QSPLIT>
__global__ void __launch_bounds__(NW * 64, 2)
attn_bwd_dq_recompute_kernel(const lt_half* __restrict__ Q, const lt_half* __restrict__ K,
                   const lt_half* __restrict__ V, int64_t q_stride, int64_t kv_stride,
                   const lt_half* __restrict__ O, const lt_half* __restrict__ dO, int64_t o_stride,
                   const float* __restrict__ LSE, float* __restrict__ lse2,
                   float* __restrict__ delta, lt_half* __restrict__ dQ, int64_t dq_stride,
                   int B, int S, int Hq, int Hkv, float scale, int causal) {
  using SM = DqrSmem<D>;
  using RT = RowTile<D, NW>;
  constexpr int KB = BKB / 32;     // 32-key blocks per slice
  constexpr int DB = D / 32;
  constexpr int KK = D / 16;
  constexpr int NQG = NW / QSPLIT;                 // query groups of 32
  constexpr int BQ = NQG * 32;                     // queries per workgroup
  static_assert(NW % QSPLIT == 0 && KB % QSPLIT == 0, "QSPLIT must divide waves and blocks");
  static_assert(QSPLIT == 1 || NQG * DB * 4 * 64 * 16 <= 2 * SM::STAGE, "reduction fits in LDS");
  __shared__ __attribute__((aligned(1024))) char smem[2 * SM::STAGE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar addressing
  const int lrow = lane & 31;
  const int g = lane >> 5;
  const int qg = wave % NQG;                       // query group
  const int kpart = wave / NQG;                    // which of the QSPLIT key-block shares

  const int n_qt = (S + BQ - 1) / BQ;
  const int qt = causal ? n_qt - 1 - (int)(blockIdx.x / (B * Hq)) : (int)(blockIdx.x / (B * Hq));
  int b, h;
  query_head(blockIdx.x % (B * Hq), B, Hq, Hkv, b, h);
  const int kvh = h / (Hq / Hkv);
  const int q0 = qt * BQ;
  const int qw0 = q0 + qg * 32;
  const int myq = qw0 + lrow;                      // query owned by this lane

  const lt_half* Kp = K + (int64_t)b * S * kv_stride + (int64_t)kvh * D;
  const lt_half* Vp = V + (int64_t)b * S * kv_stride + (int64_t)kvh * D;
  const float c = scale * kLog2e;

  // Q and dO fragments (B operands of S^T = K Q^T and dP^T = V dO^T):
  // column = this lane's query, reduction indices kk*16 + 8g + 0..7; the
  // same half-row of O for D.  Queries past S: zero Q, dO, O and LSE2 give
  // zero dS.
  half8 qf[KK], of[KK], oo[KK];
  float l2 = 0.f, dl = 0.f;
  const int64_t ri = ((int64_t)b * Hq + h) * S + myq;   // [B, Hq, S] row entry
  if (myq < S) {
    const lt_half* qp = Q + ((int64_t)b * S + myq) * q_stride + (int64_t)h * D + g * 8;
    const int64_t orow = ((int64_t)b * S + myq) * o_stride + (int64_t)h * D + g * 8;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      qf[kk] = as_half8(ld16(qp + kk * 16));
      of[kk] = as_half8(ld16(dO + orow + kk * 16));
      oo[kk] = as_half8(ld16(O + orow + kk * 16));
    }
    l2 = LSE[ri] * kLog2e;
  } else {
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      qf[kk] = as_half8(u32x4{0, 0, 0, 0});
      of[kk] = as_half8(u32x4{0, 0, 0, 0});
      oo[kk] = as_half8(u32x4{0, 0, 0, 0});
    }
  }

  f32x16 dqacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) dqacc[db][r] = 0.f;

  const int kv_end = causal ? min(S, q0 + BQ) : S;
  const int n_kv = (kv_end + BKB - 1) / BKB;
  const int q_hi = min(qw0 + 32, S) - 1;           // last valid query of this wave
  const int klim = causal ? min(myq + 1, S) : S;   // keys < klim are visible

  // K, V rows past S read as zero (masked below)
  auto stage_load = [&](int kt, int buf) {
    char* st = smem + buf * SM::STAGE;
    const int key0 = kt * BKB;
    RT::template dma<BKB>(st, Kp + (int64_t)key0 * kv_stride, kv_stride, S - key0, wave, lane);
    RT::template dma<BKB>(st + SM::TILE, Vp + (int64_t)key0 * kv_stride, kv_stride, S - key0,
                          wave, lane);
  };
  if (n_kv > 0) stage_load(0, 0);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    loaded_here(qf[kk]);
    loaded_here(of[kk]);
    loaded_here(oo[kk]);
  }
  loaded_here(l2);
  // D_i = rowsum(dO_i * O_i): this lane's half of the row, then its
  // partner's (lanes l and l ^ 32 own the same query).  The first wave of
  // each query group stores D and the base-2 LSE for the dK/dV kernel.
  {
    float part = 0.f;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
#pragma unroll
      for (int e = 0; e < 8; ++e) part = fmaf((float)of[kk][e], (float)oo[kk][e], part);
    dl = part + __shfl_xor(part, 32);
  }
  if (myq < S && g == 0 && kpart == 0) {
    delta[ri] = dl;
    lse2[ri] = l2;
  }

  for (int kt = 0; kt < n_kv; ++kt) {
    const char* ks = smem + (kt & 1) * SM::STAGE;
    const char* vs = ks + SM::TILE;
    // that stage was last read before the previous barrier
    if (kt + 1 < n_kv) stage_load(kt + 1, (kt + 1) & 1);

    const int key0 = kt * BKB;
    const bool active = (!causal || key0 <= q_hi) && qw0 < S;
    if (active) {
      const bool need_mask = (causal && key0 + BKB - 1 > qw0) || key0 + BKB > S;   // wave-uniform
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        if (QSPLIT > 1 && kb % QSPLIT != kpart) continue;
        if (causal && key0 + kb * 32 > q_hi) continue;   // block above every query of the wave
        //   S^T = K Q^T, dP^T = V dO^T   (lane owns query `myq`, 16 key rows)
        f32x16 sacc, pacc;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          sacc[r] = 0.f;
          pacc[r] = 0.f;
        }
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
          sacc = mfma32(RT::row_frag(ks, kb * 32, kk, lane), qf[kk], sacc);
          pacc = mfma32(RT::row_frag(vs, kb * 32, kk, lane), of[kk], pacc);
        }
        //   dS^T = P^T (dP^T - D),  P^T = exp2(s*scale*log2e - LSE2)
        float ds[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float p = fast_exp2(fmaf(sacc[r], c, -l2));
          if (need_mask) {
            const int key = key0 + kb * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
            p = key < klim ? p : 0.f;
          }
          ds[r] = p * (pacc[r] - dl);
        }
        half8 dsf[2];
#pragma unroll
        for (int kc = 0; kc < 2; ++kc)
          dsf[kc] = pack8(ds[8 * kc], ds[8 * kc + 1], ds[8 * kc + 2], ds[8 * kc + 3],
                          ds[8 * kc + 4], ds[8 * kc + 5], ds[8 * kc + 6], ds[8 * kc + 7]);
        //   dQ^T += K^T dS^T   (K^T read transposed, keys in accumulator order)
#pragma unroll
        for (int kc = 0; kc < 2; ++kc)
#pragma unroll
          for (int db = 0; db < DB; ++db)
            dqacc[db] = mfma32(RT::template tr_frag<true>(ks, kb * 32 + kc * 16, db * 32, lane),
                               dsf[kc], dqacc[db]);
      }
    }

    // next slice resident for every wave; nobody reads this stage any more
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  }

  if constexpr (QSPLIT > 1) {
    // every stage is free after the loop's last barrier; the partner waves'
    // accumulators go through LDS in the accumulator layout (lane-major
    // float4, conflict-free) and are added in share order
    float4* red = reinterpret_cast<float4*>(smem);
    for (int part = QSPLIT - 1; part >= 1; --part) {
      if (kpart == part) {
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int rq = 0; rq < 4; ++rq)
            red[((qg * DB + db) * 4 + rq) * 64 + lane] =
                make_float4(dqacc[db][4 * rq], dqacc[db][4 * rq + 1], dqacc[db][4 * rq + 2],
                            dqacc[db][4 * rq + 3]);
      }
      __syncthreads();
      if (kpart == part - 1) {
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int rq = 0; rq < 4; ++rq) {
            const float4 v = red[((qg * DB + db) * 4 + rq) * 64 + lane];
            dqacc[db][4 * rq] += v.x;
            dqacc[db][4 * rq + 1] += v.y;
            dqacc[db][4 * rq + 2] += v.z;
            dqacc[db][4 * rq + 3] += v.w;
          }
      }
      __syncthreads();
    }
    if (kpart != 0) return;
  }

  // ---- dQ = scale * acc -> FP16 ----
  if (myq < S) {
    lt_half* qp = dQ + ((int64_t)b * S + myq) * dq_stride + (int64_t)h * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        half4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (_Float16)(dqacc[db][4 * rq + e] * scale);
        *reinterpret_cast<half4*>(qp + db * 32 + 8 * rq + 4 * g) = o;
      }
  }
}

// ------------------------------------------------------------ kernel 1: row terms
// D_i = rowsum(dO_i * O_i) and LSE_i * log2(e), [B, Hq, S] each.  D / 8 lanes
// per row (one 16-byte chunk each), consecutive queries of one (batch, head)
// per workgroup; the row's lanes add in a fixed order (xor shuffles).
template <int D>
__global__ void __launch_bounds__(256)
attn_bwd_rowterms_kernel(const lt_half* __restrict__ O, const lt_half* __restrict__ dO,
                         int64_t o_stride, const float* __restrict__ LSE, float* __restrict__ lse2,
                         float* __restrict__ delta, int B, int S, int Hq) {
  constexpr int CPR = D / 8;
  constexpr int RPB = 256 / CPR;                   // rows per workgroup
  const int n_sb = (S + RPB - 1) / RPB;
  const int bh = blockIdx.x / n_sb;
  const int q = (blockIdx.x % n_sb) * RPB + (int)threadIdx.x / CPR;
  const int c = threadIdx.x % CPR;
  const int b = bh / Hq;
  const int h = bh % Hq;
  float part = 0.f;
  if (q < S) {
    const int64_t off = ((int64_t)b * S + q) * o_stride + (int64_t)h * D + c * 8;
    const half8 x = as_half8(ld16(dO + off));
    const half8 y = as_half8(ld16(O + off));
#pragma unroll
    for (int e = 0; e < 8; ++e) part = fmaf((float)x[e], (float)y[e], part);
  }
#pragma unroll
  for (int m = CPR / 2; m >= 1; m >>= 1) part += __shfl_xor(part, m);
  if (q < S && c == 0) {
    const int64_t ri = (int64_t)bh * S + q;
    delta[ri] = part;
    lse2[ri] = LSE[ri] * kLog2e;
  }
}

// ------------------------------------------------------------ kernel 2b: dK/dV share sum
// Grouped queries split over several dK/dV workgroups: dK = scale * sum of
// the FP32 partials, dV = sum, in split order (deterministic).  HBM-bound.
template <int D>
__global__ void __launch_bounds__(256)
attn_bwd_dkdv_sum_kernel(const float* __restrict__ part, int nsplit, lt_half* __restrict__ dK,
                         lt_half* __restrict__ dV, int64_t dkv_stride, int B, int S, int Hkv,
                         float scale) {
  constexpr int CPR = D / 8;                       // 8-element chunks per row
  const int64_t rowsz = (int64_t)B * S * Hkv * D;
  const int64_t chunks = (int64_t)B * S * Hkv * CPR;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= chunks) return;
  const int64_t e0 = gid * 8;                      // element offset in [B*S][Hkv][D]
  const int64_t bs = gid / (Hkv * CPR);
  const int kvh = (int)((gid / CPR) % Hkv);
  const int d0 = (int)(gid % CPR) * 8;
#pragma unroll
  for (int which = 0; which < 2; ++which) {
    const float* src = part + (int64_t)which * nsplit * rowsz + e0;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int t = 0; t < nsplit; ++t) {
      const float4 x = *reinterpret_cast<const float4*>(src + (int64_t)t * rowsz);
      const float4 y = *reinterpret_cast<const float4*>(src + (int64_t)t * rowsz + 4);
      acc[0] += x.x; acc[1] += x.y; acc[2] += x.z; acc[3] += x.w;
      acc[4] += y.x; acc[5] += y.y; acc[6] += y.z; acc[7] += y.w;
    }
    const float f = which == 0 ? scale : 1.f;
    const half8 o = pack8(acc[0] * f, acc[1] * f, acc[2] * f, acc[3] * f, acc[4] * f, acc[5] * f,
                          acc[6] * f, acc[7] * f);
    lt_half* dst = (which == 0 ? dK : dV) + bs * dkv_stride + (int64_t)kvh * D + d0;
    st16(dst, as_u32x4(o));
  }
}

template <int D>
hipError_t launch_bwd(const AttnBwdArgs& a, hipStream_t s) {
  const AttnShape& sh = a.sh;
  const int64_t nblk = attn_bwd_ds_blocks(sh.S, sh.causal);
  // 1. D and the base-2 LSE, read by the dK/dV pass
  {
    constexpr int rpb = 256 / (D / 8);
    const int64_t grid = (int64_t)sh.B * sh.Hq * ((sh.S + rpb - 1) / rpb);
    hipLaunchKernelGGL((attn_bwd_rowterms_kernel<D>), dim3((unsigned)grid), dim3(256), 0, s, a.O,
                       a.dO, a.o_stride, a.LSE, a.lse2, a.delta, sh.B, sh.S, sh.Hq);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  // 2. dK, dV (and their share sum), storing dS
  const int n_kt = (sh.S + a.ktile - 1) / a.ktile;
  const dim3 kgrid((unsigned)(n_kt * sh.B * sh.Hkv * a.nsplit));
  if (a.ktile == BKV)
    hipLaunchKernelGGL((attn_bwd_dkdv_kernel<D, 1, false>), kgrid, dim3(NWA * 64), 0, s, a.Q,
                       a.K, a.V, a.q_stride, a.kv_stride, a.dO, a.o_stride, a.lse2, a.delta, a.dK,
                       a.dV, a.dkv_stride, a.ds, nullptr, nblk, a.part, a.nsplit, sh.B, sh.S,
                       sh.Hq, sh.Hkv, sh.scale, sh.causal);
  else if (a.ktile == BKV / 2)
    hipLaunchKernelGGL((attn_bwd_dkdv_kernel<D, 2, false>), kgrid, dim3(NWA * 64), 0, s, a.Q,
                       a.K, a.V, a.q_stride, a.kv_stride, a.dO, a.o_stride, a.lse2, a.delta, a.dK,
                       a.dV, a.dkv_stride, a.ds, nullptr, nblk, a.part, a.nsplit, sh.B, sh.S,
                       sh.Hq, sh.Hkv, sh.scale, sh.causal);
  else
    return hipErrorInvalidValue;
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.nsplit > 1) {
    const int64_t chunks = (int64_t)sh.B * sh.S * sh.Hkv * (D / 8);
    hipLaunchKernelGGL((attn_bwd_dkdv_sum_kernel<D>), dim3((unsigned)((chunks + 255) / 256)),
                       dim3(256), 0, s, a.part, a.nsplit, a.dK, a.dV, a.dkv_stride, sh.B, sh.S,
                       sh.Hkv, sh.scale);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  // 3. dQ from the stored dS, longest query tiles first
  const int n_qt = (sh.S + BQQ - 1) / BQQ;
  hipLaunchKernelGGL((attn_bwd_dq_kernel<D>), dim3((unsigned)(n_qt * sh.B * sh.Hq)),
                     dim3(NWQ * 64), 0, s, a.K, a.kv_stride, a.ds, nblk, a.dQ, a.dq_stride, sh.B,
                     sh.S, sh.Hq, sh.Hkv, sh.scale, sh.causal);
  return hipGetLastError();
}

template <int D>
hipError_t launch_save_p(const AttnSavePArgs& a, hipStream_t s) {
  const AttnShape& sh = a.sh;
  const int n_kt = (sh.S + BKV - 1) / BKV;
  hipLaunchKernelGGL((attn_save_p_kernel<D>), dim3((unsigned)(n_kt * sh.B * sh.Hq)),
                     dim3(NWA * 64), 0, s, a.Q, a.K, a.q_stride, a.kv_stride, a.LSE, a.P,
                     attn_bwd_ds_blocks(sh.S, sh.causal), sh.B, sh.S, sh.Hq, sh.Hkv, sh.scale,
                     sh.causal);
  return hipGetLastError();
}

// The saved-P backward: dQ with S and dP recomputed (it also stores D and the
// base-2 LSE), then dK and dV from the saved P, then their share sum.
template <int D>
hipError_t launch_bwd_p(const AttnBwdArgs& a, hipStream_t s) {
  const AttnShape& sh = a.sh;
  const int64_t wgs256 = (int64_t)((sh.S + BQB - 1) / BQB) * sh.B * sh.Hq;
  if (wgs256 >= kDqFillWgs) {
    const int n_qt = (sh.S + BQB - 1) / BQB;
    hipLaunchKernelGGL((attn_bwd_dq_recompute_kernel<D, 1>), dim3((unsigned)(n_qt * sh.B * sh.Hq)),
                       dim3(NW * 64), 0, s, a.Q, a.K, a.V, a.q_stride, a.kv_stride, a.O, a.dO,
                       a.o_stride, a.LSE, a.lse2, a.delta, a.dQ, a.dq_stride, sh.B, sh.S, sh.Hq,
                       sh.Hkv, sh.scale, sh.causal);
  } else {
    const int n_qt = (sh.S + BQB / 2 - 1) / (BQB / 2);
    hipLaunchKernelGGL((attn_bwd_dq_recompute_kernel<D, 2>), dim3((unsigned)(n_qt * sh.B * sh.Hq)),
                       dim3(NW * 64), 0, s, a.Q, a.K, a.V, a.q_stride, a.kv_stride, a.O, a.dO,
                       a.o_stride, a.LSE, a.lse2, a.delta, a.dQ, a.dq_stride, sh.B, sh.S, sh.Hq,
                       sh.Hkv, sh.scale, sh.causal);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t nblk = attn_bwd_ds_blocks(sh.S, sh.causal);
  const int n_kt = (sh.S + a.ktile - 1) / a.ktile;
  const dim3 kgrid((unsigned)(n_kt * sh.B * sh.Hkv * a.nsplit));
  if (a.ktile == BKV)
    hipLaunchKernelGGL((attn_bwd_dkdv_kernel<D, 1, true>), kgrid, dim3(NWA * 64), 0, s, a.Q, a.K,
                       a.V, a.q_stride, a.kv_stride, a.dO, a.o_stride, a.lse2, a.delta, a.dK,
                       a.dV, a.dkv_stride, nullptr, a.psaved, nblk, a.part, a.nsplit, sh.B, sh.S,
                       sh.Hq, sh.Hkv, sh.scale, sh.causal);
  else if (a.ktile == BKV / 2)
    hipLaunchKernelGGL((attn_bwd_dkdv_kernel<D, 2, true>), kgrid, dim3(NWA * 64), 0, s, a.Q, a.K,
                       a.V, a.q_stride, a.kv_stride, a.dO, a.o_stride, a.lse2, a.delta, a.dK,
                       a.dV, a.dkv_stride, nullptr, a.psaved, nblk, a.part, a.nsplit, sh.B, sh.S,
                       sh.Hq, sh.Hkv, sh.scale, sh.causal);
  else
    return hipErrorInvalidValue;
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.nsplit > 1) {
    const int64_t chunks = (int64_t)sh.B * sh.S * sh.Hkv * (D / 8);
    hipLaunchKernelGGL((attn_bwd_dkdv_sum_kernel<D>), dim3((unsigned)((chunks + 255) / 256)),
                       dim3(256), 0, s, a.part, a.nsplit, a.dK, a.dV, a.dkv_stride, sh.B, sh.S,
                       sh.Hkv, sh.scale);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace

hipError_t attn_save_p_launch(const AttnSavePArgs& a, hipStream_t s) {
  if (a.sh.D == 128) return launch_save_p<128>(a, s);
  return launch_save_p<64>(a, s);
}

hipError_t attn_bwd_p_launch(const AttnBwdArgs& a, hipStream_t s) {
  if (a.sh.D == 128) return launch_bwd_p<128>(a, s);
  return launch_bwd_p<64>(a, s);
}

hipError_t attn_bwd_launch(const AttnBwdArgs& a, hipStream_t s) {
  if (a.sh.D == 128) return launch_bwd<128>(a, s);
  return launch_bwd<64>(a, s);
}

}  // namespace lt
