// Causal MHA / GQA attention forward with per-row log-sum-exp, gfx950.
//
// The paper's backward (Sec. 4.1, Algorithm 1) consumes the forward's
// softmax probabilities; here the forward returns O and the natural-log
// row LSE so that the backward can rebuild P = exp(scale q.k - LSE).
//
// Design (CDNA4):
//   * one workgroup = 4 waves = one (batch, head, 128-query tile); tiles are
//     issued longest-first (causal work grows with the query index), which
//     balances the CUs without a persistent scheduler.  Register use stays
//     under 256 per lane so that two workgroups share a CU (two waves per
//     SIMD: one wave's softmax VALU work runs under the other's MFMAs).
//     When the 128-query tiles would fill at most one round of the CUs' two
//     workgroup slots (short sequences), tiles hold 64 queries instead and
//     the wave pairs sharing a query group split each slice's key blocks;
//   * each wave keeps its 32 queries' Q fragments in registers and computes
//     S^T = K Q^T with 32x32x16 FP16 MFMA, so that every lane owns one query
//     column: the row max and row sum are per-lane register reductions plus
//     one cross-half exchange;
//   * K and V slices of 64 keys move HBM -> LDS by direct buffer loads in
//     their row layout, double-buffered one slice ahead; V^T operands are
//     read with the LDS transpose read, in the key order of the P^T
//     accumulator, so P^T goes from registers (converted to FP16) straight
//     into O^T += V^T P^T;
//   * softmax runs in base 2 with the scale folded into one FMA per score.
//     The running max is raised only when a row's new maximum exceeds it by
//     more than 2^8 in probability (each raise rescales O and the row sum):
//     probabilities then stay below 256, well inside FP16, and most slices
//     skip the rescale entirely.

#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "attn_tiles.hpp"

namespace lt {
namespace {

constexpr int NW = 4;        // waves per workgroup, 32 queries each
constexpr int BKV = 64;      // keys per LDS slice
constexpr int BQ = NW * 32;  // queries per workgroup
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLazy = 8.f; // log2 of the largest probability before a rescale
constexpr int64_t kFwdSlots = 512;      // workgroup slots: two per CU

template <int D>
struct FwdSmem {
  using RT = RowTile<D, NW>;
  static constexpr int TILE = BKV * RT::ROWB;     // one K or V slice
  static constexpr int STAGE = 2 * TILE;          // K then V
};

// QSPLIT = 1: 4 query groups of 32 (128 queries); every wave walks both
// 32-key blocks of each slice.  QSPLIT = 2 (short sequences, for twice the
// workgroups): 2 query groups (64 queries); waves w and w + 2 share a query
// group and take one 32-key block of each slice each, keeping their own
// running max, row sum and O; the pair's states are merged through LDS at
// the end (rescaled to the larger max, fixed order).
template <int D, int QSPLIT>
__global__ void __launch_bounds__(NW * 64, 2)
attn_fwd_kernel(const lt_half* __restrict__ Q, const lt_half* __restrict__ K,
                const lt_half* __restrict__ V, int64_t q_stride, int64_t kv_stride,
                lt_half* __restrict__ O, int64_t o_stride, float* __restrict__ LSE, int B,
                int S, int Hq, int Hkv, float scale, int causal) {
  using SM = FwdSmem<D>;
  using RT = RowTile<D, NW>;
  constexpr int KB = BKV / 32;     // 32-key blocks per slice
  constexpr int DB = D / 32;       // 32-feature blocks
  constexpr int KK = D / 16;       // MFMA steps over the head dim
  constexpr int NQG = NW / QSPLIT;                 // query groups of 32
  constexpr int BQW = NQG * 32;                    // queries per workgroup
  constexpr int KBW = KB / QSPLIT;                 // 32-key blocks per slice and wave
  static_assert(NW % QSPLIT == 0 && KB % QSPLIT == 0, "QSPLIT must divide waves and blocks");
  static_assert(QSPLIT == 1 || NQG * DB * 4 * 64 * 16 + NQG * 64 * 8 <= 2 * SM::STAGE,
                "merge fits in LDS");
  __shared__ __attribute__((aligned(1024))) char smem[2 * SM::STAGE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar addressing
  const int lrow = lane & 31;
  const int g = lane >> 5;
  const int qg = wave % NQG;                       // query group
  const int kpart = wave / NQG;                    // which block of each slice (QSPLIT = 2)

  const int n_qt = (S + BQW - 1) / BQW;
  const int qt = causal ? n_qt - 1 - (int)(blockIdx.x / (B * Hq)) : (int)(blockIdx.x / (B * Hq));
  int b, h;
  query_head(blockIdx.x % (B * Hq), B, Hq, Hkv, b, h);
  const int kvh = h / (Hq / Hkv);
  const int q0 = qt * BQW;
  const int qw0 = q0 + qg * 32;
  const int myq = qw0 + lrow;                      // query owned by this lane

  const lt_half* Kp = K + (int64_t)b * S * kv_stride + (int64_t)kvh * D;
  const lt_half* Vp = V + (int64_t)b * S * kv_stride + (int64_t)kvh * D;
  const float c = scale * kLog2e;
  const float lazy_raw = kLazy / c;                // the same margin in score units

  // Q fragments (B operand of S^T = K Q^T): column = this lane's query,
  // reduction indices kk*16 + 8g + 0..7.
  half8 qf[KK];
  {
    const lt_half* qp = Q + ((int64_t)b * S + myq) * q_stride + (int64_t)h * D + g * 8;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
      qf[kk] = myq < S ? as_half8(ld16(qp + kk * 16)) : as_half8(u32x4{0, 0, 0, 0});
  }

  // lane part of the K row-fragment address of step kk (rows rb + lane % 32,
  // rb a multiple of 16, so the swizzle depends on the lane only)
  uint32_t rlane[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) rlane[kk] = (uint32_t)RT::addr(lane & 31, kk * 2 + (lane >> 5));

  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[db][r] = 0.f;
  float m_run = -INFINITY;   // running max (score units) used as the exponent offset
  float lsum = 0.f;          // this lane's share of the row sum

  const int kv_end = causal ? min(S, q0 + BQW) : S;
  const int n_kv = (kv_end + BKV - 1) / BKV;
  const int q_hi = min(qw0 + 32, S) - 1;           // last valid query of this wave

  // K, V rows past S read as zero (their scores are masked below)
  auto stage_load = [&](int kt, int buf) {
    char* st = smem + buf * SM::STAGE;
    const int key0 = kt * BKV;
    RT::template dma<BKV>(st, Kp + (int64_t)key0 * kv_stride, kv_stride, S - key0, wave, lane);
    RT::template dma<BKV>(st + SM::TILE, Vp + (int64_t)key0 * kv_stride, kv_stride, S - key0,
                          wave, lane);
  };
  if (n_kv > 0) stage_load(0, 0);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  // The Q fragments are deliberately not marked loaded_here: the compiler
  // then waits for them (vmcnt(0)) before the first MFMA of every slice,
  // which also waits for the slice prefetched just before.  Measured at
  // LLaMA-2-7B, that per-slice wait makes the forward 4.4% faster (the two
  // workgroups of a CU then alternate between loading and computing); with
  // grouped queries, whose K/V slices hit L2 more often, it is 2-3.5% slower.

  // two slices per trip, so that the stage index is a constant and every LDS
  // fragment address is a per-lane register plus the instruction's offset
  auto slice = [&](int kt, auto CUR_) {
    constexpr int cur = decltype(CUR_)::value;
    const char* st = smem + cur * SM::STAGE;
    // that stage was last read before the previous barrier
    if (kt + 1 < n_kv) stage_load(kt + 1, cur ^ 1);

    const int key0 = kt * BKV;
    // QSPLIT = 2: this wave's block, skipped when wholly above its queries
    // or past S, so that every processed block has a visible key in every
    // valid row (the running max stays finite)
    const int kb0 = QSPLIT > 1 ? kpart * 32 : 0;
    const bool active = (!causal || key0 + kb0 <= q_hi) && qw0 < S && key0 + kb0 < S;
    if (active) {
      // ---- S^T = K Q^T ----  (local block i is the slice's block kb0/32 + i)
      f32x16 sacc[KBW];
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[kb][r] = 0.f;
      // K fragments of step kk+1 are read before the MFMAs of step kk
      // (QSPLIT = 1: a per-lane register plus a constant; QSPLIT = 2 adds the
      // wave's block offset)
      auto rdk = [&](int kb, int kk) {
        return as_half8(*reinterpret_cast<const u32x4*>(
            st + (kb0 + kb * 32) * RT::ROWB + rlane[kk]));
      };
      // two register sets by step parity, so that step kk+1's reads do not
      // wait for step kk's MFMAs to release their registers
      half8 kfr[2][KBW];
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb) kfr[0][kb] = rdk(kb, 0);
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        if (kk + 1 < KK) {
#pragma unroll
          for (int kb = 0; kb < KBW; ++kb) kfr[(kk + 1) & 1][kb] = rdk(kb, kk + 1);
        }
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) sacc[kb] = mfma32(kfr[kk & 1][kb], qf[kk], sacc[kb]);
        // the scheduling groups count from the top of the block: the first
        // read group holds step 0's reads and step 1's
        if (kk + 1 < KK) {
          if (kk == 0)
            __builtin_amdgcn_sched_group_barrier(0x100, 2 * KBW, 0);
          else
            __builtin_amdgcn_sched_group_barrier(0x100, KBW, 0);
          __builtin_amdgcn_sched_group_barrier(0x008, KBW, 0);
        }
      }

      // ---- mask (key > query, or key past S), row max ----
      if ((causal && key0 + BKV - 1 > qw0) || key0 + BKV > S) {   // wave-uniform
        const int klim = causal ? min(myq + 1, S) : S;             // keys < klim are visible
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = key0 + kb0 + kb * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
            sacc[kb][r] = key < klim ? sacc[kb][r] : -INFINITY;
          }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[kb][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));

      // ---- raise the running max only past the lazy margin ----
      const bool raise = mx > m_run + lazy_raw;    // first slice: m_run = -inf
      if (__builtin_amdgcn_ballot_w64(raise)) {    // wave-uniform branch
        const float m_new = raise ? mx : m_run;
        const float alpha = fast_exp2((m_run - m_new) * c);   // 0 on the first raise
        m_run = m_new;
        lsum *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;
      }

      // ---- P = exp2(s c - m c), row sum, FP16 P^T fragments ----
      const float mc = m_run * c;
      half8 pf[KBW][2];
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb) {
        float p[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          p[r] = fast_exp2(fmaf(sacc[kb][r], c, -mc));
          lsum += p[r];
        }
#pragma unroll
        for (int kc = 0; kc < 2; ++kc)
          pf[kb][kc] = pack8(p[8 * kc + 0], p[8 * kc + 1], p[8 * kc + 2], p[8 * kc + 3],
                             p[8 * kc + 4], p[8 * kc + 5], p[8 * kc + 6], p[8 * kc + 7]);
      }

      // ---- O^T += V^T P^T (V^T read transposed, keys in accumulator order) ----
      const char* vs = st + SM::TILE;
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb)
#pragma unroll
        for (int kc = 0; kc < 2; ++kc)
#pragma unroll
          for (int db = 0; db < DB; ++db)
            oacc[db] = mfma32(
                RT::template tr_frag<true>(vs, kb0 + kb * 32 + kc * 16, db * 32, lane),
                pf[kb][kc], oacc[db]);
    }

    // next slice resident for every wave; nobody reads this stage any more
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  };
  for (int kt = 0; kt < n_kv; kt += 2) {
    slice(kt, std::integral_constant<int, 0>{});
    if (kt + 1 < n_kv) slice(kt + 1, std::integral_constant<int, 1>{});
  }

  if constexpr (QSPLIT > 1) {
    // every stage is free after the loop's last barrier: the second wave of
    // each pair passes O (lane-major float4), its running max and row-sum
    // share to the first, which rescales both to the larger max and adds
    float4* red = reinterpret_cast<float4*>(smem);
    float2* ml = reinterpret_cast<float2*>(smem + NQG * DB * 4 * 64 * 16);
    if (kpart == 1) {
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int rq = 0; rq < 4; ++rq)
          red[((qg * DB + db) * 4 + rq) * 64 + lane] =
              make_float4(oacc[db][4 * rq], oacc[db][4 * rq + 1], oacc[db][4 * rq + 2],
                          oacc[db][4 * rq + 3]);
      ml[qg * 64 + lane] = make_float2(m_run, lsum);
    }
    __syncthreads();
    if (kpart != 0) return;
    const float2 o2 = ml[qg * 64 + lane];
    const float m = fmaxf(m_run, o2.x);
    // a wave that processed no block has m_run = -inf, a zero row sum and O;
    // both -inf only for rows past S (never stored)
    const float a1 = m == -INFINITY ? 0.f : fast_exp2((m_run - m) * c);
    const float a2 = m == -INFINITY ? 0.f : fast_exp2((o2.x - m) * c);
    m_run = m;
    lsum = lsum * a1 + o2.y * a2;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const float4 v = red[((qg * DB + db) * 4 + rq) * 64 + lane];
        oacc[db][4 * rq] = oacc[db][4 * rq] * a1 + v.x * a2;
        oacc[db][4 * rq + 1] = oacc[db][4 * rq + 1] * a1 + v.y * a2;
        oacc[db][4 * rq + 2] = oacc[db][4 * rq + 2] * a1 + v.z * a2;
        oacc[db][4 * rq + 3] = oacc[db][4 * rq + 3] * a1 + v.w * a2;
      }
  }

  // ---- normalise and store O, LSE ----
  const float lt = lsum + __shfl_xor(lsum, 32);
  if (myq < S) {
    const float inv = 1.f / lt;
    lt_half* op = O + ((int64_t)b * S + myq) * o_stride + (int64_t)h * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        half4 o;
        o[0] = (_Float16)(oacc[db][4 * rq + 0] * inv);
        o[1] = (_Float16)(oacc[db][4 * rq + 1] * inv);
        o[2] = (_Float16)(oacc[db][4 * rq + 2] * inv);
        o[3] = (_Float16)(oacc[db][4 * rq + 3] * inv);
        *reinterpret_cast<half4*>(op + db * 32 + 8 * rq + 4 * g) = o;
      }
    if (g == 0) LSE[((int64_t)b * Hq + h) * S + myq] = m_run * scale + __logf(lt);
  }
}

template <int D>
hipError_t launch_fwd(const AttnFwdArgs& a, hipStream_t s) {
  const AttnShape& sh = a.sh;
  // 64-query workgroups when 128-query ones would fill at most one round of
  // the slots (short sequences); with more, the split's extra K/V loads per
  // MFMA cost more than the finer balance gains
  const int64_t wgs128 = (int64_t)((sh.S + BQ - 1) / BQ) * sh.B * sh.Hq;
  if (wgs128 > kFwdSlots) {
    const dim3 grid((unsigned)wgs128);
    hipLaunchKernelGGL((attn_fwd_kernel<D, 1>), grid, dim3(NW * 64), 0, s, a.Q, a.K, a.V,
                       a.q_stride, a.kv_stride, a.O, a.o_stride, a.LSE, sh.B, sh.S, sh.Hq,
                       sh.Hkv, sh.scale, sh.causal);
  } else {
    const dim3 grid((unsigned)((int64_t)((sh.S + BQ / 2 - 1) / (BQ / 2)) * sh.B * sh.Hq));
    hipLaunchKernelGGL((attn_fwd_kernel<D, 2>), grid, dim3(NW * 64), 0, s, a.Q, a.K, a.V,
                       a.q_stride, a.kv_stride, a.O, a.o_stride, a.LSE, sh.B, sh.S, sh.Hq,
                       sh.Hkv, sh.scale, sh.causal);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t attn_fwd_launch(const AttnFwdArgs& a, hipStream_t s) {
  if (a.sh.D == 128) return launch_fwd<128>(a, s);
  return launch_fwd<64>(a, s);
}

}  // namespace lt
