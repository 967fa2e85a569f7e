// Causal MHA / GQA attention backward (recomputed P), gfx950.
//
// Sec. 4.1 / Algorithm 1 of the paper: per key/value tile j and query tile i
//   GP = GO V^T,  GS = SoftmaxBackward(P, GP),  GV_j += P^T GO,
//   GQ_i += GS K,  GK_j += GS^T Q,
// with the partial GV / GK of the processing units reduced before write-back.
// Here P is rebuilt from the forward's row LSE, P = exp(scale q.k - LSE), and
// SoftmaxBackward is GS = P * (GP - D) with D_i = rowsum(GO_i * O_i).
//
// Three kernels:
//   1. attn_bwd_pre : D_i = rowsum(dO_i * O_i) (one 8/16-lane group per row,
//                     shuffle reduction), LSE in base 2, and zeroing of the
//                     FP32 dQ accumulator.  HBM-bound.
//   2. attn_bwd_main: one workgroup per (batch, kv head, 128-key tile); the
//                     4 waves own 32 keys each and keep K, V fragments and the
//                     dK, dV accumulators in registers for the whole loop over
//                     the GQA group's query heads and the causal query tiles
//                     (the paper's GSM reduction of GV / GK becomes register
//                     accumulation, and the GQA sum over query heads is the
//                     same loop).  Q and dO tiles (64 queries) stream HBM ->
//                     LDS by direct buffer loads, double-buffered one tile
//                     ahead.  S = Q K^T and dP = dO V^T put one key per lane,
//                     so P and dS feed the dV / dK MFMAs from registers; the
//                     Q^T / dO^T operands of those MFMAs are read from the
//                     same row-layout tiles with the LDS transpose read, in
//                     the reduction order of the P / dS accumulators.  dS goes
//                     to LDS once (as dS^T, 8-byte stores) for dQ = dS K, whose
//                     FP32 partials are added to the workspace with coalesced
//                     global atomics.
//   3. attn_bwd_dq  : dQ = scale * accumulator -> FP16.  HBM-bound.
#include "common.hpp"
#include "kernels.hpp"
#include "attn_tiles.hpp"

namespace lt {
namespace {

constexpr int NW = 4;          // waves per workgroup
constexpr int BKV = 128;       // keys per workgroup (32 per wave)
constexpr int BQ = 64;         // queries per inner tile
constexpr float kLog2e = 1.4426950408889634f;

// ------------------------------------------------------------ kernel 1
template <int D>
__global__ void __launch_bounds__(256)
attn_bwd_pre_kernel(const lt_half* __restrict__ O, const lt_half* __restrict__ dO, int64_t o_stride,
                    const float* __restrict__ LSE, float* __restrict__ delta,
                    float* __restrict__ lse2, float* __restrict__ dq_acc, int B, int S, int Hq) {
  constexpr int LPR = D / 8;                       // lanes per row
  const int64_t rows = (int64_t)B * S * Hq;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t row = gid / LPR;
  const int part = (int)(gid % LPR);
  float s = 0.f;
  if (row < rows) {
    const int h = (int)(row % Hq);
    const int64_t bi = row / Hq;                   // b*S + i
    const int64_t off = bi * o_stride + (int64_t)h * D + part * 8;
    const half8 o = as_half8(ld16(O + off));
    const half8 d = as_half8(ld16(dO + off));
#pragma unroll
    for (int e = 0; e < 8; ++e) s += (float)o[e] * (float)d[e];
    float4* z = reinterpret_cast<float4*>(dq_acc + row * D + part * 8);
    z[0] = make_float4(0.f, 0.f, 0.f, 0.f);
    z[1] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
#pragma unroll
  for (int m = LPR / 2; m >= 1; m >>= 1) s += __shfl_xor(s, m);
  if (row < rows && part == 0) {
    const int h = (int)(row % Hq);
    const int64_t bi = row / Hq;
    const int64_t b = bi / S;
    const int64_t i = bi % S;
    const int64_t idx = (b * Hq + h) * S + i;
    delta[idx] = s;
    lse2[idx] = LSE[idx] * kLog2e;
  }
}

// ------------------------------------------------------------ kernel 2
// dS^T [key][query] tile, 128-byte rows.  Byte offset of (key r, query q):
// the 64-byte half is XORed with bit 1 of r and the 8-byte slot inside it
// with bits 2..4 of r, so 32 consecutive keys writing one 8-byte query run
// hit 32 different bank groups, and the transpose reads of 4 consecutive keys
// land in 4 different 64-byte windows.
__device__ __forceinline__ int dst_off(int r, int q) {
  return r * (BQ * 2) + ((q * 2) ^ (((r >> 1) & 1) << 6) ^ (((r >> 2) & 7) << 3));
}

template <int D>
struct BwdSmem {
  using RT = RowTile<D, NW>;
  static constexpr int TILE_Q = BQ * RT::ROWB;
  static constexpr int DST_PITCH = BQ * 2;          // dS^T row: 64 queries
  static constexpr int K_OFF = 0;                     // K tile [BKV][D]
  static constexpr int Q_OFF = K_OFF + BKV * RT::ROWB;          // 2 buffers
  static constexpr int DO_OFF = Q_OFF + 2 * TILE_Q;             // 2 buffers
  static constexpr int LSE_OFF = DO_OFF + 2 * TILE_Q;           // 2 x BQ floats
  static constexpr int DEL_OFF = LSE_OFF + 2 * BQ * 4;          // 2 x BQ floats
  static constexpr int DST_OFF = DEL_OFF + 2 * BQ * 4;          // dS^T [BKV][BQ]
  static constexpr int BYTES = DST_OFF + BKV * DST_PITCH;
};

template <int D>
__global__ void __launch_bounds__(NW * 64)
attn_bwd_main_kernel(const lt_half* __restrict__ Q, const lt_half* __restrict__ K,
                     const lt_half* __restrict__ V, int64_t q_stride, int64_t kv_stride,
                     const lt_half* __restrict__ dO, int64_t o_stride, const float* __restrict__ lse2,
                     const float* __restrict__ delta, float* __restrict__ dq_acc,
                     lt_half* __restrict__ dK, lt_half* __restrict__ dV, int64_t dkv_stride, int B,
                     int S, int Hq, int Hkv, float scale, int causal) {
  using SM = BwdSmem<D>;
  using RT = RowTile<D, NW>;
  constexpr int KK = D / 16;       // MFMA steps over the head dim
  constexpr int DB = D / 32;       // 32-feature blocks
  constexpr int QBS = BQ / 32;     // 32-query blocks per tile
  constexpr int DQ_BLK = DB * QBS / NW;   // dQ output blocks per wave
  static_assert(DQ_BLK >= 1, "dQ blocks must cover the waves");
  __shared__ __attribute__((aligned(1024))) char smem[SM::BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int lrow = lane & 31;
  const int g = lane >> 5;

  const int bkv = blockIdx.x % (B * Hkv);
  const int jt = blockIdx.x / (B * Hkv);          // ascending key tile = descending work
  const int b = bkv / Hkv;
  const int kvh = bkv % Hkv;
  const int grp = Hq / Hkv;
  const int kbase = jt * BKV;
  const int kw0 = kbase + wave * 32;               // this wave's first key
  const int mykey = kw0 + lrow;                    // key owned by this lane (S, dP columns)

  const lt_half* Kp = K + (int64_t)b * S * kv_stride + (int64_t)kvh * D;
  const lt_half* Vp = V + (int64_t)b * S * kv_stride + (int64_t)kvh * D;

  // ---- K tile -> LDS (B operand of dQ = dS K, read transposed) ----
  RT::template dma<BKV>(smem + SM::K_OFF, Kp + (int64_t)kbase * kv_stride, kv_stride, S - kbase,
                        wave, lane);
  // ---- K, V fragments (B operands of S = Q K^T and dP = dO V^T) ----
  half8 kf[KK], vf[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    if (mykey < S) {
      kf[kk] = as_half8(ld16(Kp + (int64_t)mykey * kv_stride + kk * 16 + g * 8));
      vf[kk] = as_half8(ld16(Vp + (int64_t)mykey * kv_stride + kk * 16 + g * 8));
    } else {
      kf[kk] = as_half8(u32x4{0, 0, 0, 0});
      vf[kk] = as_half8(u32x4{0, 0, 0, 0});
    }
  }

  f32x16 dkacc[DB], dvacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      dkacc[db][r] = 0.f;
      dvacc[db][r] = 0.f;
    }

  const float c = scale * kLog2e;
  const int n_qt = (S + BQ - 1) / BQ;
  const int qt0 = causal ? kbase / BQ : 0;
  const int per_head = n_qt - qt0;
  const int n_iter = grp * per_head;

  // Query tile `it` = (query head, 64 queries).  Q, dO (rows past S read as
  // zero) and the base-2 LSE and D rows (zero past S: with zero Q and dO rows
  // those queries contribute nothing) go to LDS by direct loads.
  auto tile_of = [&](int it, int& h, int& qbase) {
    h = kvh * grp + it / per_head;
    qbase = (qt0 + it % per_head) * BQ;
  };
  auto stage = [&](int it, int buf) {
    int h, qbase;
    tile_of(it, h, qbase);
    RT::template dma<BQ>(smem + SM::Q_OFF + buf * SM::TILE_Q,
                         Q + ((int64_t)b * S + qbase) * q_stride + (int64_t)h * D, q_stride,
                         S - qbase, wave, lane);
    RT::template dma<BQ>(smem + SM::DO_OFF + buf * SM::TILE_Q,
                         dO + ((int64_t)b * S + qbase) * o_stride + (int64_t)h * D, o_stride,
                         S - qbase, wave, lane);
    if (wave < 2) {
      const float* rowp = (wave == 0 ? lse2 : delta) + ((int64_t)b * Hq + h) * S + qbase;
      const int nv = S - qbase < BQ ? S - qbase : BQ;
      lds_dma4_opaque(rowp, (uint32_t)(nv * 4),
                      smem + (wave == 0 ? SM::LSE_OFF : SM::DEL_OFF) + buf * BQ * 4,
                      (uint32_t)(lane * 4));
    }
  };

  if (n_iter > 0) stage(0, 0);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  for (int it = 0; it < n_iter; ++it) {
    const int cur = it & 1;
    int h, qbase;
    tile_of(it, h, qbase);
    const bool more = it + 1 < n_iter;
    if (more) stage(it + 1, cur ^ 1);
    const char* qs = smem + SM::Q_OFF + cur * SM::TILE_Q;
    const char* dos = smem + SM::DO_OFF + cur * SM::TILE_Q;
    const float* lse_s = reinterpret_cast<const float*>(smem + SM::LSE_OFF + cur * BQ * 4);
    const float* del_s = reinterpret_cast<const float*>(smem + SM::DEL_OFF + cur * BQ * 4);

    // One 32-query half at a time (keeps the live accumulators small):
    //   S = Q K^T, dP = dO V^T          (lane owns key `mykey`, 16 query rows)
    //   P = exp2(s*scale*log2e - LSE2), dS = P (dP - D)
    //   dS^T -> LDS;  dV^T += dO^T P,  dK^T += Q^T dS
    // (queries past S have zero Q and dO rows and zero LSE2 and D: finite P,
    // zero dS and zero contributions)
    const bool need_mask = (causal && kw0 + 31 > qbase) || kw0 + 32 > S;
    const int keyl = wave * 32 + lrow;
#pragma unroll
    for (int qb = 0; qb < QBS; ++qb) {
      f32x16 sacc, pacc;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        sacc[r] = 0.f;
        pacc[r] = 0.f;
      }
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        sacc = mfma32(RT::row_frag(qs, qb * 32, kk, lane), kf[kk], sacc);
        pacc = mfma32(RT::row_frag(dos, qb * 32, kk, lane), vf[kk], pacc);
      }

      float p[16], ds[16];
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int ql0 = qb * 32 + 8 * rq + 4 * g;
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
      if (need_mask) {   // wave-uniform: diagonal or ragged key tile
        // key > query (causal) or key past S -> P = 0
        const int qlim = causal ? mykey : 0;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int q = qbase + qb * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
          const bool masked = (q < qlim) | (mykey >= S);
          p[r] = masked ? 0.f : p[r];
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
      // dS^T row `keyl`, queries ql0..ql0+3 (8 bytes) for each 4-run
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        const int ql0 = qb * 32 + 8 * rq + 4 * g;
        const half8& src = pds[rq >> 1];
        half4 d4h;
#pragma unroll
        for (int e = 0; e < 4; ++e) d4h[e] = src[4 * (rq & 1) + e];
        *reinterpret_cast<half4*>(smem + SM::DST_OFF + dst_off(keyl, ql0)) = d4h;
      }
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
          const int kb = qb * 32 + kc * 16;
          dvacc[db] = mfma32(RT::template tr_frag<true>(dos, kb, db * 32, lane), pp[kc], dvacc[db]);
          dkacc[db] = mfma32(RT::template tr_frag<true>(qs, kb, db * 32, lane), pds[kc], dkacc[db]);
        }
    }

    __syncthreads();   // dS^T complete

    // ---- dQ (partial over this workgroup's keys) = dS K -> atomics ----
    // Result lane layout: column d (one per lane), rows q in 4-runs, so each
    // atomic instruction covers two 128-byte runs of one dQ row.
#pragma unroll
    for (int t = 0; t < DQ_BLK; ++t) {
      const int bi = wave * DQ_BLK + t;
      const int db = bi / QBS;
      const int qb = bi % QBS;
      f32x16 acc;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
      for (int kc = 0; kc < BKV / 16; ++kc) {
        // dS as A: rows q (qb*32 + lane%32), keys kc*16 + 8*(lane/32) + 0..7,
        // read transposed from dS^T[key][q]
        const int q = qb * 32 + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
        v4s part[2];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const int key = kc * 16 + 8 * (lane >> 5) + 4 * hh + ((lane & 15) >> 2);
          part[hh] = lds_read_tr16(smem + SM::DST_OFF + dst_off(key, q));
        }
        const half8 sa = as_half8(pack_v4s_pair(part[0], part[1]));
        const half8 kb = RT::template tr_frag<false>(smem + SM::K_OFF, kc * 16, db * 32, lane);
        acc = mfma32(sa, kb, acc);
      }
      // rows qbase + qb*32 + 0..31 of this head; rows past S are outside the
      // buffer and their atomics are dropped
      const int q0 = qbase + qb * 32;
      const int nv = S - q0 < 32 ? S - q0 : 32;
      const int rowb = Hq * D * 4;
      const rsrc_t rs = make_rsrc(dq_acc + (((int64_t)b * S + q0) * Hq + h) * D,
                                  nv > 0 ? (uint32_t)(nv * rowb) : 0u);
      const uint32_t lane_off = (uint32_t)((4 * g * Hq * D + db * 32 + lrow) * 4);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const uint32_t off = lane_off + (uint32_t)((8 * (r >> 2) + (r & 3)) * rowb);
        __builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(acc[r], rs, (int)off, 0, 0);
      }
    }

    // own direct loads of the next tile are done (only the dQ atomics may
    // still be in flight), then everyone's are
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(DQ_BLK * 16) : "memory");
    __syncthreads();
  }

  // ---- write dK = scale * acc, dV ----
  if (mykey < S) {
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
        const int d0 = db * 32 + 8 * rq + 4 * g;
        *reinterpret_cast<half4*>(dkp + d0) = k4;
        *reinterpret_cast<half4*>(dvp + d0) = v4;
      }
  }
}

// ------------------------------------------------------------ kernel 3
template <int D>
__global__ void __launch_bounds__(256)
attn_bwd_dq_kernel(const float* __restrict__ dq_acc, lt_half* __restrict__ dQ, int64_t dq_stride,
                   int B, int S, int Hq, float scale) {
  constexpr int LPR = D / 8;
  const int64_t rows = (int64_t)B * S * Hq;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t row = gid / LPR;
  const int part = (int)(gid % LPR);
  if (row >= rows) return;
  const int h = (int)(row % Hq);
  const int64_t bi = row / Hq;
  const float4* src = reinterpret_cast<const float4*>(dq_acc + row * D + part * 8);
  const float4 a = src[0], bb = src[1];
  const half8 o = pack8(a.x * scale, a.y * scale, a.z * scale, a.w * scale, bb.x * scale,
                        bb.y * scale, bb.z * scale, bb.w * scale);
  st16(dQ + bi * dq_stride + (int64_t)h * D + part * 8, as_u32x4(o));
}

template <int D>
hipError_t launch_bwd(const AttnBwdArgs& a, hipStream_t s) {
  const AttnShape& sh = a.sh;
  const int64_t rows = (int64_t)sh.B * sh.S * sh.Hq;
  const int64_t threads = rows * (D / 8);
  const unsigned eblocks = (unsigned)((threads + 255) / 256);
  hipLaunchKernelGGL((attn_bwd_pre_kernel<D>), dim3(eblocks), dim3(256), 0, s, a.O, a.dO,
                     a.o_stride, a.LSE, a.delta, a.lse2, a.dq_acc, sh.B, sh.S, sh.Hq);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int n_kt = (sh.S + BKV - 1) / BKV;
  hipLaunchKernelGGL((attn_bwd_main_kernel<D>), dim3((unsigned)(n_kt * sh.B * sh.Hkv)),
                     dim3(NW * 64), 0, s, a.Q, a.K, a.V, a.q_stride, a.kv_stride, a.dO, a.o_stride,
                     a.lse2, a.delta, a.dq_acc, a.dK, a.dV, a.dkv_stride, sh.B, sh.S, sh.Hq, sh.Hkv,
                     sh.scale, sh.causal);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_bwd_dq_kernel<D>), dim3(eblocks), dim3(256), 0, s, a.dq_acc, a.dQ,
                     a.dq_stride, sh.B, sh.S, sh.Hq, sh.scale);
  return hipGetLastError();
}

}  // namespace

hipError_t attn_bwd_launch(const AttnBwdArgs& a, hipStream_t s) {
  if (a.sh.D == 128) return launch_bwd<128>(a, s);
  return launch_bwd<64>(a, s);
}

}  // namespace lt
