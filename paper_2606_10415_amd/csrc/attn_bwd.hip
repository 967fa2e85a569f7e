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
//   1. attn_bwd_pre   : D_i = rowsum(dO_i * O_i) (one 8/16-lane group per row,
//                       lane-group shuffle reduction) and zeroing of the FP32
//                       dQ accumulator.  HBM-bound.
//   2. attn_bwd_main  : one workgroup per (batch, kv head, 128-key tile); the
//                       4 waves own 32 keys each and keep K, V fragments and
//                       the dK, dV accumulators in registers for the whole
//                       loop over the GQA group's query heads and the causal
//                       query tiles (the paper's GSM reduction of GV / GK
//                       becomes register accumulation inside the workgroup,
//                       and the GQA sum over query heads is the same loop).
//                       Q, dO and their transposes are staged through LDS in
//                       64-query tiles (the next tile's global loads overlap
//                       the current tile's MFMA work); S = Q K^T and
//                       dP = dO V^T put one key per lane, so P and dS feed the
//                       dV / dK MFMAs straight from registers; dS goes through
//                       LDS once for dQ = dS K, whose FP32 partials are added
//                       to the workspace with global atomics.
//   3. attn_bwd_dq    : dQ = scale * accumulator -> FP16.  HBM-bound.
#include "common.hpp"
#include "kernels.hpp"

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
                    float* __restrict__ delta, float* __restrict__ dq_acc, int B, int S, int Hq) {
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
    delta[(b * Hq + h) * S + i] = s;
  }
}

// ------------------------------------------------------------ kernel 2
template <int D>
struct BwdSmem {
  static constexpr int ROW_B = D * 2;               // Q / dO row (features contiguous)
  static constexpr int QT_ROWB = BQ * 2;            // Q^T / dO^T row (64 queries = 128 B)
  static constexpr int DS_ROWB = BKV * 2;           // dS row (128 keys = 256 B)
  static constexpr int KT_ROWB = BKV * 2;           // K^T row (128 keys = 256 B)
  static constexpr int Q_OFF = 0;
  static constexpr int DO_OFF = Q_OFF + BQ * ROW_B;
  static constexpr int QT_OFF = DO_OFF + BQ * ROW_B;
  static constexpr int DOT_OFF = QT_OFF + D * QT_ROWB;
  static constexpr int LSE_OFF = DOT_OFF + D * QT_ROWB;
  static constexpr int DEL_OFF = LSE_OFF + BQ * 4;
  static constexpr int DS_OFF = DEL_OFF + BQ * 4;
  static constexpr int KT_OFF = DS_OFF + BQ * DS_ROWB;
  static constexpr int BYTES = KT_OFF + D * KT_ROWB;
};

// 16-byte chunk c of a row r at chunk c ^ (r & 7); 8-byte unit u at u ^ (r & 15).
__device__ __forceinline__ int cswz(int r, int c) { return c ^ (r & 7); }
__device__ __forceinline__ int uswz(int r, int u) { return u ^ (r & 15); }

// Write 8 consecutive halves (16 bytes, 8-byte units 2k and 2k+1 of a row whose
// units are swizzled by uswz) into row r of a transposed tile.
__device__ __forceinline__ void st_units(char* row_base, int r, int k8, u32x4 w) {
  const int s = r & 15;
  const int u = (2 * k8) ^ s;
  if (s & 1) w = u32x4{w[2], w[3], w[0], w[1]};
  *reinterpret_cast<u32x4*>(row_base + (u & ~1) * 8) = w;
}

// A-operand read from a transposed tile: 8 halves at columns
// c0 + 4g .. c0 + 4g + 3 and c0 + 8 + 4g .. c0 + 8 + 4g + 3 of row r.
__device__ __forceinline__ half8 ld_perm8(const char* row_base, int r, int c0, int g) {
  const int u0 = c0 / 4 + g;
  const u32x2 lo = *reinterpret_cast<const u32x2*>(row_base + uswz(r, u0) * 8);
  const u32x2 hi = *reinterpret_cast<const u32x2*>(row_base + uswz(r, u0 + 2) * 8);
  return as_half8(u32x4{lo[0], lo[1], hi[0], hi[1]});
}

// Per-thread staging of one query tile: thread t < 128 owns one 8x8 block of
// Q, thread t >= 128 one of dO (8 queries x 8 features); threads < BQ also
// fetch LSE (as log2) and D for one query.
template <int D>
struct QLoader {
  static_assert((BQ / 8) * (D / 8) <= 128, "one block per thread");
  static constexpr int NBLK = (BQ / 8) * (D / 8);
  u32x4 v[8];
  float lse2, dl;

  __device__ __forceinline__ void load(const lt_half* __restrict__ Q, const lt_half* __restrict__ dO,
                                       int64_t q_stride, int64_t o_stride, const float* __restrict__ LSE,
                                       const float* __restrict__ delta, int b, int h, int S, int Hq,
                                       int qbase, int tid) {
    const bool isdo = tid >= 128;
    const int blk = tid & 127;
    if (blk < NBLK) {
      const int db = blk % (D / 8);
      const int qb = blk / (D / 8);
      const lt_half* base = isdo ? dO : Q;
      const int64_t stride = isdo ? o_stride : q_stride;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int q = qbase + qb * 8 + j;
        v[j] = q < S ? ld16(base + ((int64_t)b * S + q) * stride + (int64_t)h * D + db * 8)
                     : u32x4{0, 0, 0, 0};
      }
    }
    if (tid < BQ) {
      const int q = qbase + tid;
      const int64_t idx = ((int64_t)b * Hq + h) * S + q;
      lse2 = q < S ? LSE[idx] * kLog2e : INFINITY;
      dl = q < S ? delta[idx] : 0.f;
    }
  }

  __device__ __forceinline__ void store(char* smem, int tid) {
    using SM = BwdSmem<D>;
    const bool isdo = tid >= 128;
    const int blk = tid & 127;
    if (blk < NBLK) {
      const int db = blk % (D / 8);
      const int qb = blk / (D / 8);
      char* rows = smem + (isdo ? SM::DO_OFF : SM::Q_OFF);
      char* trows = smem + (isdo ? SM::DOT_OFF : SM::QT_OFF);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int r = qb * 8 + j;
        *reinterpret_cast<u32x4*>(rows + r * SM::ROW_B + cswz(r, db) * 16) = v[j];
      }
      u32x4 t[8];
      transpose8x8(v, t);     // t[c] = queries qb*8..+7 of feature db*8+c
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const int r = db * 8 + c;
        st_units(trows + r * SM::QT_ROWB, r, qb, t[c]);
      }
    }
    if (tid < BQ) {
      reinterpret_cast<float*>(smem + SM::LSE_OFF)[tid] = lse2;
      reinterpret_cast<float*>(smem + SM::DEL_OFF)[tid] = dl;
    }
  }
};

template <int D>
__global__ void __launch_bounds__(NW * 64)
attn_bwd_main_kernel(const lt_half* __restrict__ Q, const lt_half* __restrict__ K,
                     const lt_half* __restrict__ V, int64_t q_stride, int64_t kv_stride,
                     const lt_half* __restrict__ dO, int64_t o_stride, const float* __restrict__ LSE,
                     const float* __restrict__ delta, float* __restrict__ dq_acc,
                     lt_half* __restrict__ dK, lt_half* __restrict__ dV, int64_t dkv_stride, int B,
                     int S, int Hq, int Hkv, float scale, int causal) {
  using SM = BwdSmem<D>;
  constexpr int KK = D / 16;       // MFMA steps over the head dim
  constexpr int DB = D / 32;       // 32-feature blocks
  constexpr int QBS = BQ / 32;     // 32-query blocks per tile
  constexpr int DQ_BLK = DB * QBS / NW;   // dQ output blocks per wave
  static_assert(DQ_BLK >= 1, "dQ blocks must cover the waves");
  __shared__ __attribute__((aligned(16))) char smem[SM::BYTES];

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
  // ---- K^T tile in LDS (A operand of dQ^T = K^T dS^T) ----
  {
    constexpr int NB = (BKV / 8) * (D / 8);
    for (int blk = tid; blk < NB; blk += NW * 64) {
      const int db = blk % (D / 8);
      const int kb = blk / (D / 8);
      u32x4 v[8], t[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int key = kbase + kb * 8 + j;
        v[j] = key < S ? ld16(Kp + (int64_t)key * kv_stride + db * 8) : u32x4{0, 0, 0, 0};
      }
      transpose8x8(v, t);
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const int r = db * 8 + c;
        *reinterpret_cast<u32x4*>(smem + SM::KT_OFF + r * SM::KT_ROWB + cswz(r, kb) * 16) = t[c];
      }
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

  QLoader<D> ql;
  if (n_iter > 0) {
    ql.load(Q, dO, q_stride, o_stride, LSE, delta, b, kvh * grp, S, Hq, qt0 * BQ, tid);
    ql.store(smem, tid);
  }
  __syncthreads();

  const float* lse_s = reinterpret_cast<const float*>(smem + SM::LSE_OFF);
  const float* del_s = reinterpret_cast<const float*>(smem + SM::DEL_OFF);

  for (int it = 0; it < n_iter; ++it) {
    const int h = kvh * grp + it / per_head;
    const int qbase = (qt0 + it % per_head) * BQ;
    const bool more = it + 1 < n_iter;
    if (more) {
      const int h1 = kvh * grp + (it + 1) / per_head;
      const int qb1 = (qt0 + (it + 1) % per_head) * BQ;
      ql.load(Q, dO, q_stride, o_stride, LSE, delta, b, h1, S, Hq, qb1, tid);
    }

    // ---- S = Q K^T, dP = dO V^T (lane owns key `mykey`) ----
    f32x16 sacc[QBS], pacc[QBS];
#pragma unroll
    for (int qb = 0; qb < QBS; ++qb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        sacc[qb][r] = 0.f;
        pacc[qb][r] = 0.f;
      }
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
#pragma unroll
      for (int qb = 0; qb < QBS; ++qb) {
        const int r = qb * 32 + lrow;
        const half8 qa = as_half8(*reinterpret_cast<const u32x4*>(
            smem + SM::Q_OFF + r * SM::ROW_B + cswz(r, kk * 2 + g) * 16));
        const half8 da = as_half8(*reinterpret_cast<const u32x4*>(
            smem + SM::DO_OFF + r * SM::ROW_B + cswz(r, kk * 2 + g) * 16));
        sacc[qb] = mfma32(qa, kf[kk], sacc[qb]);
        pacc[qb] = mfma32(da, vf[kk], pacc[qb]);
      }
    }

    // ---- P = exp(scale s - LSE), dS = P (dP - D) ----
    half8 pp[QBS][2], pds[QBS][2];
    const bool need_mask = (causal && kw0 + 31 > qbase) || kw0 + 32 > S;
#pragma unroll
    for (int qb = 0; qb < QBS; ++qb) {
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
          float pv = fast_exp2(fmaf(sacc[qb][r], c, -lv[e]));
          if (need_mask) {
            const int q = qbase + ql0 + e;
            if ((causal && mykey > q) || mykey >= S) pv = 0.f;
          }
          p[r] = pv;
          ds[r] = pv * (pacc[qb][r] - dv[e]);
        }
      }
#pragma unroll
      for (int kc = 0; kc < 2; ++kc) {
        pp[qb][kc] = pack8(p[8 * kc], p[8 * kc + 1], p[8 * kc + 2], p[8 * kc + 3], p[8 * kc + 4],
                           p[8 * kc + 5], p[8 * kc + 6], p[8 * kc + 7]);
        pds[qb][kc] = pack8(ds[8 * kc], ds[8 * kc + 1], ds[8 * kc + 2], ds[8 * kc + 3],
                            ds[8 * kc + 4], ds[8 * kc + 5], ds[8 * kc + 6], ds[8 * kc + 7]);
      }
      // dS -> LDS [query][key] for dQ
      const int keyl = wave * 32 + lrow;
#pragma unroll
      for (int kc = 0; kc < 2; ++kc)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int r = 8 * kc + e;
          const int q = qb * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
          *reinterpret_cast<_Float16*>(smem + SM::DS_OFF + q * SM::DS_ROWB +
                                       cswz(q, keyl >> 3) * 16 + (keyl & 7) * 2) = pds[qb][kc][e];
        }
    }

    // ---- dV^T += dO^T P,  dK^T += Q^T dS ----
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int r = db * 32 + lrow;
#pragma unroll
      for (int qb = 0; qb < QBS; ++qb)
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
          const half8 doT = ld_perm8(smem + SM::DOT_OFF + r * SM::QT_ROWB, r, qb * 32 + kc * 16, g);
          const half8 qT = ld_perm8(smem + SM::QT_OFF + r * SM::QT_ROWB, r, qb * 32 + kc * 16, g);
          dvacc[db] = mfma32(doT, pp[qb][kc], dvacc[db]);
          dkacc[db] = mfma32(qT, pds[qb][kc], dkacc[db]);
        }
    }

    __syncthreads();   // dS complete; Q-side tiles no longer read
    if (more) ql.store(smem, tid);

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
      const int kr = db * 32 + lrow;
      const int qr = qb * 32 + lrow;
#pragma unroll
      for (int kc = 0; kc < BKV / 16; ++kc) {
        const half8 ka = as_half8(*reinterpret_cast<const u32x4*>(
            smem + SM::KT_OFF + kr * SM::KT_ROWB + cswz(kr, kc * 2 + g) * 16));
        const half8 sa = as_half8(*reinterpret_cast<const u32x4*>(
            smem + SM::DS_OFF + qr * SM::DS_ROWB + cswz(qr, kc * 2 + g) * 16));
        acc = mfma32(sa, ka, acc);
      }
      float* dst = dq_acc + ((int64_t)b * S * Hq + h) * D + db * 32 + lrow;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int q = qbase + qb * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
        if (q < S) unsafeAtomicAdd(dst + (int64_t)q * Hq * D, acc[r]);
      }
    }
    __syncthreads();   // next tile's Q-side data visible; dS reads done
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
                     a.o_stride, a.delta, a.dq_acc, sh.B, sh.S, sh.Hq);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int n_kt = (sh.S + BKV - 1) / BKV;
  hipLaunchKernelGGL((attn_bwd_main_kernel<D>), dim3((unsigned)(n_kt * sh.B * sh.Hkv)),
                     dim3(NW * 64), 0, s, a.Q, a.K, a.V, a.q_stride, a.kv_stride, a.dO, a.o_stride,
                     a.LSE, a.delta, a.dq_acc, a.dK, a.dV, a.dkv_stride, sh.B, sh.S, sh.Hq, sh.Hkv,
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
