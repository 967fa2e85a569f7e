// Causal MHA / GQA attention forward with per-row log-sum-exp, gfx950.
//
// The paper's backward (Sec. 4.1, Algorithm 1) consumes the forward's
// softmax probabilities; here the forward returns O and the natural-log
// row LSE so that the backward can rebuild P = exp(scale q.k - LSE).
//
// Design (CDNA4):
//   * one workgroup = 4 waves = one (batch, head, 32*QB*4-query tile);
//     tiles are issued longest-first (causal work grows with the query
//     index), which balances the 256 CUs without a persistent scheduler;
//   * each wave keeps its queries' Q fragments in registers for the whole
//     key loop and computes S^T = K Q^T with 32x32x16 FP16 MFMA, so that
//     every lane owns one query column: the row max / row sum of the online
//     softmax are per-lane register reductions plus one cross-half exchange;
//   * K (row layout) and V^T (transposed while staging, 8x8 half blocks in
//     registers) are double-buffered in LDS in 64-key slices, the next
//     slice's global loads overlapping the current slice's MFMA work;
//   * P^T is converted to FP16 in registers and fed straight back as the B
//     operand of O^T += V^T P^T; the key order inside each 16-key MFMA step
//     follows the accumulator layout, and V^T is read in the same order;
//   * softmax runs in base 2 with the scale folded into one FMA per score.
#include "common.hpp"
#include "kernels.hpp"

namespace lt {
namespace {

constexpr int NW = 4;        // waves per workgroup
constexpr int BKV = 64;      // keys per LDS slice
constexpr float kLog2e = 1.4426950408889634f;

template <int D>
struct FwdSmem {
  static constexpr int K_ROWB = D * 2;            // bytes per K row
  static constexpr int VT_ROWB = BKV * 2;         // bytes per V^T row (128)
  static constexpr int K_BYTES = BKV * K_ROWB;
  static constexpr int VT_BYTES = D * VT_ROWB;
  static constexpr int STAGE = K_BYTES + VT_BYTES;
};

// 16-byte chunk c of K row r lives at chunk c ^ (r & 7).
__device__ __forceinline__ int kswz(int r, int c) { return c ^ (r & 7); }
// 8-byte unit u of V^T row r lives at unit u ^ (r & 15).
__device__ __forceinline__ int vswz(int r, int u) { return u ^ (r & 15); }

template <int D>
struct KVLoader {
  static constexpr int KCH = BKV * D / 8;          // 16-byte chunks of a K slice
  static constexpr int KPER = KCH / (NW * 64);
  static constexpr int VBLK = (BKV / 8) * (D / 8); // 8x8 blocks of a V slice
  static_assert(KCH % (NW * 64) == 0, "K slice must split evenly");
  static_assert(VBLK <= NW * 64, "one V block per thread at most");
  u32x4 k[KPER];
  u32x4 v[8];

  __device__ __forceinline__ void load(const lt_half* __restrict__ Kp, const lt_half* __restrict__ Vp,
                                       int64_t stride, int S, int key0, int tid) {
#pragma unroll
    for (int i = 0; i < KPER; ++i) {
      const int id = tid + i * NW * 64;
      const int r = id / (D / 8);
      const int c = id % (D / 8);
      const int key = key0 + r;
      k[i] = key < S ? ld16(Kp + (int64_t)key * stride + c * 8) : u32x4{0, 0, 0, 0};
    }
    if (tid < VBLK) {
      const int db = tid % (D / 8);
      const int kb = tid / (D / 8);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int key = key0 + kb * 8 + j;
        v[j] = key < S ? ld16(Vp + (int64_t)key * stride + db * 8) : u32x4{0, 0, 0, 0};
      }
    }
  }

  __device__ __forceinline__ void store(char* stage, int tid) {
    using SM = FwdSmem<D>;
#pragma unroll
    for (int i = 0; i < KPER; ++i) {
      const int id = tid + i * NW * 64;
      const int r = id / (D / 8);
      const int c = id % (D / 8);
      *reinterpret_cast<u32x4*>(stage + r * SM::K_ROWB + kswz(r, c) * 16) = k[i];
    }
    if (tid < VBLK) {
      const int db = tid % (D / 8);
      const int kb = tid / (D / 8);
      u32x4 t[8];
      transpose8x8(v, t);   // t[c] = keys kb*8..+7 of feature db*8+c
      char* vt = stage + SM::K_BYTES;
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const int r = db * 8 + c;
        const int s = r & 15;
        const int u = (kb * 2) ^ s;          // position of the first 8-byte unit
        u32x4 w = t[c];
        if (s & 1) w = u32x4{w[2], w[3], w[0], w[1]};
        *reinterpret_cast<u32x4*>(vt + r * SM::VT_ROWB + (u & ~1) * 8) = w;
      }
    }
  }
};

template <int D, int QB>
__global__ void __launch_bounds__(NW * 64)
attn_fwd_kernel(const lt_half* __restrict__ Q, const lt_half* __restrict__ K,
                const lt_half* __restrict__ V, int64_t q_stride, int64_t kv_stride,
                lt_half* __restrict__ O, int64_t o_stride, float* __restrict__ LSE, int B,
                int S, int Hq, int Hkv, float scale, int causal) {
  using SM = FwdSmem<D>;
  constexpr int BQ = NW * QB * 32;
  constexpr int KB = BKV / 32;     // 32-key blocks per slice
  constexpr int DB = D / 32;       // 32-feature blocks
  constexpr int KK = D / 16;       // MFMA steps over the head dim
  __shared__ __attribute__((aligned(16))) char smem[2 * SM::STAGE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int lrow = lane & 31;
  const int g = lane >> 5;

  const int n_qt = (S + BQ - 1) / BQ;
  const int bh = blockIdx.x % (B * Hq);
  const int qt = causal ? n_qt - 1 - (int)(blockIdx.x / (B * Hq)) : (int)(blockIdx.x / (B * Hq));
  const int b = bh / Hq;
  const int h = bh % Hq;
  const int kvh = h / (Hq / Hkv);
  const int q0 = qt * BQ;
  const int qw0 = q0 + wave * QB * 32;

  const lt_half* Kp = K + (int64_t)b * S * kv_stride + (int64_t)kvh * D;
  const lt_half* Vp = V + (int64_t)b * S * kv_stride + (int64_t)kvh * D;
  const float c = scale * kLog2e;

  // Q fragments (B operand of S^T = K Q^T): lane owns query qw0+qb*32+lrow.
  half8 qf[QB][KK];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int q = qw0 + qb * 32 + lrow;
    const lt_half* qp = Q + ((int64_t)b * S + q) * q_stride + (int64_t)h * D + g * 8;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
      qf[qb][kk] = q < S ? as_half8(ld16(qp + kk * 16)) : as_half8(u32x4{0, 0, 0, 0});
  }

  f32x16 oacc[DB][QB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[db][qb][r] = 0.f;
  float m_raw[QB], lsum[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m_raw[qb] = -INFINITY;
    lsum[qb] = 0.f;
  }

  const int kv_end = causal ? min(S, q0 + BQ) : S;
  const int n_kv = (kv_end + BKV - 1) / BKV;
  const int q_hi = min(qw0 + QB * 32, S) - 1;    // last valid query of this wave

  KVLoader<D> ld;
  ld.load(Kp, Vp, kv_stride, S, 0, tid);
  ld.store(smem, tid);
  __syncthreads();

  for (int kt = 0; kt < n_kv; ++kt) {
    char* st = smem + (kt & 1) * SM::STAGE;
    const bool more = kt + 1 < n_kv;
    if (more) ld.load(Kp, Vp, kv_stride, S, (kt + 1) * BKV, tid);

    const int key0 = kt * BKV;
    const bool active = !causal || key0 <= q_hi;
    if (active && qw0 < S) {
      // ---- S^T = K Q^T ----
      f32x16 sacc[KB][QB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
          for (int r = 0; r < 16; ++r) sacc[kb][qb][r] = 0.f;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        half8 kf[KB];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
          const int r = kb * 32 + lrow;
          kf[kb] = as_half8(*reinterpret_cast<const u32x4*>(st + r * SM::K_ROWB +
                                                            kswz(r, kk * 2 + g) * 16));
        }
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) sacc[kb][qb] = mfma32(kf[kb], qf[qb][kk], sacc[kb][qb]);
      }

      // ---- mask, online softmax ----
      const bool need_mask = (causal && key0 + BKV - 1 > qw0) || key0 + BKV > S;
      half8 pf[KB][2][QB];
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const int q = qw0 + qb * 32 + lrow;
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            if (need_mask) {
              const int key = key0 + kb * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
              if ((causal && key > q) || key >= S) sacc[kb][qb][r] = -INFINITY;
            }
            mx = fmaxf(mx, sacc[kb][qb][r]);
          }
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_raw[qb], mx);
        const float alpha = m_raw[qb] == -INFINITY ? 0.f : fast_exp2((m_raw[qb] - m_new) * c);
        m_raw[qb] = m_new;
        const float mc = m_new * c;
        float rs = 0.f;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float p = fast_exp2(fmaf(sacc[kb][qb][r], c, -mc));
            sacc[kb][qb][r] = p;
            rs += p;
          }
        lsum[qb] = lsum[qb] * alpha + rs;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[db][qb][r] *= alpha;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
          for (int kc = 0; kc < 2; ++kc)
            pf[kb][kc][qb] = pack8(sacc[kb][qb][8 * kc + 0], sacc[kb][qb][8 * kc + 1],
                                   sacc[kb][qb][8 * kc + 2], sacc[kb][qb][8 * kc + 3],
                                   sacc[kb][qb][8 * kc + 4], sacc[kb][qb][8 * kc + 5],
                                   sacc[kb][qb][8 * kc + 6], sacc[kb][qb][8 * kc + 7]);
      }

      // ---- O^T += V^T P^T ----
      const char* vt = st + SM::K_BYTES;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int kc = 0; kc < 2; ++kc) {
          const int u0 = (kb * 32 + kc * 16) / 4 + g;   // keys k0+4g..+3, then k0+8+4g..+3
#pragma unroll
          for (int db = 0; db < DB; ++db) {
            const int r = db * 32 + lrow;
            const u32x2 lo = *reinterpret_cast<const u32x2*>(vt + r * SM::VT_ROWB + vswz(r, u0) * 8);
            const u32x2 hi = *reinterpret_cast<const u32x2*>(vt + r * SM::VT_ROWB + vswz(r, u0 + 2) * 8);
            const half8 vf = as_half8(u32x4{lo[0], lo[1], hi[0], hi[1]});
#pragma unroll
            for (int qb = 0; qb < QB; ++qb) oacc[db][qb] = mfma32(vf, pf[kb][kc][qb], oacc[db][qb]);
          }
        }
    }

    if (more) ld.store(smem + ((kt + 1) & 1) * SM::STAGE, tid);
    __syncthreads();
  }

  // ---- normalise and store O, LSE ----
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int q = qw0 + qb * 32 + lrow;
    const float lt = lsum[qb] + __shfl_xor(lsum[qb], 32);
    if (q >= S) continue;
    const float inv = 1.f / lt;
    lt_half* op = O + ((int64_t)b * S + q) * o_stride + (int64_t)h * D;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int rq = 0; rq < 4; ++rq) {
        half4 o;
        o[0] = (_Float16)(oacc[db][qb][4 * rq + 0] * inv);
        o[1] = (_Float16)(oacc[db][qb][4 * rq + 1] * inv);
        o[2] = (_Float16)(oacc[db][qb][4 * rq + 2] * inv);
        o[3] = (_Float16)(oacc[db][qb][4 * rq + 3] * inv);
        *reinterpret_cast<half4*>(op + db * 32 + 8 * rq + 4 * g) = o;
      }
    if (g == 0) LSE[((int64_t)b * Hq + h) * S + q] = m_raw[qb] * scale + __logf(lt);
  }
}

template <int D, int QB>
hipError_t launch_fwd(const AttnFwdArgs& a, hipStream_t s) {
  constexpr int BQ = NW * QB * 32;
  const AttnShape& sh = a.sh;
  const int n_qt = (sh.S + BQ - 1) / BQ;
  const dim3 grid((unsigned)(n_qt * sh.B * sh.Hq));
  hipLaunchKernelGGL((attn_fwd_kernel<D, QB>), grid, dim3(NW * 64), 0, s, a.Q, a.K, a.V,
                     a.q_stride, a.kv_stride, a.O, a.o_stride, a.LSE, sh.B, sh.S, sh.Hq, sh.Hkv,
                     sh.scale, sh.causal);
  return hipGetLastError();
}

}  // namespace

hipError_t attn_fwd_launch(const AttnFwdArgs& a, hipStream_t s) {
  if (a.sh.D == 128) return launch_fwd<128, 1>(a, s);
  return launch_fwd<64, 1>(a, s);
}

}  // namespace lt
