// RMSNorm and rotary position embedding of the LLaMA-2 / Qwen2.5 decoder
// layers the paper evaluates (Sec. 6.1), forward and backward, gfx950.
//
// All four operations are elementwise or per-row reductions: HBM-bound.
//   * rmsnorm_fwd: one wave per token row; lane l owns the 16-byte chunks
//     l, l + 64, ... of the row (coalesced), the sum of squares is a wave
//     shuffle reduction; writes y = w * x * r (one rounding) and r.
//       r = (mean_j x_j^2 + eps)^(-1/2)
//   * rmsnorm_bwd: the same row layout, 4 waves per workgroup, one row per
//     wave for short inputs and a few for long ones (at most 512
//     workgroups); per row
//       dx = r * w * g - r^3 * x / H * sum_j g_j w_j x_j   (+ residual R)
//     with g and x held in registers between the row dot product and dx
//     (rows up to 6144 columns; wider rows are read twice, the second time
//     from L2).  Every wave keeps the FP32 partial of dw = sum_rows g * x * r
//     for the rows it visits; the workgroup adds its waves' partials in wave
//     order through LDS, writes one partial row to the workspace, and
//     rmsnorm_dw_sum adds those rows in a fixed order (deterministic, no
//     atomics).
//   * rope_table: cos / sin of p * base^(-2i/D) for p < S, i < D/2, with the
//     angle formed and reduced in FP64 (positions up to 10^4 and more keep
//     full FP32 accuracy), stored as FP32 pairs.
//   * rope: in place on `heads` consecutive heads of each token row
//     (the Q and K heads of the fused QKV buffer); rotate-half pairing
//     (i, i + D/2); inverse = rotation by the negated angle (the gradient).

#include "common.hpp"
#include "kernels.hpp"

namespace lt {
namespace {

constexpr int kRowsPerWg = 4;        // rmsnorm: one wave per row, 4 waves per workgroup

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
  return v;
}

// ---------------------------------------------------------------- forward
template <int MAXK>
__global__ void __launch_bounds__(64 * kRowsPerWg)
rmsnorm_fwd_kernel(const lt_half* __restrict__ X, int64_t ldx, const lt_half* __restrict__ W,
                   lt_half* __restrict__ Y, int64_t ldy, float* __restrict__ RSTD, int64_t T,
                   int H, float eps) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * kRowsPerWg + (threadIdx.x >> 6);
  if (row >= T) return;                          // whole wave leaves together
  const int nch = H / 8;                         // 16-byte chunks per row
  const lt_half* x = X + row * ldx;
  half8 xv[MAXK];
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < MAXK; ++k) {
    const int c = lane + 64 * k;
    xv[k] = c < nch ? as_half8(ld16(x + c * 8)) : as_half8(u32x4{0, 0, 0, 0});
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += (float)xv[k][e] * (float)xv[k][e];
  }
  ss = wave_sum(ss);
  const float r = 1.f / sqrtf(ss / (float)H + eps);
  lt_half* y = Y + row * ldy;
#pragma unroll
  for (int k = 0; k < MAXK; ++k) {
    const int c = lane + 64 * k;
    if (c < nch) {
      const half8 wv = as_half8(ld16(W + c * 8));
      half8 o;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = (_Float16)((float)wv[e] * ((float)xv[k][e] * r));
      st16(y + c * 8, as_u32x4(o));
    }
  }
  if (lane == 0) RSTD[row] = r;
}

// ---------------------------------------------------------------- backward
// Workgroup = kBwdWaves waves over a contiguous range of rows; wave w takes
// rows row0 + w, row0 + w + kBwdWaves, ...  Every wave accumulates its dw
// partial for all columns in registers; at the end the workgroup adds its
// waves' partials in wave order through LDS (8 columns per lane at a time)
// and writes one partial row, blockIdx.x, of the workspace [nblk][H] FP32.
constexpr int kBwdWaves = kRmsBwdWaves;

template <int MAXK, bool ONEPASS>
__global__ void __launch_bounds__(64 * kBwdWaves)
rmsnorm_bwd_kernel(const lt_half* __restrict__ dY, int64_t lddy, const lt_half* __restrict__ X,
                   int64_t ldx, const lt_half* __restrict__ W, const float* __restrict__ RSTD,
                   const lt_half* __restrict__ R, int64_t ldr, lt_half* __restrict__ dX,
                   int64_t lddx, float* __restrict__ part, int64_t T, int H, int rows_per_wg) {
  __shared__ float red[kBwdWaves][64 * 8];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int nch = H / 8;
  const int64_t row0 = (int64_t)blockIdx.x * rows_per_wg;
  const int64_t row_end = row0 + rows_per_wg < T ? row0 + rows_per_wg : T;
  const float inv_h = 1.f / (float)H;

  float dw[MAXK][8];
#pragma unroll
  for (int k = 0; k < MAXK; ++k)
#pragma unroll
    for (int e = 0; e < 8; ++e) dw[k][e] = 0.f;

  // ONEPASS: the row's g and x stay in registers between the dot product
  // and dx; otherwise (wide rows) the second pass re-reads them (L2).
  for (int64_t row = row0 + wave; row < row_end; row += kBwdWaves) {
    const float r = RSTD[row];
    const lt_half* gp = dY + row * lddy;
    const lt_half* xp = X + row * ldx;
    half8 gk[ONEPASS ? MAXK : 1], xk[ONEPASS ? MAXK : 1], rk[ONEPASS ? MAXK : 1];
    float dot = 0.f;
#pragma unroll
    for (int k = 0; k < MAXK; ++k) {
      const int c = lane + 64 * k;
      half8 gv = as_half8(u32x4{0, 0, 0, 0}), xv = gv, rv = gv;
      if (c < nch) {
        gv = as_half8(ld16(gp + c * 8));
        xv = as_half8(ld16(xp + c * 8));
        // rows up to 4096 columns: the residual row is loaded with g and x
        // (one memory latency per row); wider rows load it later, for registers
        if (ONEPASS && MAXK <= 8 && R) rv = as_half8(ld16(R + row * ldr + c * 8));
        const half8 wv = as_half8(ld16(W + c * 8));
#pragma unroll
        for (int e = 0; e < 8; ++e) dot += (float)gv[e] * (float)wv[e] * (float)xv[e];
      }
      if constexpr (ONEPASS) {
        gk[k] = gv;
        xk[k] = xv;
        rk[k] = rv;
      }
    }
    dot = wave_sum(dot);
    const float c3 = r * r * r * dot * inv_h;
#pragma unroll
    for (int k = 0; k < MAXK; ++k) {
      const int c = lane + 64 * k;
      if (c < nch) {
        const half8 gv = ONEPASS ? gk[k] : as_half8(ld16(gp + c * 8));
        const half8 xv = ONEPASS ? xk[k] : as_half8(ld16(xp + c * 8));
        const half8 wv = as_half8(ld16(W + c * 8));
        half8 rv = as_half8(u32x4{0, 0, 0, 0});
        if (ONEPASS && MAXK <= 8) rv = rk[k];
        else if (R) rv = as_half8(ld16(R + row * ldr + c * 8));
        half8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float g = (float)gv[e], x = (float)xv[e];
          dw[k][e] += g * x * r;
          o[e] = (_Float16)((float)rv[e] + (r * (float)wv[e] * g - c3 * x));
        }
        st16(dX + row * lddx + c * 8, as_u32x4(o));
      }
    }
  }

  // workgroup sum of the waves' partials, 512 columns at a time, in wave order
  float* dst = part + (int64_t)blockIdx.x * H;
#pragma unroll
  for (int k = 0; k < MAXK; ++k) {
    if (64 * k >= nch) break;                       // uniform
#pragma unroll
    for (int e = 0; e < 8; ++e) red[wave][lane * 8 + e] = dw[k][e];
    __syncthreads();
    // columns 512 k + t, t = thread, thread + 64 kBwdWaves, ...
#pragma unroll
    for (int t = threadIdx.x; t < 512; t += 64 * kBwdWaves) {
      if (64 * k + t / 8 < nch) {
        float sum = 0.f;
#pragma unroll
        for (int v = 0; v < kBwdWaves; ++v) sum += red[v][t];
        dst[512 * k + t] = sum;
      }
    }
    __syncthreads();
  }
}

// dW[j] = sum over the partial rows; FP16 result.  Workgroup = 16 waves over
// 64 columns (lane = column, coalesced): wave v sums partial rows v, v + 16,
// ... in order (eight loads in flight at a time), then wave 0 adds the 16
// wave sums in order (deterministic).
constexpr int kSumWaves = 16;

__global__ void __launch_bounds__(64 * kSumWaves)
rmsnorm_dw_sum_kernel(const float* __restrict__ part, int nparts, int H, lt_half* __restrict__ dW) {
  __shared__ float red[kSumWaves][64];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int j = blockIdx.x * 64 + lane;
  float s = 0.f;
  if (j < H) {
    // eight partial rows loaded together, added in row order
    for (int t = wave; t < nparts; t += 8 * kSumWaves) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int tu = t + u * kSumWaves;
        v[u] = tu < nparts ? part[(int64_t)tu * H + j] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) s += v[u];
    }
  }
  red[wave][lane] = s;
  __syncthreads();
  if (wave == 0 && j < H) {
    float tot = 0.f;
#pragma unroll
    for (int v = 0; v < kSumWaves; ++v) tot += red[v][lane];
    reinterpret_cast<_Float16*>(dW)[j] = (_Float16)tot;
  }
}

// ---------------------------------------------------------------- rotary
__global__ void __launch_bounds__(256)
rope_table_kernel(float* __restrict__ CS, int S, int D, double base) {
  const int half = D / 2;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)S * half) return;
  const int p = (int)(idx / half);
  const int i = (int)(idx % half);
  const double theta = pow(base, -2.0 * (double)i / (double)D);
  const double a = fmod((double)p * theta, 6.283185307179586476925286766559);
  double s, c;
  sincos(a, &s, &c);
  CS[2 * idx] = (float)c;
  CS[2 * idx + 1] = (float)s;
}

// One thread: 8 consecutive pair indices i (and their partners i + D/2) of
// one head of one token.
__global__ void __launch_bounds__(256)
rope_kernel(lt_half* __restrict__ X, int64_t stride, int64_t T, int S, int heads, int D,
            const float* __restrict__ CS, float sign) {
  const int half = D / 2;
  const int gph = half / 8;                      // 8-pair groups per head
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= T * heads * gph) return;
  const int gi = (int)(idx % gph);
  const int64_t th = idx / gph;
  const int h = (int)(th % heads);
  const int64_t t = th / heads;                  // token row b*S + p
  const int p = (int)(t % S);
  lt_half* x = X + t * stride + (int64_t)h * D + gi * 8;
  const half8 x1 = as_half8(ld16(x));
  const half8 x2 = as_half8(ld16(x + half));
  const float4* cs = reinterpret_cast<const float4*>(CS + ((int64_t)p * half + gi * 8) * 2);
  half8 y1, y2;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 v = cs[q];                      // (cos, sin) of pairs 2q, 2q + 1
    const float cc[2] = {v.x, v.z};
    const float ss[2] = {sign * v.y, sign * v.w};
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int e = 2 * q + u;
      const float a = (float)x1[e], b = (float)x2[e];
      y1[e] = (_Float16)(a * cc[u] - b * ss[u]);
      y2[e] = (_Float16)(b * cc[u] + a * ss[u]);
    }
  }
  st16(x, as_u32x4(y1));
  st16(x + half, as_u32x4(y2));
}

template <int MAXK>
hipError_t launch_rms_fwd(const lt_half* X, int64_t ldx, const lt_half* W, lt_half* Y, int64_t ldy,
                          float* RSTD, int64_t T, int64_t H, float eps, hipStream_t s) {
  const unsigned grid = (unsigned)((T + kRowsPerWg - 1) / kRowsPerWg);
  hipLaunchKernelGGL((rmsnorm_fwd_kernel<MAXK>), dim3(grid), dim3(64 * kRowsPerWg), 0, s, X, ldx,
                     W, Y, ldy, RSTD, T, (int)H, eps);
  return hipGetLastError();
}

template <int MAXK, bool ONEPASS>
hipError_t launch_rms_bwd(const RmsBwdArgs& a, hipStream_t s) {
  const int nblk = rmsnorm_bwd_blocks(a.T);
  const int rows_per_wg = (int)((a.T + nblk - 1) / nblk);
  hipLaunchKernelGGL((rmsnorm_bwd_kernel<MAXK, ONEPASS>), dim3((unsigned)nblk), dim3(64 * kBwdWaves), 0, s,
                     a.dY, a.lddy, a.X, a.ldx, a.W, a.RSTD, a.R, a.ldr, a.dX, a.lddx, a.part, a.T,
                     (int)a.H, rows_per_wg);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(rmsnorm_dw_sum_kernel, dim3((unsigned)((a.H + 63) / 64)), dim3(64 * kSumWaves),
                     0, s, a.part, nblk, (int)a.H, a.dW);
  return hipGetLastError();
}

}  // namespace

// H <= 8192 (validated by the caller): up to 16 chunks of 8 per lane.
hipError_t rmsnorm_fwd_launch(const lt_half* X, int64_t ldx, const lt_half* W, lt_half* Y,
                              int64_t ldy, float* RSTD, int64_t T, int64_t H, float eps,
                              hipStream_t s) {
  const int64_t k = (H / 8 + 63) / 64;
  if (k <= 4) return launch_rms_fwd<4>(X, ldx, W, Y, ldy, RSTD, T, H, eps, s);
  if (k <= 8) return launch_rms_fwd<8>(X, ldx, W, Y, ldy, RSTD, T, H, eps, s);
  return launch_rms_fwd<16>(X, ldx, W, Y, ldy, RSTD, T, H, eps, s);
}

hipError_t rmsnorm_bwd_launch(const RmsBwdArgs& a, hipStream_t s) {
  const int64_t k = (a.H / 8 + 63) / 64;
  if (k <= 4) return launch_rms_bwd<4, true>(a, s);
  if (k <= 8) return launch_rms_bwd<8, true>(a, s);
  if (k <= 12) return launch_rms_bwd<12, true>(a, s);
  return launch_rms_bwd<16, false>(a, s);
}

hipError_t rope_table_launch(float* CS, int S, int D, double base, hipStream_t s) {
  const int64_t n = (int64_t)S * (D / 2);
  hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, CS, S,
                     D, base);
  return hipGetLastError();
}

hipError_t rope_launch(lt_half* X, int64_t stride, int B, int S, int heads, int D, const float* CS,
                       int inverse, hipStream_t s) {
  const int64_t T = (int64_t)B * S;
  const int64_t n = T * heads * (D / 16);
  hipLaunchKernelGGL(rope_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, X, stride, T,
                     S, heads, D, CS, inverse ? -1.f : 1.f);
  return hipGetLastError();
}

}  // namespace lt
