// Bias gradient of a linear layer: db[n] = sum over rows t of dY[t][n].
//
// The Qwen2.5 QKV projection (Sec. 6.1's evaluated models) carries a bias
// that is broadcast over the T token rows, so its gradient is the column sum
// of the projection's output gradient.  HBM-bound: it reads 2*T*N bytes.
//
// Two passes, FP32 throughout and a fixed summation order (deterministic):
//   1. bias_grad_partial: workgroup (column tile of 512, row block); each
//      lane owns 8 columns (one 16-byte load per row), the 4 waves take every
//      4th row of the block, eight rows' loads in flight at a time, and the
//      waves' sums are combined in wave order through LDS into one FP32
//      partial row of the workspace;
//   2. bias_grad_sum: one thread per column adds the partial rows in order
//      (eight loads in flight at a time) and rounds once to FP16.

#include "common.hpp"
#include "kernels.hpp"

namespace lt {
namespace {

constexpr int kCols = 512;   // columns per workgroup (64 lanes x 8)
constexpr int kWaves = 4;
constexpr int kBatch = 8;    // rows per wave whose loads are in flight together

__global__ void __launch_bounds__(kWaves * 64)
bias_grad_partial_kernel(const lt_half* __restrict__ dY, int64_t lddy, int64_t T, int64_t N,
                         int64_t rows_per, float* __restrict__ part) {
  __shared__ float red[kWaves][kCols];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t c0 = (int64_t)blockIdx.x * kCols + lane * 8;
  const int64_t r0 = (int64_t)blockIdx.y * rows_per;
  const int64_t r1 = r0 + rows_per < T ? r0 + rows_per : T;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (c0 < N) {
    // kBatch rows' loads are issued together (rows past the block read as
    // zero from a clamped address), then added in row order: one memory
    // latency per batch instead of one per row
    for (int64_t rb = r0 + wave; rb < r1; rb += kWaves * kBatch) {
      half8 v[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int64_t r = rb + (int64_t)u * kWaves;
        v[u] = as_half8(ld16(dY + (r < r1 ? r : r0) * lddy + c0));
        if (r >= r1) v[u] = as_half8(u32x4{0, 0, 0, 0});
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += (float)v[u][e];
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[wave][lane * 8 + e] = acc[e];
  __syncthreads();
  for (int c = threadIdx.x; c < kCols; c += kWaves * 64) {
    const int64_t col = (int64_t)blockIdx.x * kCols + c;
    if (col < N) {
      float s = red[0][c];
#pragma unroll
      for (int w = 1; w < kWaves; ++w) s += red[w][c];
      part[(int64_t)blockIdx.y * N + col] = s;
    }
  }
}

__global__ void __launch_bounds__(256)
bias_grad_sum_kernel(const float* __restrict__ part, int nrb, int64_t N, lt_half* __restrict__ db) {
  const int64_t col = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (col >= N) return;
  // kBatch partial rows loaded together, added in row order
  float s = 0.f;
  for (int rb = 0; rb < nrb; rb += kBatch) {
    float v[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) v[u] = rb + u < nrb ? part[(int64_t)(rb + u) * N + col] : 0.f;
#pragma unroll
    for (int u = 0; u < kBatch; ++u) s += v[u];
  }
  reinterpret_cast<_Float16*>(db)[col] = (_Float16)s;
}

}  // namespace

hipError_t bias_grad_launch(const lt_half* dY, int64_t lddy, int64_t T, int64_t N, lt_half* db,
                            float* part, hipStream_t s) {
  const int nrb = bias_grad_blocks(T);
  const int64_t rows_per = (T + nrb - 1) / nrb;
  const dim3 g1((unsigned)((N + kCols - 1) / kCols), (unsigned)nrb);
  hipLaunchKernelGGL(bias_grad_partial_kernel, g1, dim3(kWaves * 64), 0, s, dY, lddy, T, N,
                     rows_per, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(bias_grad_sum_kernel, dim3((unsigned)((N + 255) / 256)), dim3(256), 0, s,
                     part, nrb, N, db);
  return hipGetLastError();
}

}  // namespace lt
