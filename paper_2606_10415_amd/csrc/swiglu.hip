// SwiGLU gate between the FFN gate/up projection and the down projection.
//
// Elementwise and HBM-bound: each thread moves 16-byte vectors (8 halves),
// consecutive threads touch consecutive 16-byte chunks of a row, and the
// grid is sized to a few waves per CU with a grid-stride loop.
//   forward : A = silu(G) * U
//   backward: dG = dA * U * s * (1 + G (1 - s)),  dU = dA * silu(G),  s = sigmoid(G)
// Math in fp32, one RNE rounding per output.
#include "common.hpp"
#include "kernels.hpp"

namespace lt {
namespace {

__device__ __forceinline__ float sigmoid_f(float x) {
  // 1 / (1 + e^-x); e^-x overflows to +inf for x < ~-88 and the quotient is 0.
  return 1.f / (1.f + __expf(-x));
}

__global__ void __launch_bounds__(256)
swiglu_fwd_kernel(const lt_half* __restrict__ GU, lt_half* __restrict__ A, int64_t T, int64_t F) {
  const int64_t fc = F / 8;
  const int64_t total = T * fc;
  for (int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; id < total;
       id += (int64_t)gridDim.x * blockDim.x) {
    const int64_t t = id / fc;
    const int64_t c = (id - t * fc) * 8;
    const half8 g = as_half8(ld16(GU + t * 2 * F + c));
    const half8 u = as_half8(ld16(GU + t * 2 * F + F + c));
    half8 a;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float x = (float)g[e];
      a[e] = (_Float16)(x * sigmoid_f(x) * (float)u[e]);
    }
    st16(A + t * F + c, as_u32x4(a));
  }
}

__global__ void __launch_bounds__(256)
swiglu_bwd_kernel(const lt_half* __restrict__ dA, const lt_half* __restrict__ GU,
                  lt_half* __restrict__ dGU, int64_t T, int64_t F) {
  const int64_t fc = F / 8;
  const int64_t total = T * fc;
  for (int64_t id = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; id < total;
       id += (int64_t)gridDim.x * blockDim.x) {
    const int64_t t = id / fc;
    const int64_t c = (id - t * fc) * 8;
    const half8 g = as_half8(ld16(GU + t * 2 * F + c));
    const half8 u = as_half8(ld16(GU + t * 2 * F + F + c));
    const half8 da = as_half8(ld16(dA + t * F + c));
    half8 dg, du;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float x = (float)g[e];
      const float s = sigmoid_f(x);
      const float d = (float)da[e];
      du[e] = (_Float16)(d * x * s);
      dg[e] = (_Float16)(d * (float)u[e] * s * (1.f + x * (1.f - s)));
    }
    st16(dGU + t * 2 * F + c, as_u32x4(dg));
    st16(dGU + t * 2 * F + F + c, as_u32x4(du));
  }
}

int grid_for(int64_t chunks) {
  const int64_t blocks = (chunks + 255) / 256;
  const int64_t cap = 256 * 8;   // 8 workgroups per CU, then grid-stride
  return (int)(blocks < cap ? (blocks > 0 ? blocks : 1) : cap);
}

}  // namespace

hipError_t swiglu_fwd_launch(const lt_half* GU, lt_half* A, int64_t T, int64_t F, hipStream_t s) {
  hipLaunchKernelGGL(swiglu_fwd_kernel, dim3(grid_for(T * (F / 8))), dim3(256), 0, s, GU, A, T, F);
  return hipGetLastError();
}

hipError_t swiglu_bwd_launch(const lt_half* dA, const lt_half* GU, lt_half* dGU, int64_t T,
                             int64_t F, hipStream_t s) {
  hipLaunchKernelGGL(swiglu_bwd_kernel, dim3(grid_for(T * (F / 8))), dim3(256), 0, s, dA, GU, dGU,
                     T, F);
  return hipGetLastError();
}

}  // namespace lt
