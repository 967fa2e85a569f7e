// Allocation-free GEMM entry point: lt_gemm_f16_ws with its split-K
// workspace taken from a file-scope device array instead of the caller.
//
// For callers that cannot allocate device memory (code under graph capture,
// serving loops or harnesses that forbid hipMalloc).  The array `scratch`
// holds kScratchBytes; every call on a GPU shares that GPU's copy, so calls
// that overlap on one GPU (different streams, no ordering between them)
// race on it.  The split-K partials are written in full before they are
// read within one call, so nothing needs clearing between calls.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <mutex>

#include "kernels.hpp"

namespace {

// The largest split-K workspace of the layer GEMMs of every evaluated model
// shape is 64 MiB (Baichuan2-13B and Qwen2.5-32B at 4096 tokens).
constexpr size_t kScratchBytes = LT_GEMM_NOALLOC_SCRATCH_BYTES;
static_assert(kScratchBytes % 256 == 0, "scratch size keeps 256-byte alignment");

// Device-side array: in host code its name stands for the symbol, not a
// device address; the address of each GPU's copy comes from
// hipGetSymbolAddress, once per device, and only that address is used.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch_ptr[kMaxDevices];   // per device ordinal: device address of `scratch`

// Device address of the current device's scratch array (resolved on the
// first call on that device).
lt_status scratch_for(lt_stream stream, void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return lt::set_error(LT_ERR_HIP, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return lt::set_error(LT_ERR_UNSUPPORTED, "device ordinal beyond the scratch table");
  if (stream != nullptr) {
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice(reinterpret_cast<hipStream_t>(stream), &sdev);
    if (e != hipSuccess) return lt::set_error(LT_ERR_HIP, hipGetErrorString(e));
    if (sdev != dev)
      return lt::set_error(LT_ERR_INVALID_ARG,
                           "stream belongs to another device than the current one");
  }
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return lt::set_error(LT_ERR_HIP, e != hipSuccess ? hipGetErrorString(e)
                                                       : "scratch symbol has no device address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return LT_OK;
}

}  // namespace

extern "C" lt_status lt_gemm_f16_noalloc(int transA, int transB, int64_t M, int64_t N, int64_t K,
                                         float alpha, const lt_half* A, int64_t lda,
                                         const lt_half* B, int64_t ldb, float beta,
                                         const lt_half* R, int64_t ldr, const lt_half* bias,
                                         lt_half* C, int64_t ldc, lt_stream stream) {
  const size_t need = lt_gemm_f16_workspace_size(transA, transB, M, N, K);
  if (need > kScratchBytes) {
    char msg[160];
    std::snprintf(msg, sizeof(msg),
                  "split-K partials of this shape need %zu bytes; the static scratch holds %zu",
                  need, kScratchBytes);
    return lt::set_error(LT_ERR_WORKSPACE, msg);
  }
  void* ws = nullptr;
  const lt_status st = scratch_for(stream, &ws);
  if (st != LT_OK) return st;
  return lt::gemm_checked(transA, transB, M, N, K, alpha, A, lda, B, ldb, beta, R, ldr, bias, C,
                          ldc, stream, ws, kScratchBytes);
}
