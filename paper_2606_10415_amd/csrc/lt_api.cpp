// C ABI of liblt: host-side argument validation and dispatch to the gfx950
// kernels.  Declarations and the full contract are in include/lt.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>

#include "kernels.hpp"

namespace {

thread_local std::string g_last_error;

lt_status fail(lt_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

lt_status ok() {
  g_last_error.clear();
  return LT_OK;
}

lt_status from_hip(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(LT_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// B * S * Hq rows of the [B, Hq, S] row terms above 2^31 (checked without overflow)
bool too_many_rows(int B, int S, int Hq) {
  return (int64_t)B * S > (((int64_t)1 << 31) / Hq);
}

// Row tiles of up to 256 rows are loaded by buffer instructions with 32-bit
// byte offsets: rows * stride * 2 bytes must stay below 2^31.
constexpr int64_t kMaxAttnStride = (int64_t)1 << 22;

lt_status check_attn_common(const void* Q, const void* K, const void* V, int64_t q_stride,
                            int64_t kv_stride, int B, int S, int Hq, int Hkv, int D, float scale,
                            int causal) {
  if (!Q || !K || !V) return fail(LT_ERR_INVALID_ARG, "NULL Q/K/V pointer");
  if (B < 1 || S < 1 || Hq < 1 || Hkv < 1 || D < 1)
    return fail(LT_ERR_INVALID_ARG, "B, S, Hq, Hkv, D must be >= 1 (got %d %d %d %d %d)", B, S, Hq,
                Hkv, D);
  if (Hq % Hkv != 0) return fail(LT_ERR_INVALID_ARG, "Hq (%d) must be a multiple of Hkv (%d)", Hq, Hkv);
  if (causal != 0 && causal != 1) return fail(LT_ERR_INVALID_ARG, "causal must be 0 or 1");
  if (!(scale > 0.f) || !std::isfinite(scale))
    return fail(LT_ERR_INVALID_ARG, "scale must be finite and > 0");
  if (q_stride < (int64_t)Hq * D)
    return fail(LT_ERR_INVALID_ARG, "q_row_stride %lld < Hq*D", (long long)q_stride);
  if (kv_stride < (int64_t)Hkv * D)
    return fail(LT_ERR_INVALID_ARG, "kv_row_stride %lld < Hkv*D", (long long)kv_stride);
  if (D != 64 && D != 128) return fail(LT_ERR_UNSUPPORTED, "head dim %d not in {64, 128}", D);
  if ((q_stride & 7) || (kv_stride & 7))
    return fail(LT_ERR_UNSUPPORTED, "row strides must be multiples of 8 elements");
  if (q_stride >= kMaxAttnStride || kv_stride >= kMaxAttnStride)
    return fail(LT_ERR_UNSUPPORTED, "q/kv row strides must be < 2^22 elements (32-bit buffer offsets)");
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V))
    return fail(LT_ERR_UNSUPPORTED, "Q/K/V must be 16-byte aligned");
  if (too_many_rows(B, S, Hq)) return fail(LT_ERR_UNSUPPORTED, "B*S*Hq too large");
  return LT_OK;
}

lt_status check_attn_bwd(const void* Q, const void* K, const void* V, int64_t q_row_stride,
                         int64_t kv_row_stride, const void* O, const void* dO, int64_t o_row_stride,
                         const float* LSE, const void* dQ, const void* dK, const void* dV,
                         int64_t dq_row_stride, int64_t dkv_row_stride, int B, int S, int Hq,
                         int Hkv, int D, float scale, int causal) {
  lt_status st = check_attn_common(Q, K, V, q_row_stride, kv_row_stride, B, S, Hq, Hkv, D, scale,
                                   causal);
  if (st != LT_OK) return st;
  if (!O || !dO || !LSE || !dQ || !dK || !dV)
    return fail(LT_ERR_INVALID_ARG, "NULL O/dO/LSE/dQ/dK/dV pointer");
  if (o_row_stride < (int64_t)Hq * D || dq_row_stride < (int64_t)Hq * D ||
      dkv_row_stride < (int64_t)Hkv * D)
    return fail(LT_ERR_INVALID_ARG, "o/dq/dkv row stride smaller than the row length");
  if ((o_row_stride | dq_row_stride | dkv_row_stride) & 7)
    return fail(LT_ERR_UNSUPPORTED, "row strides must be multiples of 8 elements");
  if (o_row_stride >= kMaxAttnStride || dq_row_stride >= kMaxAttnStride ||
      dkv_row_stride >= kMaxAttnStride)
    return fail(LT_ERR_UNSUPPORTED, "o/dq/dkv row strides must be < 2^22 elements");
  if (!aligned16(O) || !aligned16(dO) || !aligned16(dQ) || !aligned16(dK) || !aligned16(dV))
    return fail(LT_ERR_UNSUPPORTED, "O/dO/dQ/dK/dV must be 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(LSE) & 3u) return fail(LT_ERR_UNSUPPORTED, "LSE must be 4-byte aligned");
  return LT_OK;
}

}  // namespace

static lt_status gemm_common(int transA, int transB, int64_t M, int64_t N, int64_t K, float alpha,
                             const lt_half* A, int64_t lda, const lt_half* B, int64_t ldb,
                             float beta, const lt_half* R, int64_t ldr, const lt_half* bias,
                             lt_half* C, int64_t ldc, lt_stream stream,
                             void* workspace = nullptr, size_t ws_bytes = 0) {
  if ((transA != 0 && transA != 1) || (transB != 0 && transB != 1))
    return fail(LT_ERR_INVALID_ARG, "transA/transB must be 0 or 1");
  if (M < 0 || N < 0 || K < 0) return fail(LT_ERR_INVALID_ARG, "negative GEMM size");
  if (M == 0 || N == 0) return ok();
  if (!C) return fail(LT_ERR_INVALID_ARG, "NULL C");
  if (K > 0 && (!A || !B)) return fail(LT_ERR_INVALID_ARG, "NULL A or B");
  if (beta != 0.f && !R) return fail(LT_ERR_INVALID_ARG, "beta != 0 needs R");
  const int64_t a_row = transA ? M : K;
  const int64_t b_row = transB ? K : N;
  if (K > 0 && (lda < a_row || ldb < b_row))
    return fail(LT_ERR_INVALID_ARG, "lda/ldb smaller than the stored row length");
  if (ldc < N) return fail(LT_ERR_INVALID_ARG, "ldc %lld < N %lld", (long long)ldc, (long long)N);
  if (beta != 0.f && ldr < N) return fail(LT_ERR_INVALID_ARG, "ldr %lld < N %lld", (long long)ldr, (long long)N);
  if (((K > 0 ? (lda | ldb) : 0) | ldc | (beta != 0.f ? ldr : 0)) & 7)
    return fail(LT_ERR_UNSUPPORTED, "leading dimensions must be multiples of 8");
  if ((K > 0 && (!aligned16(A) || !aligned16(B))) || !aligned16(C) ||
      (beta != 0.f && !aligned16(R)))
    return fail(LT_ERR_UNSUPPORTED, "A, B, R, C must be 16-byte aligned");
  if (M > (int64_t)1 << 30 || N > (int64_t)1 << 30 || K > (int64_t)1 << 30)
    return fail(LT_ERR_UNSUPPORTED, "M, N or K too large for the tile grid");
  if (lda >= ((int64_t)1 << 22) || ldb >= ((int64_t)1 << 22))
    return fail(LT_ERR_UNSUPPORTED, "lda/ldb must be < 2^22 elements (32-bit buffer offsets)");
  if (bias && !aligned16(bias)) return fail(LT_ERR_UNSUPPORTED, "bias must be 16-byte aligned");
  if (workspace) {
    const size_t need = K > 0 ? lt::gemm_splitk_ws_bytes(M, N, K) : 0;
    if (ws_bytes < need) return fail(LT_ERR_WORKSPACE, "workspace needs %zu bytes", need);
    if (!aligned16(workspace)) return fail(LT_ERR_UNSUPPORTED, "workspace must be 16-byte aligned");
  }
  lt::GemmArgs g{transA, transB, M, N, K, alpha, beta, A, lda, B, ldb,
                 beta != 0.f ? R : C, beta != 0.f ? ldr : ldc, C, ldc};
  g.bias = bias;
  g.ws = static_cast<float*>(workspace);
  g.ws_bytes = workspace ? ws_bytes : 0;
  return from_hip(lt::gemm_f16_launch(g, reinterpret_cast<hipStream_t>(stream)), "gemm launch");
}

namespace lt {
lt_status gemm_checked(int transA, int transB, int64_t M, int64_t N, int64_t K, float alpha,
                       const lt_half* A, int64_t lda, const lt_half* B, int64_t ldb, float beta,
                       const lt_half* R, int64_t ldr, const lt_half* bias, lt_half* C, int64_t ldc,
                       lt_stream stream, void* workspace, size_t ws_bytes) {
  return gemm_common(transA, transB, M, N, K, alpha, A, lda, B, ldb, beta, R, ldr, bias, C, ldc,
                     stream, workspace, ws_bytes);
}
lt_status set_error(lt_status s, const char* msg) { return fail(s, "%s", msg); }
}  // namespace lt

extern "C" {

const char* lt_status_string(lt_status s) {
  switch (s) {
    case LT_OK: return "LT_OK";
    case LT_ERR_INVALID_ARG: return "LT_ERR_INVALID_ARG";
    case LT_ERR_UNSUPPORTED: return "LT_ERR_UNSUPPORTED";
    case LT_ERR_WORKSPACE: return "LT_ERR_WORKSPACE";
    case LT_ERR_HIP: return "LT_ERR_HIP";
  }
  return "LT_ERR_UNKNOWN";
}

const char* lt_last_error(void) { return g_last_error.c_str(); }

int lt_version(void) { return 100; }

lt_status lt_gemm_f16_res(int transA, int transB, int64_t M, int64_t N, int64_t K, float alpha,
                          const lt_half* A, int64_t lda, const lt_half* B, int64_t ldb, float beta,
                          const lt_half* R, int64_t ldr, lt_half* C, int64_t ldc,
                          lt_stream stream) {
  return gemm_common(transA, transB, M, N, K, alpha, A, lda, B, ldb, beta, R, ldr, nullptr, C,
                     ldc, stream);
}

lt_status lt_gemm_f16_bias(int transA, int transB, int64_t M, int64_t N, int64_t K, float alpha,
                           const lt_half* A, int64_t lda, const lt_half* B, int64_t ldb,
                           float beta, const lt_half* R, int64_t ldr, const lt_half* bias,
                           lt_half* C, int64_t ldc, lt_stream stream) {
  if (!bias && M > 0 && N > 0) return fail(LT_ERR_INVALID_ARG, "NULL bias");
  return gemm_common(transA, transB, M, N, K, alpha, A, lda, B, ldb, beta, R, ldr, bias, C, ldc,
                     stream);
}

size_t lt_gemm_f16_workspace_size(int transA, int transB, int64_t M, int64_t N, int64_t K) {
  if ((transA != 0 && transA != 1) || (transB != 0 && transB != 1)) return 0;
  if (M <= 0 || N <= 0 || K <= 0) return 0;
  return lt::gemm_splitk_ws_bytes(M, N, K);
}

lt_status lt_gemm_f16_ws(int transA, int transB, int64_t M, int64_t N, int64_t K, float alpha,
                         const lt_half* A, int64_t lda, const lt_half* B, int64_t ldb, float beta,
                         const lt_half* R, int64_t ldr, const lt_half* bias, lt_half* C,
                         int64_t ldc, void* workspace, size_t workspace_bytes, lt_stream stream) {
  return gemm_common(transA, transB, M, N, K, alpha, A, lda, B, ldb, beta, R, ldr, bias, C, ldc,
                     stream, workspace, workspace_bytes);
}

size_t lt_bias_grad_workspace_size(int64_t T, int64_t N) {
  if (T < 1 || N < 1 || N > ((int64_t)1 << 40)) return 0;
  return lt::bias_grad_ws_bytes(T, N);
}

lt_status lt_bias_grad_f16(const lt_half* dY, int64_t lddy, int64_t T, int64_t N, lt_half* db,
                           void* workspace, size_t ws_bytes, lt_stream stream) {
  if (T < 0 || N < 0) return fail(LT_ERR_INVALID_ARG, "negative size");
  if (N == 0) return ok();
  if (!db) return fail(LT_ERR_INVALID_ARG, "NULL db");
  if (T == 0) return fail(LT_ERR_INVALID_ARG, "T == 0: the bias gradient needs at least one row");
  if (!dY) return fail(LT_ERR_INVALID_ARG, "NULL dY");
  if (lddy < N) return fail(LT_ERR_INVALID_ARG, "lddy < N");
  if ((N & 7) || (lddy & 7)) return fail(LT_ERR_UNSUPPORTED, "N and lddy must be multiples of 8");
  if (!aligned16(dY)) return fail(LT_ERR_UNSUPPORTED, "dY must be 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(db) & 1u) return fail(LT_ERR_UNSUPPORTED, "db must be 2-byte aligned");
  if (!workspace || ws_bytes < lt::bias_grad_ws_bytes(T, N))
    return fail(LT_ERR_WORKSPACE, "workspace needs %zu bytes", lt::bias_grad_ws_bytes(T, N));
  if (reinterpret_cast<uintptr_t>(workspace) & 15u)
    return fail(LT_ERR_UNSUPPORTED, "workspace must be 16-byte aligned");
  return from_hip(lt::bias_grad_launch(dY, lddy, T, N, db, static_cast<float*>(workspace),
                                       reinterpret_cast<hipStream_t>(stream)),
                  "bias_grad launch");
}

lt_status lt_gemm_f16(int transA, int transB, int64_t M, int64_t N, int64_t K, float alpha,
                      const lt_half* A, int64_t lda, const lt_half* B, int64_t ldb, float beta,
                      lt_half* C, int64_t ldc, lt_stream stream) {
  return lt_gemm_f16_res(transA, transB, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc, C, ldc,
                         stream);
}

lt_status lt_attn_fwd(const lt_half* Q, const lt_half* K, const lt_half* V, int64_t q_row_stride,
                      int64_t kv_row_stride, lt_half* O, int64_t o_row_stride, float* LSE, int B,
                      int S, int Hq, int Hkv, int D, float scale, int causal, lt_stream stream) {
  lt_status st = check_attn_common(Q, K, V, q_row_stride, kv_row_stride, B, S, Hq, Hkv, D, scale,
                                   causal);
  if (st != LT_OK) return st;
  if (!O || !LSE) return fail(LT_ERR_INVALID_ARG, "NULL O or LSE");
  if (o_row_stride < (int64_t)Hq * D) return fail(LT_ERR_INVALID_ARG, "o_row_stride < Hq*D");
  if ((o_row_stride & 7) || !aligned16(O))
    return fail(LT_ERR_UNSUPPORTED, "O must be 16-byte aligned with stride % 8 == 0");
  if (o_row_stride >= kMaxAttnStride)
    return fail(LT_ERR_UNSUPPORTED, "o_row_stride must be < 2^22 elements");
  if (reinterpret_cast<uintptr_t>(LSE) & 3u) return fail(LT_ERR_UNSUPPORTED, "LSE must be 4-byte aligned");
  lt::AttnFwdArgs a{{B, S, Hq, Hkv, D, scale, causal}, Q, K, V, q_row_stride, kv_row_stride, O,
                    o_row_stride, LSE};
  return from_hip(lt::attn_fwd_launch(a, reinterpret_cast<hipStream_t>(stream)), "attn_fwd launch");
}

size_t lt_attn_bwd_workspace_size(int B, int S, int Hq, int Hkv, int D, int causal) {
  if (B < 1 || S < 1 || Hq < 1 || Hkv < 1 || D < 1 || Hq % Hkv || (causal != 0 && causal != 1))
    return 0;
  if (too_many_rows(B, S, Hq) || (D != 64 && D != 128)) return 0;   // lt_attn_bwd rejects these
  return lt::attn_bwd_delta_bytes(B, S, Hq) + lt::attn_bwd_lse2_bytes(B, S, Hq) +
         lt::attn_bwd_ds_bytes(B, S, Hq, causal) + lt::attn_bwd_part_bytes(B, S, Hq, Hkv, D);
}

lt_status lt_attn_bwd(const lt_half* Q, const lt_half* K, const lt_half* V, int64_t q_row_stride,
                      int64_t kv_row_stride, const lt_half* O, const lt_half* dO,
                      int64_t o_row_stride, const float* LSE, lt_half* dQ, lt_half* dK, lt_half* dV,
                      int64_t dq_row_stride, int64_t dkv_row_stride, void* workspace,
                      size_t ws_bytes, int B, int S, int Hq, int Hkv, int D, float scale,
                      int causal, lt_stream stream) {
  lt_status st = check_attn_bwd(Q, K, V, q_row_stride, kv_row_stride, O, dO, o_row_stride, LSE, dQ,
                                dK, dV, dq_row_stride, dkv_row_stride, B, S, Hq, Hkv, D, scale,
                                causal);
  if (st != LT_OK) return st;
  const size_t need = lt_attn_bwd_workspace_size(B, S, Hq, Hkv, D, causal);
  if (!workspace || ws_bytes < need)
    return fail(LT_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                workspace ? ws_bytes : (size_t)0);
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(LT_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  char* ws = static_cast<char*>(workspace);
  const size_t off_lse2 = lt::attn_bwd_delta_bytes(B, S, Hq);
  const size_t off_ds = off_lse2 + lt::attn_bwd_lse2_bytes(B, S, Hq);
  const size_t off_part = off_ds + lt::attn_bwd_ds_bytes(B, S, Hq, causal);
  lt::AttnBwdArgs a{{B, S, Hq, Hkv, D, scale, causal},
                    Q, K, V, q_row_stride, kv_row_stride, O, dO, o_row_stride, LSE, dQ, dK, dV,
                    dq_row_stride, dkv_row_stride,
                    reinterpret_cast<float*>(ws),
                    reinterpret_cast<float*>(ws + off_lse2),
                    reinterpret_cast<lt_half*>(ws + off_ds),
                    reinterpret_cast<float*>(ws + off_part),
                    0, 0};
  const lt::DkdvPlan plan = lt::attn_bwd_dkdv_plan(B, S, Hq, Hkv);
  a.nsplit = plan.nsplit;
  a.ktile = plan.ktile;
  return from_hip(lt::attn_bwd_launch(a, reinterpret_cast<hipStream_t>(stream)), "attn_bwd launch");
}

size_t lt_attn_p_size(int B, int S, int Hq, int causal) {
  if (B < 1 || S < 1 || Hq < 1 || (causal != 0 && causal != 1)) return 0;
  if (too_many_rows(B, S, Hq)) return 0;
  return lt::attn_bwd_ds_bytes(B, S, Hq, causal);
}

lt_status lt_attn_fwd_p(const lt_half* Q, const lt_half* K, const lt_half* V,
                        int64_t q_row_stride, int64_t kv_row_stride, lt_half* O,
                        int64_t o_row_stride, float* LSE, lt_half* P, size_t p_bytes, int B, int S,
                        int Hq, int Hkv, int D, float scale, int causal, lt_stream stream) {
  if (!P) return fail(LT_ERR_INVALID_ARG, "NULL P");
  lt_status st = lt_attn_fwd(Q, K, V, q_row_stride, kv_row_stride, O, o_row_stride, LSE, B, S, Hq,
                             Hkv, D, scale, causal, stream);
  if (st != LT_OK) return st;
  // lt_attn_fwd validated the shape; the P blocks follow it on the same stream
  const size_t need = lt_attn_p_size(B, S, Hq, causal);
  if (p_bytes < need)
    return fail(LT_ERR_WORKSPACE, "P buffer of %zu bytes needed, %zu given", need, p_bytes);
  if (!aligned16(P)) return fail(LT_ERR_UNSUPPORTED, "P must be 16-byte aligned");
  lt::AttnSavePArgs a{{B, S, Hq, Hkv, D, scale, causal}, Q, K, q_row_stride, kv_row_stride, LSE, P};
  return from_hip(lt::attn_save_p_launch(a, reinterpret_cast<hipStream_t>(stream)),
                  "attn_save_p launch");
}

size_t lt_attn_bwd_p_workspace_size(int B, int S, int Hq, int Hkv, int D) {
  if (B < 1 || S < 1 || Hq < 1 || Hkv < 1 || D < 1 || Hq % Hkv) return 0;
  if (too_many_rows(B, S, Hq) || (D != 64 && D != 128)) return 0;
  return lt::attn_bwd_delta_bytes(B, S, Hq) + lt::attn_bwd_lse2_bytes(B, S, Hq) +
         lt::attn_bwd_part_bytes(B, S, Hq, Hkv, D);
}

lt_status lt_attn_bwd_p(const lt_half* Q, const lt_half* K, const lt_half* V, int64_t q_row_stride,
                        int64_t kv_row_stride, const lt_half* O, const lt_half* dO,
                        int64_t o_row_stride, const float* LSE, const lt_half* P, size_t p_bytes,
                        lt_half* dQ, lt_half* dK, lt_half* dV, int64_t dq_row_stride,
                        int64_t dkv_row_stride, void* workspace, size_t ws_bytes, int B, int S,
                        int Hq, int Hkv, int D, float scale, int causal, lt_stream stream) {
  lt_status st = check_attn_bwd(Q, K, V, q_row_stride, kv_row_stride, O, dO, o_row_stride, LSE, dQ,
                                dK, dV, dq_row_stride, dkv_row_stride, B, S, Hq, Hkv, D, scale,
                                causal);
  if (st != LT_OK) return st;
  if (!P) return fail(LT_ERR_INVALID_ARG, "NULL P");
  const size_t pneed = lt_attn_p_size(B, S, Hq, causal);
  if (p_bytes < pneed)
    return fail(LT_ERR_INVALID_ARG, "P buffer of %zu bytes expected, %zu given", pneed, p_bytes);
  if (!aligned16(P)) return fail(LT_ERR_UNSUPPORTED, "P must be 16-byte aligned");
  const size_t need = lt_attn_bwd_p_workspace_size(B, S, Hq, Hkv, D);
  if (!workspace || ws_bytes < need)
    return fail(LT_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                workspace ? ws_bytes : (size_t)0);
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(LT_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  char* ws = static_cast<char*>(workspace);
  const size_t off_lse2 = lt::attn_bwd_delta_bytes(B, S, Hq);
  const size_t off_part = off_lse2 + lt::attn_bwd_lse2_bytes(B, S, Hq);
  lt::AttnBwdArgs a{{B, S, Hq, Hkv, D, scale, causal},
                    Q, K, V, q_row_stride, kv_row_stride, O, dO, o_row_stride, LSE, dQ, dK, dV,
                    dq_row_stride, dkv_row_stride,
                    reinterpret_cast<float*>(ws),
                    reinterpret_cast<float*>(ws + off_lse2),
                    nullptr,
                    reinterpret_cast<float*>(ws + off_part),
                    0, 0, P};
  const lt::DkdvPlan plan = lt::attn_bwd_dkdv_plan(B, S, Hq, Hkv);
  a.nsplit = plan.nsplit;
  a.ktile = plan.ktile;
  return from_hip(lt::attn_bwd_p_launch(a, reinterpret_cast<hipStream_t>(stream)),
                  "attn_bwd_p launch");
}

lt_status lt_gemm_gu_swiglu_f16(const lt_half* X, int64_t ldx, const lt_half* Wgu, int64_t ldw,
                                lt_half* GU, int64_t ldgu, lt_half* A, int64_t lda, int64_t T,
                                int64_t H, int64_t F, lt_stream stream) {
  if (T < 0 || H < 0 || F < 0) return fail(LT_ERR_INVALID_ARG, "negative size");
  if (T == 0 || F == 0) return ok();
  if (!X || !Wgu || !GU || !A) return fail(LT_ERR_INVALID_ARG, "NULL pointer");
  if (T > (int64_t)1 << 30 || F > (int64_t)1 << 29 || H > (int64_t)1 << 30)
    return fail(LT_ERR_UNSUPPORTED, "T, H or F too large for the tile grid");
  if (ldx < H || ldw < H || ldgu < 2 * F || lda < F)
    return fail(LT_ERR_INVALID_ARG, "row stride smaller than the row length");
  if ((T | H | F) & 7) return fail(LT_ERR_UNSUPPORTED, "T, H, F must be multiples of 8");
  if ((ldx | ldw | ldgu | lda) & 7)
    return fail(LT_ERR_UNSUPPORTED, "leading dimensions must be multiples of 8");
  if (!aligned16(X) || !aligned16(Wgu) || !aligned16(GU) || !aligned16(A))
    return fail(LT_ERR_UNSUPPORTED, "X, Wgu, GU, A must be 16-byte aligned");
  if (ldx >= ((int64_t)1 << 22) || ldw >= ((int64_t)1 << 22) || 2 * F * ldw >= ((int64_t)1 << 30) - 128)
    return fail(LT_ERR_UNSUPPORTED, "operands too large for 32-bit buffer offsets");
  lt::GemmArgs g{0, 1, T, 2 * F, H, 1.f, 0.f, X, ldx, Wgu, ldw, GU, ldgu, GU, ldgu};
  g.epi = 1;
  g.X1 = A;
  g.ldx1 = lda;
  g.F = F;
  return from_hip(lt::gemm_f16_launch(g, reinterpret_cast<hipStream_t>(stream)),
                  "gemm_gu_swiglu launch");
}

lt_status lt_gemm_swiglu_bwd_f16(const lt_half* dY, int64_t lddy, const lt_half* Wd, int64_t ldwd,
                                 const lt_half* GU, int64_t ldgu, lt_half* dGU, int64_t lddgu,
                                 int64_t T, int64_t H, int64_t F, lt_stream stream) {
  if (T < 0 || H < 0 || F < 0) return fail(LT_ERR_INVALID_ARG, "negative size");
  if (T == 0 || F == 0) return ok();
  if (!dY || !Wd || !GU || !dGU) return fail(LT_ERR_INVALID_ARG, "NULL pointer");
  if (T > (int64_t)1 << 30 || F > (int64_t)1 << 30 || H > (int64_t)1 << 30)
    return fail(LT_ERR_UNSUPPORTED, "T, H or F too large for the tile grid");
  if (lddy < H || ldwd < F || ldgu < 2 * F || lddgu < 2 * F)
    return fail(LT_ERR_INVALID_ARG, "row stride smaller than the row length");
  if ((T | H | F) & 7) return fail(LT_ERR_UNSUPPORTED, "T, H, F must be multiples of 8");
  if ((lddy | ldwd | ldgu | lddgu) & 7)
    return fail(LT_ERR_UNSUPPORTED, "leading dimensions must be multiples of 8");
  if (!aligned16(dY) || !aligned16(Wd) || !aligned16(GU) || !aligned16(dGU))
    return fail(LT_ERR_UNSUPPORTED, "dY, Wd, GU, dGU must be 16-byte aligned");
  if (lddy >= ((int64_t)1 << 22) || ldwd >= ((int64_t)1 << 22))
    return fail(LT_ERR_UNSUPPORTED, "lddy/ldwd must be < 2^22 elements (32-bit buffer offsets)");
  lt::GemmArgs g{0, 0, T, F, H, 1.f, 0.f, dY, lddy, Wd, ldwd, dGU, lddgu, dGU, lddgu};
  g.epi = 2;
  g.X1 = const_cast<lt_half*>(GU);
  g.ldx1 = ldgu;
  g.F = F;
  return from_hip(lt::gemm_f16_launch(g, reinterpret_cast<hipStream_t>(stream)),
                  "gemm_swiglu_bwd launch");
}

size_t lt_rmsnorm_bwd_workspace_size(int64_t T, int64_t H) {
  if (T < 1 || H < 1 || H > 8192) return 0;           // H above the supported row width

  return lt::rmsnorm_bwd_ws_bytes(T, H);
}

static lt_status check_rms(int64_t T, int64_t H, int64_t lds[], int n_ld, const void* ptrs[],
                           int n_ptr) {
  if (T < 0 || H < 1) return fail(LT_ERR_INVALID_ARG, "T < 0 or H < 1");
  for (int i = 0; i < n_ptr; ++i)
    if (!ptrs[i]) return fail(LT_ERR_INVALID_ARG, "NULL pointer");
  for (int i = 0; i < n_ld; ++i)
    if (lds[i] < H) return fail(LT_ERR_INVALID_ARG, "row stride smaller than H");
  if (H & 7 || H > 8192) return fail(LT_ERR_UNSUPPORTED, "H must be a multiple of 8 and <= 8192");
  for (int i = 0; i < n_ld; ++i)
    if (lds[i] & 7) return fail(LT_ERR_UNSUPPORTED, "row strides must be multiples of 8 elements");
  for (int i = 0; i < n_ptr; ++i)
    if (!aligned16(ptrs[i])) return fail(LT_ERR_UNSUPPORTED, "pointers must be 16-byte aligned");
  return LT_OK;
}

lt_status lt_rmsnorm_fwd(const lt_half* X, int64_t ldx, const lt_half* W, lt_half* Y, int64_t ldy,
                         float* RSTD, int64_t T, int64_t H, float eps, lt_stream stream) {
  int64_t lds[2] = {ldx, ldy};
  const void* ptrs[4] = {X, W, Y, RSTD};
  lt_status st = check_rms(T, H, lds, 2, ptrs, 4);
  if (st != LT_OK) return st;
  if (!(eps >= 0.f) || !std::isfinite(eps)) return fail(LT_ERR_INVALID_ARG, "eps must be finite and >= 0");
  if (T == 0) return ok();
  return from_hip(lt::rmsnorm_fwd_launch(X, ldx, W, Y, ldy, RSTD, T, H, eps,
                                         reinterpret_cast<hipStream_t>(stream)),
                  "rmsnorm_fwd launch");
}

lt_status lt_rmsnorm_bwd(const lt_half* dY, int64_t lddy, const lt_half* X, int64_t ldx,
                         const lt_half* W, const float* RSTD, const lt_half* R, int64_t ldr,
                         lt_half* dX, int64_t lddx, lt_half* dW, void* workspace, size_t ws_bytes,
                         int64_t T, int64_t H, lt_stream stream) {
  int64_t lds[4] = {lddy, ldx, lddx, R ? ldr : H};
  const void* ptrs[6] = {dY, X, W, RSTD, dX, dW};
  lt_status st = check_rms(T, H, lds, 4, ptrs, 6);
  if (st != LT_OK) return st;
  if (R && !aligned16(R)) return fail(LT_ERR_UNSUPPORTED, "R must be 16-byte aligned");
  if (T == 0) return fail(LT_ERR_INVALID_ARG, "T must be >= 1 (dW is a sum over rows)");
  const size_t need = lt_rmsnorm_bwd_workspace_size(T, H);
  if (!workspace || ws_bytes < need)
    return fail(LT_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                workspace ? ws_bytes : (size_t)0);
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(LT_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  lt::RmsBwdArgs a{dY, lddy, X, ldx, W, RSTD, R, ldr, dX, lddx, dW,
                   static_cast<float*>(workspace), T, H};
  return from_hip(lt::rmsnorm_bwd_launch(a, reinterpret_cast<hipStream_t>(stream)),
                  "rmsnorm_bwd launch");
}

lt_status lt_rope_table(float* CS, int S, int D, double base, lt_stream stream) {
  if (!CS) return fail(LT_ERR_INVALID_ARG, "NULL pointer");
  if (S < 1 || D < 2) return fail(LT_ERR_INVALID_ARG, "S < 1 or D < 2");
  if (!(base > 0.0) || !std::isfinite(base)) return fail(LT_ERR_INVALID_ARG, "base must be finite and > 0");
  if (D & 15) return fail(LT_ERR_UNSUPPORTED, "D must be a multiple of 16");
  if (!aligned16(CS)) return fail(LT_ERR_UNSUPPORTED, "CS must be 16-byte aligned");
  return from_hip(lt::rope_table_launch(CS, S, D, base, reinterpret_cast<hipStream_t>(stream)),
                  "rope_table launch");
}

lt_status lt_rope_f16(lt_half* X, int64_t row_stride, int B, int S, int heads, int D,
                      const float* CS, int inverse, lt_stream stream) {
  if (!X || !CS) return fail(LT_ERR_INVALID_ARG, "NULL pointer");
  if (B < 1 || S < 1 || heads < 1 || D < 2) return fail(LT_ERR_INVALID_ARG, "non-positive size");
  if (inverse != 0 && inverse != 1) return fail(LT_ERR_INVALID_ARG, "inverse must be 0 or 1");
  if (row_stride < (int64_t)heads * D) return fail(LT_ERR_INVALID_ARG, "row stride smaller than heads * D");
  if (D & 15) return fail(LT_ERR_UNSUPPORTED, "D must be a multiple of 16");
  if ((row_stride & 7) || !aligned16(X) || !aligned16(CS))
    return fail(LT_ERR_UNSUPPORTED, "X, CS must be 16-byte aligned and row_stride % 8 == 0");
  return from_hip(lt::rope_launch(X, row_stride, B, S, heads, D, CS, inverse,
                                  reinterpret_cast<hipStream_t>(stream)),
                  "rope launch");
}

lt_status lt_swiglu_fwd(const lt_half* GU, lt_half* A, int64_t T, int64_t F, lt_stream stream) {
  if (T < 0 || F < 0) return fail(LT_ERR_INVALID_ARG, "negative size");
  if (T == 0 || F == 0) return ok();
  if (!GU || !A) return fail(LT_ERR_INVALID_ARG, "NULL pointer");
  if (F & 7) return fail(LT_ERR_UNSUPPORTED, "F must be a multiple of 8");
  if (!aligned16(GU) || !aligned16(A)) return fail(LT_ERR_UNSUPPORTED, "pointers must be 16-byte aligned");
  return from_hip(lt::swiglu_fwd_launch(GU, A, T, F, reinterpret_cast<hipStream_t>(stream)),
                  "swiglu_fwd launch");
}

lt_status lt_swiglu_bwd(const lt_half* dA, const lt_half* GU, lt_half* dGU, int64_t T, int64_t F,
                        lt_stream stream) {
  if (T < 0 || F < 0) return fail(LT_ERR_INVALID_ARG, "negative size");
  if (T == 0 || F == 0) return ok();
  if (!dA || !GU || !dGU) return fail(LT_ERR_INVALID_ARG, "NULL pointer");
  if (F & 7) return fail(LT_ERR_UNSUPPORTED, "F must be a multiple of 8");
  if (!aligned16(dA) || !aligned16(GU) || !aligned16(dGU))
    return fail(LT_ERR_UNSUPPORTED, "pointers must be 16-byte aligned");
  return from_hip(lt::swiglu_bwd_launch(dA, GU, dGU, T, F, reinterpret_cast<hipStream_t>(stream)),
                  "swiglu_bwd launch");
}

}  // extern "C"
