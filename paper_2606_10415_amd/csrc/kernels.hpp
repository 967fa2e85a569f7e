// Internal launcher interface between the C ABI layer (lt_api.cpp) and the
// kernel translation units.  Arguments are validated before these are called.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/lt.h"

namespace lt {

struct GemmArgs {
  int transA, transB;
  int64_t M, N, K;
  float alpha, beta;
  const lt_half* A;
  int64_t lda;
  const lt_half* B;
  int64_t ldb;
  const lt_half* R;   // residual / accumulation input (may equal C)
  int64_t ldr;
  lt_half* C;
  int64_t ldc;
  // fused SwiGLU epilogues (0: none)
  //   1: B = Wgu [2F, K] (gate rows, then up rows), C = GU [M, 2F]; each tile
  //      pairs gate and up columns and also writes X1 = A = silu(G) * U [M, F]
  //   2: C = dGU [M, 2F] from dA = op(A) op(B) [M, F = N] and X1 = GU [M, 2F]
  int epi = 0;
  lt_half* X1 = nullptr;
  int64_t ldx1 = 0;
  int64_t F = 0;
  // optional bias [N] added to every row (epilogue 0 only)
  const lt_half* bias = nullptr;
  // gate/up epilogues: distance between gate and up rows of B (1) / columns
  // of C and X1 (1, 2); 0 means F (set for launches over part of the columns)
  int64_t pair_off = 0;
  // optional FP32 workspace (epilogue 0): a last wave at most half full then
  // runs with its K split (gemm_splitk_tail), when ws_bytes suffices
  float* ws = nullptr;
  size_t ws_bytes = 0;
};

// Split-K plan for the last, at most half full, wave of 256x256 tiles: the
// tiles right of column split_at (columns) or below row split_at (rows), an
// Mt x Nt region, computed as S partial products over K.  False: no split.
struct SplitTail {
  bool columns;
  int64_t split_at;
  int64_t Mt, Nt;
  int S;
};
bool gemm_splitk_tail(int64_t M, int64_t N, int64_t K, SplitTail* p);
// FP32 workspace bytes the split needs (0 when gemm_splitk_tail is false)
size_t gemm_splitk_ws_bytes(int64_t M, int64_t N, int64_t K);

struct AttnShape {
  int B, S, Hq, Hkv, D;
  float scale;
  int causal;
};

struct AttnFwdArgs {
  AttnShape sh;
  const lt_half* Q;
  const lt_half* K;
  const lt_half* V;
  int64_t q_stride, kv_stride;
  lt_half* O;
  int64_t o_stride;
  float* LSE;
};

struct AttnBwdArgs {
  AttnShape sh;
  const lt_half* Q;
  const lt_half* K;
  const lt_half* V;
  int64_t q_stride, kv_stride;
  const lt_half* O;
  const lt_half* dO;
  int64_t o_stride;
  const float* LSE;
  lt_half* dQ;
  lt_half* dK;
  lt_half* dV;
  int64_t dq_stride, dkv_stride;
  float* delta;   // workspace: [B, Hq, S]  rowsum(dO * O)
  float* lse2;    // workspace: [B, Hq, S]  LSE * log2(e)
  lt_half* ds;    // workspace: dS blocks [B, Hq, n_blocks(S, causal)][64 lanes][16] FP16
  float* part;    // workspace: [2][nsplit][B, S, Hkv, D] partial dK, dV (nsplit > 1 only)
  int nsplit;     // shares of each key tile's work in the dK/dV pass
  int ktile;      // keys per dK/dV workgroup (256 or 128)
  const lt_half* psaved = nullptr;   // saved P blocks (saved-P backward only)
};

// Saved P (written after the forward, read by the saved-P backward): the
// dS block layout (attn_bwd_ds_blocks) holding P instead of dS.
struct AttnSavePArgs {
  AttnShape sh;
  const lt_half* Q;
  const lt_half* K;
  int64_t q_stride, kv_stride;
  const float* LSE;
  lt_half* P;
};

// Workspace layout of the attention backward (offsets in bytes).
inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
inline size_t attn_bwd_delta_bytes(int B, int S, int Hq) {
  return align256((size_t)B * Hq * S * sizeof(float));
}
inline size_t attn_bwd_lse2_bytes(int B, int S, int Hq) { return attn_bwd_delta_bytes(B, S, Hq); }
// dS of every (32-key group, 32-query group) pair the mask keeps, as the
// dK/dV pass holds it in registers: one 2 KiB block per pair, lane l's 16
// FP16 values (key l % 32; queries 8 (j / 4) + 4 (l / 32) + j % 4, j = 0..15)
// at bytes 32 l.  Blocks of a head are query-major: under the causal mask
// query group qg holds key groups 0..qg, at qg (qg + 1) / 2 + kg; otherwise
// qg * n32 + kg.  The dQ pass streams a query group's blocks in order.
constexpr int kDsBlockBytes = 2048;
inline int64_t attn_bwd_ds_blocks(int S, int causal) {   // per (batch, query head)
  const int64_t n32 = ((int64_t)S + 31) / 32;
  return causal ? n32 * (n32 + 1) / 2 : n32 * n32;
}
inline size_t attn_bwd_ds_bytes(int B, int S, int Hq, int causal) {
  return align256((size_t)B * Hq * (size_t)attn_bwd_ds_blocks(S, causal) * kDsBlockBytes);
}
// The dK/dV pass runs one workgroup per (key tile, batch, kv head, share),
// one workgroup per CU.  Key tiles hold 256 keys (8 waves of 32), except
// for MHA (Hq = Hkv) when those give fewer than 512 workgroups: then 128
// keys, waves w and w + 4 owning the same 32 keys and taking the two
// 32-query halves of every 64-query block.  (With grouped queries the 256-key
// tile's shares of whole query heads measured faster.)
// A key tile's work is the (query head, 64-query block) pairs of its group;
// when the tiles alone give fewer than 512 workgroups it is split into n
// contiguous shares, each writing FP32 partial sums:
//   * the smallest divisor n of Hq/Hkv that gives >= 512 workgroups (shares
//     of whole query heads), if there is one;
//   * otherwise n = min(max(Hq/Hkv, ceil(256 / tiles)), 16, the pairs of
//     the last key tile, which has the fewest) -- e.g. a short causal MHA
//     sequence.
constexpr int64_t kDkdvFillWgs = 256;   // fallback split target: one workgroup per CU
struct DkdvPlan {
  int ktile;    // keys per workgroup: 256 or 128
  int nsplit;   // shares of each key tile's work
};
inline DkdvPlan attn_bwd_dkdv_plan(int B, int S, int Hq, int Hkv) {
  const int grp = Hq / Hkv;
  const int64_t S64 = S;
  const int ktile = grp > 1 || ((S64 + 255) / 256) * B * Hkv >= 512 ? 256 : 128;
  const int64_t n_kt = (S64 + ktile - 1) / ktile;
  const int64_t wgs = n_kt * B * Hkv;
  if (wgs >= 512) return {ktile, 1};
  for (int n = 2; n <= grp; ++n)
    if (grp % n == 0 && wgs * n >= 512) return {ktile, n};
  const int64_t n_qb = (S64 + 63) / 64;
  const int64_t last_pairs = (int64_t)grp * (n_qb - (n_kt - 1) * (ktile / 64));
  int64_t n = (kDkdvFillWgs + wgs - 1) / wgs;
  if (n < grp) n = grp;                                  // at least one share per query head
  if (n > 16) n = 16;
  if (n > last_pairs) n = last_pairs;
  return {ktile, n < 1 ? 1 : (int)n};
}
inline size_t attn_bwd_part_bytes(int B, int S, int Hq, int Hkv, int D) {
  const int n = attn_bwd_dkdv_plan(B, S, Hq, Hkv).nsplit;
  return n > 1 ? align256((size_t)2 * n * B * S * Hkv * D * sizeof(float)) : 0;
}

// RMSNorm backward (norm_rope.hip).  dW partial sums: one FP32 row of H per
// workgroup (4 waves), rmsnorm_bwd_blocks(T) workgroups.
struct RmsBwdArgs {
  const lt_half* dY;
  int64_t lddy;
  const lt_half* X;
  int64_t ldx;
  const lt_half* W;
  const float* RSTD;
  const lt_half* R;      // optional residual added to dX (may be null)
  int64_t ldr;
  lt_half* dX;
  int64_t lddx;
  lt_half* dW;
  float* part;           // workspace
  int64_t T, H;
};
constexpr int kRmsBwdWaves = 4;
// One row per wave up to 2048 rows, then at most 512 workgroups (two rows per
// wave at T = 4096): a wave's second row loads while other waves store their
// first, and the dW pass has half the partial rows of one row per wave.
inline int rmsnorm_bwd_blocks(int64_t T) {
  const int64_t b = T / kRmsBwdWaves + (T % kRmsBwdWaves != 0);   // no overflow at any T
  return (int)(b < 512 ? (b < 1 ? 1 : b) : 512);
}
inline size_t rmsnorm_bwd_ws_bytes(int64_t T, int64_t H) {
  return align256((size_t)rmsnorm_bwd_blocks(T) * H * sizeof(float));
}

// bias gradient (column sum): FP32 partial rows of the workspace
inline int bias_grad_blocks(int64_t T) {
  const int64_t b = T / 64 + (T % 64 != 0);
  return (int)(b < 128 ? (b < 1 ? 1 : b) : 128);
}
inline size_t bias_grad_ws_bytes(int64_t T, int64_t N) {
  return align256((size_t)bias_grad_blocks(T) * (size_t)N * sizeof(float));
}

// lt_api.cpp: the argument checks and dispatch behind the GEMM entry points
// (also used by the allocation-free entry point), and the calling thread's
// error message.
lt_status gemm_checked(int transA, int transB, int64_t M, int64_t N, int64_t K, float alpha,
                       const lt_half* A, int64_t lda, const lt_half* B, int64_t ldb, float beta,
                       const lt_half* R, int64_t ldr, const lt_half* bias, lt_half* C, int64_t ldc,
                       lt_stream stream, void* workspace, size_t ws_bytes);
lt_status set_error(lt_status s, const char* msg);

hipError_t gemm_f16_launch(const GemmArgs& a, hipStream_t s);
hipError_t bias_grad_launch(const lt_half* dY, int64_t lddy, int64_t T, int64_t N, lt_half* db,
                            float* part, hipStream_t s);
hipError_t attn_fwd_launch(const AttnFwdArgs& a, hipStream_t s);
hipError_t attn_bwd_launch(const AttnBwdArgs& a, hipStream_t s);
hipError_t attn_save_p_launch(const AttnSavePArgs& a, hipStream_t s);
hipError_t attn_bwd_p_launch(const AttnBwdArgs& a, hipStream_t s);
hipError_t rmsnorm_fwd_launch(const lt_half* X, int64_t ldx, const lt_half* W, lt_half* Y,
                              int64_t ldy, float* RSTD, int64_t T, int64_t H, float eps,
                              hipStream_t s);
hipError_t rmsnorm_bwd_launch(const RmsBwdArgs& a, hipStream_t s);
hipError_t rope_table_launch(float* CS, int S, int D, double base, hipStream_t s);
hipError_t rope_launch(lt_half* X, int64_t stride, int B, int S, int heads, int D, const float* CS,
                       int inverse, hipStream_t s);
hipError_t swiglu_fwd_launch(const lt_half* GU, lt_half* A, int64_t T, int64_t F, hipStream_t s);
hipError_t swiglu_bwd_launch(const lt_half* dA, const lt_half* GU, lt_half* dGU, int64_t T,
                             int64_t F, hipStream_t s);

}  // namespace lt
