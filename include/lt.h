/*
 * lt.h -- C ABI of the MI355X (gfx950) decoder-layer training kernels.
 *
 * The operations are the training-critical-path compute of one dense
 * decoder layer as described in Sec. 4.1 of the paper: the FP16 GEMM
 * primitive used by the QKV, output and FFN projections (forward, data
 * gradient and weight gradient), causal multi-head / grouped-query
 * attention forward, and the attention backward of Algorithm 1 (computed
 * here with recomputed probabilities from a saved per-row log-sum-exp),
 * plus the SwiGLU gate that joins the two FFN projections.
 *
 * General conventions
 *   - lt_half is the bit pattern of an IEEE-754 binary16 value.
 *   - All matrices are row-major.  "ld" / "row_stride" arguments are in
 *     elements, not bytes.
 *   - Every pointer argument named as a tensor is a DEVICE pointer that the
 *     caller allocated and owns (typically a PyTorch CUDA/HIP tensor).  The
 *     library allocates no device memory and keeps no state besides the
 *     loaded code objects; it is re-entrant and may be called concurrently
 *     on different streams.
 *   - Every call is asynchronous on `stream` (NULL = the default stream).
 *     Argument checks run on the host before any launch; a non-LT_OK return
 *     means nothing was launched, except LT_ERR_HIP (a launch failed).
 *   - Calls only launch kernels on `stream`: no allocation, memset, copy or
 *     synchronisation, so a sequence of calls may be captured into a HIP
 *     graph and replayed (the buffers, workspaces included, must then stay
 *     allocated for the graph's lifetime).
 *   - Inputs must not alias outputs (the GEMM's C is both).
 *   - Float16 outputs are rounded once, round-to-nearest-even, from the
 *     FP32 accumulator; FP16 subnormals are kept.
 *   - Fast-path alignment: every half pointer must be 16-byte aligned and
 *     every leading dimension / row stride a multiple of 8 elements.
 *     Otherwise the call returns LT_ERR_UNSUPPORTED (it never computes a
 *     wrong result).  The plain GEMMs take any M, N, K; the fused entry
 *     points state their own size rules.
 */
#ifndef LT_H_
#define LT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t lt_half;
typedef struct ihipStream_t* lt_stream;

typedef enum {
  LT_OK = 0,
  LT_ERR_INVALID_ARG = 1,  /* NULL pointer, negative size, ld too small, ... */
  LT_ERR_UNSUPPORTED = 2,  /* valid arguments outside what the kernels handle */
  LT_ERR_WORKSPACE = 3,    /* workspace missing or smaller than required */
  LT_ERR_HIP = 4           /* a HIP launch or runtime call failed */
} lt_status;

/* Static description of a status code (never NULL). */
const char* lt_status_string(lt_status s);

/* Human-readable detail of the last non-LT_OK return on the calling host
 * thread ("" if none).  The pointer stays valid until the next lt_* call on
 * this thread. */
const char* lt_last_error(void);

/* Library version as MAJOR*10000 + MINOR*100 + PATCH. */
int lt_version(void);

/*
 * GEMM update (Sec. 4.1, FP16 GEMM backend; the output tile is loaded as the
 * accumulation buffer):
 *
 *     C[M,N] = alpha * op(A)[M,K] * op(B)[K,N] + beta * C[M,N]
 *
 *   op(X) = X for trans == 0, X^T for trans == 1.
 *   A is stored [M, K] (transA = 0, lda >= K) or [K, M] (transA = 1, lda >= M).
 *   B is stored [K, N] (transB = 0, ldb >= N) or [N, K] (transB = 1, ldb >= K).
 *   C is stored [M, N], ldc >= N.
 *   FP32 accumulation, one RNE rounding to FP16 per output element.
 *   beta == 0 never reads C (NaN / uninitialised C is fine).
 *   M == 0 or N == 0: no-op.  K == 0: C = beta * C.
 *   Layer usage with nn.Linear weights W[out, in]:
 *     forward  Y  = X  W^T  -> (transA, transB) = (0, 1)
 *     dgrad    dX = dY W    -> (0, 0)
 *     wgrad    dW = dY^T X  -> (1, 0)   (beta = 1 accumulates micro-batches)
 *   Tails: any M, N, K.  Operand rows are read in whole 8-element (16-byte)
 *   chunks, so each stored row of A, B (and R below) must be readable up to
 *   its length rounded up to a multiple of 8 -- within its leading
 *   dimension, so true of any buffer that spans whole leading dimensions;
 *   elements past the row length never reach a stored result.  C is written
 *   only inside its M x N part.
 *   Errors: LT_ERR_INVALID_ARG for NULL A/B/C (C may be NULL only if M or N
 *   is 0), negative sizes, trans not 0/1, ld smaller than the row length;
 *   LT_ERR_UNSUPPORTED for an ld not a multiple of 8, a pointer not 16-byte
 *   aligned, M, N or K > 2^30, or lda / ldb >= 2^22 elements.
 */
lt_status lt_gemm_f16(int transA, int transB, int64_t M, int64_t N, int64_t K,
                      float alpha, const lt_half* A, int64_t lda,
                      const lt_half* B, int64_t ldb, float beta, lt_half* C,
                      int64_t ldc, lt_stream stream);

/*
 * GEMM with a separate accumulation input (Sec. 4.1's accumulation buffer
 * read from one place and written to another, e.g. a residual add):
 *
 *     C[M,N] = alpha * op(A) op(B) + beta * R[M,N]
 *
 *   Same conventions and errors as lt_gemm_f16; R is stored [M, N] with
 *   ldr >= N and is read only when beta != 0 (then R must not be NULL).
 *   R may be the same buffer as C (with ldr == ldc; this is lt_gemm_f16) but
 *   must not partially overlap it.  Layer usage: H1 = X + O Wo^T with
 *   R = X, C = H1.
 */
lt_status lt_gemm_f16_res(int transA, int transB, int64_t M, int64_t N,
                          int64_t K, float alpha, const lt_half* A,
                          int64_t lda, const lt_half* B, int64_t ldb,
                          float beta, const lt_half* R, int64_t ldr,
                          lt_half* C, int64_t ldc, lt_stream stream);

/*
 * GEMM with a bias broadcast over the rows (the biased linear layers of the
 * evaluated Qwen2.5 models, Sec. 6.1: its QKV projection):
 *
 *     C[M,N] = alpha * op(A) op(B) + beta * R[M,N] + bias[N]
 *
 *   Same conventions and errors as lt_gemm_f16_res; bias is [N] FP16, read
 *   by every row, 16-byte aligned (else LT_ERR_UNSUPPORTED), never NULL
 *   (LT_ERR_INVALID_ARG).  The bias is added in FP32 before the single
 *   rounding of C.
 */
lt_status lt_gemm_f16_bias(int transA, int transB, int64_t M, int64_t N,
                           int64_t K, float alpha, const lt_half* A,
                           int64_t lda, const lt_half* B, int64_t ldb,
                           float beta, const lt_half* R, int64_t ldr,
                           const lt_half* bias, lt_half* C, int64_t ldc,
                           lt_stream stream);

/*
 * GEMM with residual, optional bias and a caller-owned workspace (Sec. 4.1's
 * GEMM primitive, as lt_gemm_f16_bias with bias optional):
 *
 *     C[M,N] = alpha * op(A) op(B) + beta * R[M,N] (+ bias[N])
 *
 *   Same conventions and errors as lt_gemm_f16_res; bias may be NULL (no
 *   bias), else [N] FP16, 16-byte aligned.  The workspace lets the kernel
 *   split the reduction (K) of output tiles over several workgroups: the
 *   tiles of a last, at most half full, wave of 256x256 tiles, or all tiles
 *   of a launch of less than about one wave when the split gives 8 shares or
 *   keeps at least 2048 of K per share.  Their FP32 partial sums go to the
 *   workspace and are added in a fixed order (deterministic) before the
 *   single rounding of C.  The result can differ from lt_gemm_f16_res in the
 *   last bits of those tiles (another FP32 summation order).  There is no
 *   split (workspace size 0) when N or K is not a multiple of 8.
 *   workspace: device memory owned by the caller, 16-byte aligned (else
 *   LT_ERR_UNSUPPORTED), of at least lt_gemm_f16_workspace_size(...) bytes
 *   (else LT_ERR_WORKSPACE); its contents on entry do not matter and it is
 *   in use until the stream reaches the end of the call.  NULL: no split
 *   (the call is then lt_gemm_f16_res / lt_gemm_f16_bias).  Calls that may
 *   run concurrently need separate workspaces.
 */
size_t lt_gemm_f16_workspace_size(int transA, int transB, int64_t M, int64_t N,
                                  int64_t K);
lt_status lt_gemm_f16_ws(int transA, int transB, int64_t M, int64_t N,
                         int64_t K, float alpha, const lt_half* A, int64_t lda,
                         const lt_half* B, int64_t ldb, float beta,
                         const lt_half* R, int64_t ldr, const lt_half* bias,
                         lt_half* C, int64_t ldc, void* workspace,
                         size_t workspace_bytes, lt_stream stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops, harnesses that forbid hipMalloc): lt_gemm_f16_ws
 * with its split-K workspace taken from a static device array of
 * LT_GEMM_NOALLOC_SCRATCH_BYTES per GPU, held until the process ends, instead
 * of a caller buffer.  Same product, same split and the same bits as
 * lt_gemm_f16_ws with a sufficient workspace.  The call allocates nothing;
 * its first call on a device looks up that device's array (once).  The
 * current device must be the device of `stream` (else LT_ERR_INVALID_ARG).
 * 64 MiB is what the largest split of any shape needs (a split covers at
 * most 256 partial 256x256 FP32 tiles); a shape needing more
 * (lt_gemm_f16_workspace_size) would be rejected with LT_ERR_WORKSPACE.  Every
 * call on a GPU shares that GPU's array: calls that may overlap on one GPU
 * (unordered streams) race and must not be issued.  Other errors as
 * lt_gemm_f16_ws.
 */
#define LT_GEMM_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
lt_status lt_gemm_f16_noalloc(int transA, int transB, int64_t M, int64_t N,
                              int64_t K, float alpha, const lt_half* A,
                              int64_t lda, const lt_half* B, int64_t ldb,
                              float beta, const lt_half* R, int64_t ldr,
                              const lt_half* bias, lt_half* C, int64_t ldc,
                              lt_stream stream);

/*
 * Bias gradient of a linear layer: db[n] = sum over t < T of dY[t][n]
 * (dY row-major [T, N] with row stride lddy).  FP32 sums in a fixed order
 * (deterministic), one rounding to FP16.  The caller-owned workspace, of at
 * least lt_bias_grad_workspace_size(T, N) bytes (16-byte aligned), holds FP32
 * partial sums.  Errors: T == 0 or NULL pointers -> LT_ERR_INVALID_ARG
 * (N == 0 is a no-op); N or lddy not a multiple of 8, dY not 16-byte
 * aligned -> LT_ERR_UNSUPPORTED; workspace too small -> LT_ERR_WORKSPACE.
 */
size_t lt_bias_grad_workspace_size(int64_t T, int64_t N);
lt_status lt_bias_grad_f16(const lt_half* dY, int64_t lddy, int64_t T, int64_t N,
                           lt_half* db, void* workspace, size_t ws_bytes,
                           lt_stream stream);

/*
 * Attention forward (the forward whose probabilities Algorithm 1 consumes;
 * Sec. 4.1).  Per batch b and query head h, with key/value head
 * kv = h / (Hq / Hkv) (contiguous GQA grouping):
 *
 *     s_ij   = scale * q_i . k_j           (j <= i when causal)
 *     P      = row softmax of s
 *     O_i    = sum_j P_ij v_j
 *     LSE_i  = ln sum_j exp(s_ij)          (natural log, FP32)
 *
 *   Element (b, i, h, c) of Q is Q[(b*S + i) * q_row_stride + h*D + c];
 *   K and V likewise with kv_row_stride and kv heads; O with o_row_stride.
 *   So Q, K, V may be column slices of one fused QKV projection output
 *   [B*S, (Hq + 2 Hkv) D] (K = QKV + Hq*D, V = QKV + (Hq+Hkv)*D).
 *   LSE is a dense FP32 array [B, Hq, S].  Queries and keys have the same
 *   length S; causal masking is top-left aligned (query i sees keys 0..i).
 *   Errors: INVALID_ARG for NULL pointers, B/S/Hq/Hkv < 1, Hq % Hkv != 0,
 *   causal not 0/1, scale not finite and > 0, strides smaller than the row
 *   length;
 *   UNSUPPORTED for D not in {64, 128}, misaligned pointers or strides, or a
 *   row stride of 2^22 elements or more (tiles are loaded with 32-bit byte
 *   offsets).
 */
lt_status lt_attn_fwd(const lt_half* Q, const lt_half* K, const lt_half* V,
                      int64_t q_row_stride, int64_t kv_row_stride, lt_half* O,
                      int64_t o_row_stride, float* LSE, int B, int S, int Hq,
                      int Hkv, int D, float scale, int causal,
                      lt_stream stream);

/*
 * Bytes of device workspace lt_attn_bwd needs, each part 256-byte aligned,
 * in this order:
 *   D_i = rowsum(dO_i * O_i)              [B, Hq, S] FP32 (offset 0)
 *   the row LSE in base 2                 [B, Hq, S] FP32
 *   dS = P * (dP - D) in FP16, one 2 KiB block per (32-key group, 32-query
 *   group) pair the mask keeps (n32 (n32 + 1) / 2 per (batch, query head)
 *   under the causal mask, n32^2 without, n32 = ceil(S / 32)): written by the
 *   dK/dV pass, read by the dQ pass;
 *   FP32 partial dK and dV sums [2][n][B, S, Hkv, D] when the dK/dV work is
 *   split into n > 1 shares.
 * The dK/dV pass takes 256-key tiles, except for MHA (Hq = Hkv) when those
 * give fewer than 512 workgroups over all batches and key/value heads: then
 * 128-key tiles.  When the chosen tiles still give fewer than 512 workgroups
 * (few kv heads, short sequences) each key tile's (query head, 64-query
 * block) pairs are split into n contiguous shares, one workgroup each, and
 * the partials are summed in a fixed order, so results stay deterministic.
 * 0 for invalid sizes.
 */
size_t lt_attn_bwd_workspace_size(int B, int S, int Hq, int Hkv, int D, int causal);

/*
 * Attention backward (Sec. 4.1, Algorithm 1: GP = GO V^T,
 * GS = SoftmaxBackward(P, GP), GV = P^T GO, GQ = GS K, GK = GS^T Q).
 * P is recomputed as exp(scale * q.k - LSE) from the forward's LSE instead of
 * being read back; SoftmaxBackward is GS_ij = P_ij (GP_ij - D_i) with
 * D_i = rowsum(dO_i * O_i).  GS is kept in FP16 between the key-major pass
 * (GV, GK) and the query-major GQ = GS K.  dQ and dK carry the factor `scale`.
 * dK and dV of a key/value head sum over its Hq/Hkv query heads.
 *
 *   Q, K, V, O, dO, LSE: as written by / passed to lt_attn_fwd (O and dO share
 *   o_row_stride).  dQ uses dq_row_stride, dK and dV use dkv_row_stride, so
 *   they may be column slices of one fused dQKV buffer.  dQ, dK, dV are
 *   overwritten.  `workspace` is a device buffer of at least
 *   lt_attn_bwd_workspace_size(B, S, Hq, Hkv, D, causal) bytes, 256-byte
 *   aligned, owned by the caller; its contents on entry are ignored.
 *   Errors: as lt_attn_fwd (every row stride, dq_row_stride and
 *   dkv_row_stride included, must be < 2^22 elements), plus LT_ERR_WORKSPACE
 *   if workspace is NULL or ws_bytes is too small.
 */
lt_status lt_attn_bwd(const lt_half* Q, const lt_half* K, const lt_half* V,
                      int64_t q_row_stride, int64_t kv_row_stride,
                      const lt_half* O, const lt_half* dO,
                      int64_t o_row_stride, const float* LSE, lt_half* dQ,
                      lt_half* dK, lt_half* dV, int64_t dq_row_stride,
                      int64_t dkv_row_stride, void* workspace, size_t ws_bytes,
                      int B, int S, int Hq, int Hkv, int D, float scale,
                      int causal, lt_stream stream);

/*
 * Saved-P attention (Algorithm 1 as the paper states it: the backward loads
 * the probability tiles P_ij the forward produced instead of recomputing
 * them).  An alternative to lt_attn_bwd's recomputed P that trades HBM
 * traffic and residency for MFMA work.
 *
 * lt_attn_p_size: bytes of the P buffer, one 2 KiB FP16 block per
 *   (32-key group, 32-query group) pair the mask keeps (n32 (n32 + 1) / 2 per
 *   (batch, query head) under the causal mask, n32^2 without,
 *   n32 = ceil(S / 32)); 0 for invalid sizes.  0.54 GB at LLaMA-2-7B's 32
 *   heads and S = 4096.
 * lt_attn_fwd_p: lt_attn_fwd, then P = exp(scale q.k - LSE) of those blocks
 *   into the caller's buffer P (p_bytes >= lt_attn_p_size, 16-byte aligned);
 *   masked entries are exactly 0.  P stays valid for the matching
 *   lt_attn_bwd_p.  Errors: as lt_attn_fwd; LT_ERR_WORKSPACE if p_bytes is
 *   too small.
 * lt_attn_bwd_p: the backward of lt_attn_bwd with P read from that buffer
 *   (written by lt_attn_fwd_p for the same Q, K, shapes, scale and causal):
 *   GV = P^T GO and GK = GS^T Q in a key-major pass whose GP = GO V^T is the
 *   only product it forms, and GQ = GS K in a query-major pass that forms S
 *   and GP itself (and D_i = rowsum(dO_i * O_i), run first).  The workspace
 *   (lt_attn_bwd_p_workspace_size bytes, 256-byte aligned) holds D and the
 *   base-2 LSE [B, Hq, S] FP32 and, when the dK/dV work is split into
 *   shares, FP32 partial dK, dV as for lt_attn_bwd.  Errors: as lt_attn_bwd,
 *   plus LT_ERR_INVALID_ARG for a NULL or too small P.
 */
size_t lt_attn_p_size(int B, int S, int Hq, int causal);
lt_status lt_attn_fwd_p(const lt_half* Q, const lt_half* K, const lt_half* V,
                        int64_t q_row_stride, int64_t kv_row_stride, lt_half* O,
                        int64_t o_row_stride, float* LSE, lt_half* P,
                        size_t p_bytes, int B, int S, int Hq, int Hkv, int D,
                        float scale, int causal, lt_stream stream);
size_t lt_attn_bwd_p_workspace_size(int B, int S, int Hq, int Hkv, int D);
lt_status lt_attn_bwd_p(const lt_half* Q, const lt_half* K, const lt_half* V,
                        int64_t q_row_stride, int64_t kv_row_stride,
                        const lt_half* O, const lt_half* dO,
                        int64_t o_row_stride, const float* LSE,
                        const lt_half* P, size_t p_bytes, lt_half* dQ,
                        lt_half* dK, lt_half* dV, int64_t dq_row_stride,
                        int64_t dkv_row_stride, void* workspace,
                        size_t ws_bytes, int B, int S, int Hq, int Hkv, int D,
                        float scale, int causal, lt_stream stream);

/*
 * SwiGLU gate joining the FFN gate/up projection and the down projection.
 *   GU is [T, 2F] (row stride 2F): columns 0..F-1 gate G, F..2F-1 up U.
 *   forward : A[T, F]   = silu(G) * U,  silu(x) = x / (1 + exp(-x))
 *   backward: dGU[T,2F] = [dA * U * s * (1 + G (1 - s)) | dA * silu(G)],
 *             s = sigmoid(G)
 *   Math in FP32, one RNE rounding of each output.
 *   T == 0 or F == 0: no-op.  Errors: INVALID_ARG for NULL pointers or
 *   negative sizes; UNSUPPORTED for F not a multiple of 8 or misaligned
 *   pointers.
 */
lt_status lt_swiglu_fwd(const lt_half* GU, lt_half* A, int64_t T, int64_t F,
                        lt_stream stream);
lt_status lt_swiglu_bwd(const lt_half* dA, const lt_half* GU, lt_half* dGU,
                        int64_t T, int64_t F, lt_stream stream);

/*
 * Gate/up projection with the SwiGLU gate in its epilogue (the FFN
 * projection of Sec. 4.1 followed by the evaluated models' gate, fused):
 *   GU = X Wgu^T   (X [T, H], Wgu [2F, H]: gate rows 0..F-1, then up rows;
 *                   GU [T, 2F]: G in columns 0..F-1, U in F..2F-1)
 *   A  = silu(G) * U   [T, F]
 * G and U are rounded once from the FP32 accumulators and equal those of
 * lt_gemm_f16(0, 1, T, 2F, H, 1, X, ldx, Wgu, ldw, 0, GU, ldgu) bit for bit;
 * A is computed from the same FP32 values (not from the rounded G, U).
 * T, H, F multiples of 8, strides multiples of 8, pointers 16-byte aligned,
 * 2*F*ldw < 2^30 - 128 (else LT_ERR_UNSUPPORTED).  GU and A must not overlap X,
 * Wgu or each other.
 */
lt_status lt_gemm_gu_swiglu_f16(const lt_half* X, int64_t ldx, const lt_half* Wgu,
                                int64_t ldw, lt_half* GU, int64_t ldgu, lt_half* A,
                                int64_t lda, int64_t T, int64_t H, int64_t F,
                                lt_stream stream);

/*
 * Down-projection data gradient with the SwiGLU backward in its epilogue:
 *   dA  = dY Wd   (dY [T, H], Wd [H, F]; FP32, never stored)
 *   dGU = [dA * U * s * (1 + G (1 - s)),  dA * silu(G)],  s = sigmoid(G),
 * G and U read from GU [T, 2F]; dGU [T, 2F] is written once per element.
 * Limits as lt_gemm_gu_swiglu_f16; dGU must not overlap the inputs.
 */
lt_status lt_gemm_swiglu_bwd_f16(const lt_half* dY, int64_t lddy, const lt_half* Wd,
                                 int64_t ldwd, const lt_half* GU, int64_t ldgu,
                                 lt_half* dGU, int64_t lddgu, int64_t T, int64_t H,
                                 int64_t F, lt_stream stream);

/*
 * RMSNorm of the evaluated models' decoder layers (Sec. 6.1 names LLaMA-2,
 * Baichuan2 and Qwen2.5; the paper itself defines no normalisation), per
 * token row x of width H:  r = (mean_j x_j^2 + eps)^(-1/2),  y = w * x * r.
 *   X [T, H] (row stride ldx), W [H], Y [T, H] (ldy): FP16; RSTD [T]: FP32,
 *   the r of every row, kept for the backward.  Math in FP32, one rounding
 *   per output.  H must be a multiple of 8 and <= 8192, strides multiples of
 *   8 elements, pointers 16-byte aligned (else LT_ERR_UNSUPPORTED); eps
 *   finite and >= 0.  T = 0 is a no-op.
 */
lt_status lt_rmsnorm_fwd(const lt_half* X, int64_t ldx, const lt_half* W,
                         lt_half* Y, int64_t ldy, float* RSTD, int64_t T,
                         int64_t H, float eps, lt_stream stream);

/*
 * Bytes of device workspace lt_rmsnorm_bwd needs (FP32 partial sums of dW,
 * 256-byte aligned); 0 for invalid sizes.
 */
size_t lt_rmsnorm_bwd_workspace_size(int64_t T, int64_t H);

/*
 * RMSNorm backward, given dY (the gradient of y) and the forward's X, W, RSTD:
 *   dX = R + r * w * dY - r^3 * x / H * sum_j dY_j w_j x_j   (R optional,
 *        NULL for none: the residual-branch gradient added in the same pass),
 *   dW = sum over rows of dY * x * r   (FP16, summed in FP32 in a fixed
 *        order: deterministic).
 * Layouts and limits as lt_rmsnorm_fwd; T >= 1.  `workspace` is a device
 * buffer of at least lt_rmsnorm_bwd_workspace_size(T, H) bytes, 256-byte
 * aligned, owned by the caller.
 */
lt_status lt_rmsnorm_bwd(const lt_half* dY, int64_t lddy, const lt_half* X,
                         int64_t ldx, const lt_half* W, const float* RSTD,
                         const lt_half* R, int64_t ldr, lt_half* dX,
                         int64_t lddx, lt_half* dW, void* workspace,
                         size_t ws_bytes, int64_t T, int64_t H,
                         lt_stream stream);

/*
 * Rotary position embedding table of the evaluated models (rotate-half
 * pairing): CS[p][i] = (cos a, sin a), a = p * base^(-2i/D), for p < S and
 * i < D/2, FP32 pairs ([S][D/2][2], caller-owned, 16-byte aligned).  The
 * angle is formed and reduced in FP64.  D must be a multiple of 16.
 */
lt_status lt_rope_table(float* CS, int S, int D, double base,
                        lt_stream stream);

/*
 * Rotary embedding in place on `heads` consecutive heads of width D of every
 * token row: element (b, p, h, :) at X + (b*S + p) * row_stride + h*D (in
 * the fused QKV buffer the Q heads and then the K heads, heads = Hq + Hkv).
 * Pairs (i, i + D/2) rotate by the angle of CS[p][i]; inverse = 1 rotates by
 * the negated angle, which is the gradient of the forward rotation.  FP32
 * math, one rounding per output.  D % 16 == 0, row_stride % 8 == 0, X and
 * CS 16-byte aligned (else LT_ERR_UNSUPPORTED).
 */
lt_status lt_rope_f16(lt_half* X, int64_t row_stride, int B, int S, int heads,
                      int D, const float* CS, int inverse, lt_stream stream);

#ifdef __cplusplus
}
#endif

#endif /* LT_H_ */
