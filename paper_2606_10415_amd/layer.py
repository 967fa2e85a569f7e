"""One dense decoder layer, forward + backward, as a sequence of liblt calls.

The layer is the unit the paper's backend executes per pipeline stage
(Sec. 4.1: QKV / output / FFN projections and attention backward; Sec. 6.1
workload shapes).  Every step is a call into the HIP library on one stream;
PyTorch only provides the device buffers.

Forward  : QKV = X Wqkv^T ; (O, LSE) = attn(QKV) ; H1 = X + O Wo^T ;
           GU = H1 Wgu^T ; A = silu(G) U ; Y = H1 + A Wd^T
Backward : dWd = dY^T A ; dA = dY Wd ; dGU = swiglu_bwd ; dWgu = dGU^T H1 ;
           dH1 = dY + dGU Wgu ; dWo = dH1^T O ; dO = dH1 Wo ;
           dQKV = attn_bwd ; dWqkv = dQKV^T X ; dX = dH1 + dQKV Wqkv

With ``norm`` the layer is the full block of the evaluated models: X and H1
are RMSNorm-ed before the QKV and gate/up projections (Xn, H1n), Q and K are
rotated in place in QKV, and the backward runs the inverse rotation on dQ, dK
and RMSNorm backward (with the residual gradient added in the same pass):
    dH1 = dY + rmsnorm_bwd(dGU Wgu) ;  dX = dH1 + rmsnorm_bwd(dQKV Wqkv)

A norm with a QKV bias (Qwen2.5) adds it in the QKV GEMM's epilogue and
takes its gradient as the column sum of dQKV after the inverse rotation.

With ``fuse_swiglu`` the SwiGLU gate runs in the epilogues of the gate/up
GEMM (A from the FP32 accumulators, GU still stored for the backward) and of
the down-projection dgrad (dGU written directly, dA never stored).
"""

import math

import torch

from . import lt


class DecoderLayer:
    """Device buffers and the liblt call sequence of one layer.

    ``shape`` needs attributes B, S, H, Hq, Hkv, D, F.  ``params`` maps
    X, dY, Wqkv, Wo, Wgu, Wd to float16 tensors (host or device).  ``norm``
    (optional) has attributes wn1, wn2 (RMSNorm weights [H]), eps, rope_base and
    optionally bqkv (QKV projection bias, or None).
    ``fuse_swiglu`` selects the GEMMs with the SwiGLU epilogues.
    """

    def __init__(self, shape, params, device="cuda", norm=None, fuse_swiglu=True,
                 share_bwd=None, share_acts=None):
        self.sh = sh = shape
        self.fuse_swiglu = bool(fuse_swiglu)
        self.accumulate = False
        self.dev = torch.device(device)
        T = sh.B * sh.S
        self.T = T
        self.qkv = (sh.Hq + 2 * sh.Hkv) * sh.D
        self.hd = sh.Hq * sh.D
        self.scale = 1.0 / math.sqrt(sh.D)

        def dev(x):
            t = x if isinstance(x, torch.Tensor) else torch.from_numpy(x)
            return t.to(self.dev, torch.float16).contiguous()

        self.X = dev(params["X"]) if params.get("X") is not None else None
        self.dY = dev(params["dY"]) if params.get("dY") is not None else None
        self.Wqkv = dev(params["Wqkv"])
        self.Wo = dev(params["Wo"])
        self.Wgu = dev(params["Wgu"])
        self.Wd = dev(params["Wd"])

        e = lambda *s: torch.empty(*s, dtype=torch.float16, device=self.dev)
        # forward activations the backward reads (shareable between layers
        # whose forward is recomputed right before their backward)
        if share_acts is not None:
            for k in ("QKV", "O", "LSE", "H1", "GU", "A"):
                setattr(self, k, getattr(share_acts, k))
        else:
            self.QKV = e(T, self.qkv)
            self.O = e(T, self.hd)
            self.LSE = torch.empty(sh.B, sh.Hq, sh.S, dtype=torch.float32, device=self.dev)
            self.H1 = e(T, sh.H)
            self.GU = e(T, 2 * sh.F)
            self.A = e(T, sh.F)
        self.Y = e(T, sh.H)
        # backward temporaries (shareable between the layers of a stage)
        if share_bwd is not None:
            for k in ("dA", "dGU", "dH1", "dO", "dQKV", "dX", "ws", "ws_bytes", "gemm_ws",
                      "gemm_ws_bytes"):
                setattr(self, k, getattr(share_bwd, k))
        else:
            self.dA = e(T, sh.F)
            self.dGU = e(T, 2 * sh.F)
            self.dH1 = e(T, sh.H)
            self.dO = e(T, self.hd)
            self.dQKV = e(T, self.qkv)
            self.dX = e(T, sh.H)
            self.ws_bytes = lt.lt_attn_bwd_workspace_size(sh.B, sh.S, sh.Hq, sh.Hkv, sh.D, 1)
            self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.dev)
            # split-K workspace of the plain GEMM calls (one at a time on the
            # stream); the fused SwiGLU GEMMs take none
            fused = ("gu_fwd", "down_dgrad") if self.fuse_swiglu else ()
            self.gemm_ws_bytes = max(lt.lt_gemm_f16_workspace_size(ta, tb, M, N, K)
                                     for n, ta, tb, M, N, K in self._gemm_calls() if n not in fused)
            self.gemm_ws = (torch.empty(self.gemm_ws_bytes, dtype=torch.uint8, device=self.dev)
                            if self.gemm_ws_bytes else None)
        self.dWqkv = e(*self.Wqkv.shape)
        self.dWo = e(*self.Wo.shape)
        self.dWgu = e(*self.Wgu.shape)
        self.dWd = e(*self.Wd.shape)

        self.norm = norm
        if norm is not None:
            self.eps = float(norm.eps)
            self.Wn1 = dev(norm.wn1)
            self.Wn2 = dev(norm.wn2)
            self.Xn = e(T, sh.H)
            self.H1n = e(T, sh.H)
            self.dXn = e(T, sh.H)
            self.dH1n = e(T, sh.H)
            self.dWn1 = e(sh.H)
            self.dWn2 = e(sh.H)
            f32 = lambda *s_: torch.empty(*s_, dtype=torch.float32, device=self.dev)
            self.rstd1 = f32(T)
            self.rstd2 = f32(T)
            self.CS = f32(sh.S, sh.D // 2, 2)
            lt.lt_rope_table(self.CS, sh.S, sh.D, float(norm.rope_base))
            self.rms_ws_bytes = lt.lt_rmsnorm_bwd_workspace_size(T, sh.H)
            self.rms_ws = torch.empty(self.rms_ws_bytes, dtype=torch.uint8, device=self.dev)
        self.bqkv = None
        if norm is not None and getattr(norm, "bqkv", None) is not None:
            self.bqkv = dev(norm.bqkv)
            self.dbqkv = e(self.qkv)
            self.bias_ws_bytes = lt.lt_bias_grad_workspace_size(T, self.qkv)
            self.bias_ws = torch.empty(self.bias_ws_bytes, dtype=torch.uint8, device=self.dev)

    # ------------------------------------------------------------ steps
    def _gemm(self, ta, tb, M, N, K, A, lda, B, ldb, beta, C, ldc, stream, R=None, ldr=None,
              bias=None):
        """C = op(A) op(B) + beta R (+ bias), R defaulting to C, with the layer's
        split-K workspace (a last, at most half full, wave of output tiles
        splits its K over several workgroups)."""
        if R is None:
            R, ldr = C, ldc
        lt.lt_gemm_f16_ws(ta, tb, M, N, K, 1.0, A, lda, B, ldb, beta, R, ldr, bias, C, ldc,
                          self.gemm_ws, self.gemm_ws_bytes, stream)

    def _attn_ptrs(self, base):
        p = base.data_ptr()
        return p, p + 2 * self.hd, p + 2 * (self.hd + self.sh.Hkv * self.sh.D)

    def forward(self, stream=None, hook=None):
        """Layer forward.  ``hook(name)`` (optional) is called after each launch."""
        sh, T = self.sh, self.T
        mark = hook or (lambda name: None)
        xin = self.X
        if self.norm is not None:
            lt.lt_rmsnorm_fwd(self.X, sh.H, self.Wn1, self.Xn, sh.H, self.rstd1, T, sh.H, self.eps,
                              stream)
            mark("rmsnorm1_fwd")
            xin = self.Xn
        if self.bqkv is not None:
            self._gemm(0, 1, T, self.qkv, sh.H, xin, sh.H, self.Wqkv, sh.H, 0.0, self.QKV, self.qkv,
                       stream, bias=self.bqkv)
        else:
            self._gemm(0, 1, T, self.qkv, sh.H, xin, sh.H, self.Wqkv, sh.H, 0.0, self.QKV, self.qkv,
                       stream)
        mark("qkv_fwd")
        if self.norm is not None:
            lt.lt_rope_f16(self.QKV, self.qkv, sh.B, sh.S, sh.Hq + sh.Hkv, sh.D, self.CS, 0, stream)
            mark("rope_fwd")
        q, k, v = self._attn_ptrs(self.QKV)
        lt.lt_attn_fwd(q, k, v, self.qkv, self.qkv, self.O, self.hd, self.LSE, sh.B, sh.S, sh.Hq,
                       sh.Hkv, sh.D, self.scale, 1, stream)
        mark("attn_fwd")
        self._gemm(0, 1, T, sh.H, self.hd, self.O, self.hd, self.Wo, self.hd, 1.0, self.H1, sh.H,
                   stream, R=self.X, ldr=sh.H)
        mark("o_fwd")
        hin = self.H1
        if self.norm is not None:
            lt.lt_rmsnorm_fwd(self.H1, sh.H, self.Wn2, self.H1n, sh.H, self.rstd2, T, sh.H,
                              self.eps, stream)
            mark("rmsnorm2_fwd")
            hin = self.H1n
        if self.fuse_swiglu:
            lt.lt_gemm_gu_swiglu_f16(hin, sh.H, self.Wgu, sh.H, self.GU, 2 * sh.F, self.A, sh.F, T,
                                     sh.H, sh.F, stream)
            mark("gu_fwd")
        else:
            self._gemm(0, 1, T, 2 * sh.F, sh.H, hin, sh.H, self.Wgu, sh.H, 0.0, self.GU, 2 * sh.F,
                       stream)
            mark("gu_fwd")
            lt.lt_swiglu_fwd(self.GU, self.A, T, sh.F, stream)
            mark("swiglu_fwd")
        self._gemm(0, 1, T, sh.H, sh.F, self.A, sh.F, self.Wd, sh.F, 1.0, self.Y, sh.H, stream,
                   R=self.H1, ldr=sh.H)
        mark("down_fwd")

    def backward(self, stream=None, hook=None):
        sh, T = self.sh, self.T
        mark = hook or (lambda name: None)
        # down projection
        if self.accumulate and (self.norm is not None or self.bqkv is not None):
            raise ValueError("gradient accumulation covers the four projection weights only")
        wb = 1.0 if self.accumulate else 0.0     # weight gradients: overwrite or accumulate
        self._gemm(1, 0, sh.H, sh.F, T, self.dY, sh.H, self.A, sh.F, wb, self.dWd, sh.F, stream)
        mark("down_wgrad")
        if self.fuse_swiglu:
            lt.lt_gemm_swiglu_bwd_f16(self.dY, sh.H, self.Wd, sh.F, self.GU, 2 * sh.F, self.dGU,
                                      2 * sh.F, T, sh.H, sh.F, stream)
            mark("down_dgrad")
        else:
            self._gemm(0, 0, T, sh.F, sh.H, self.dY, sh.H, self.Wd, sh.F, 0.0, self.dA, sh.F,
                       stream)
            mark("down_dgrad")
            lt.lt_swiglu_bwd(self.dA, self.GU, self.dGU, T, sh.F, stream)
            mark("swiglu_bwd")
        # gate/up projection
        hin = self.H1n if self.norm is not None else self.H1
        self._gemm(1, 0, 2 * sh.F, sh.H, T, self.dGU, 2 * sh.F, hin, sh.H, wb, self.dWgu, sh.H,
                   stream)
        mark("gu_wgrad")
        if self.norm is not None:
            self._gemm(0, 0, T, sh.H, 2 * sh.F, self.dGU, 2 * sh.F, self.Wgu, sh.H, 0.0, self.dH1n,
                       sh.H, stream)
            mark("gu_dgrad")
            lt.lt_rmsnorm_bwd(self.dH1n, sh.H, self.H1, sh.H, self.Wn2, self.rstd2, self.dY, sh.H,
                              self.dH1, sh.H, self.dWn2, self.rms_ws, self.rms_ws_bytes, T, sh.H,
                              stream)
            mark("rmsnorm2_bwd")
        else:
            self._gemm(0, 0, T, sh.H, 2 * sh.F, self.dGU, 2 * sh.F, self.Wgu, sh.H, 1.0, self.dH1,
                       sh.H, stream, R=self.dY, ldr=sh.H)
            mark("gu_dgrad")
        # output projection
        self._gemm(1, 0, sh.H, self.hd, T, self.dH1, sh.H, self.O, self.hd, wb, self.dWo, self.hd,
                   stream)
        mark("o_wgrad")
        self._gemm(0, 0, T, self.hd, sh.H, self.dH1, sh.H, self.Wo, self.hd, 0.0, self.dO, self.hd,
                   stream)
        mark("o_dgrad")
        # attention
        q, k, v = self._attn_ptrs(self.QKV)
        dq, dk, dv = self._attn_ptrs(self.dQKV)
        lt.lt_attn_bwd(q, k, v, self.qkv, self.qkv, self.O, self.dO, self.hd, self.LSE, dq, dk, dv,
                       self.qkv, self.qkv, self.ws, self.ws_bytes, sh.B, sh.S, sh.Hq, sh.Hkv, sh.D,
                       self.scale, 1, stream)
        mark("attn_bwd")
        if self.norm is not None:
            lt.lt_rope_f16(self.dQKV, self.qkv, sh.B, sh.S, sh.Hq + sh.Hkv, sh.D, self.CS, 1, stream)
            mark("rope_bwd")
        if self.bqkv is not None:
            lt.lt_bias_grad_f16(self.dQKV, self.qkv, T, self.qkv, self.dbqkv, self.bias_ws,
                                self.bias_ws_bytes, stream)
            mark("qkv_bias_grad")
        # QKV projection
        xin = self.Xn if self.norm is not None else self.X
        self._gemm(1, 0, self.qkv, sh.H, T, self.dQKV, self.qkv, xin, sh.H, wb, self.dWqkv, sh.H,
                   stream)
        mark("qkv_wgrad")
        if self.norm is not None:
            self._gemm(0, 0, T, sh.H, self.qkv, self.dQKV, self.qkv, self.Wqkv, sh.H, 0.0, self.dXn,
                       sh.H, stream)
            mark("qkv_dgrad")
            lt.lt_rmsnorm_bwd(self.dXn, sh.H, self.X, sh.H, self.Wn1, self.rstd1, self.dH1, sh.H,
                              self.dX, sh.H, self.dWn1, self.rms_ws, self.rms_ws_bytes, T, sh.H,
                              stream)
            mark("rmsnorm1_bwd")
        else:
            self._gemm(0, 0, T, sh.H, self.qkv, self.dQKV, self.qkv, self.Wqkv, sh.H, 1.0, self.dX,
                       sh.H, stream, R=self.dH1, ldr=sh.H)
            mark("qkv_dgrad")

    def step(self, stream=None, hook=None):
        self.forward(stream, hook)
        self.backward(stream, hook)

    # plain GEMM calls of one step as (name, transA, transB, M, N, K): forward
    # NT, weight gradients TN, data gradients NN
    def _gemm_calls(self):
        lay = {"fwd": (0, 1), "wgrad": (1, 0), "dgrad": (0, 0)}
        return [(n,) + lay[n.split("_")[1]] + (M, N, K) for n, M, N, K in self.gemm_shapes()]

    # GEMM launches of one step, in call order, as (name, M, N, K)
    def gemm_shapes(self):
        sh, T = self.sh, self.T
        return [("qkv_fwd", T, self.qkv, sh.H), ("o_fwd", T, sh.H, self.hd),
                ("gu_fwd", T, 2 * sh.F, sh.H), ("down_fwd", T, sh.H, sh.F),
                ("down_wgrad", sh.H, sh.F, T), ("down_dgrad", T, sh.F, sh.H),
                ("gu_wgrad", 2 * sh.F, sh.H, T), ("gu_dgrad", T, sh.H, 2 * sh.F),
                ("o_wgrad", sh.H, self.hd, T), ("o_dgrad", T, self.hd, sh.H),
                ("qkv_wgrad", self.qkv, sh.H, T), ("qkv_dgrad", T, sh.H, self.qkv)]
