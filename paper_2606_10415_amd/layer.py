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
"""

import math

import torch

from . import lt


class DecoderLayer:
    """Device buffers and the liblt call sequence of one layer.

    ``shape`` needs attributes B, S, H, Hq, Hkv, D, F.  ``params`` maps
    X, dY, Wqkv, Wo, Wgu, Wd to float16 tensors (host or device).
    """

    def __init__(self, shape, params, device="cuda"):
        self.sh = sh = shape
        self.dev = torch.device(device)
        T = sh.B * sh.S
        self.T = T
        self.qkv = (sh.Hq + 2 * sh.Hkv) * sh.D
        self.hd = sh.Hq * sh.D
        self.scale = 1.0 / math.sqrt(sh.D)

        def dev(x):
            t = x if isinstance(x, torch.Tensor) else torch.from_numpy(x)
            return t.to(self.dev, torch.float16).contiguous()

        self.X = dev(params["X"])
        self.dY = dev(params["dY"])
        self.Wqkv = dev(params["Wqkv"])
        self.Wo = dev(params["Wo"])
        self.Wgu = dev(params["Wgu"])
        self.Wd = dev(params["Wd"])

        e = lambda *s: torch.empty(*s, dtype=torch.float16, device=self.dev)
        self.QKV = e(T, self.qkv)
        self.O = e(T, self.hd)
        self.LSE = torch.empty(sh.B, sh.Hq, sh.S, dtype=torch.float32, device=self.dev)
        self.H1 = e(T, sh.H)
        self.GU = e(T, 2 * sh.F)
        self.A = e(T, sh.F)
        self.Y = e(T, sh.H)
        self.dA = e(T, sh.F)
        self.dGU = e(T, 2 * sh.F)
        self.dH1 = e(T, sh.H)
        self.dO = e(T, self.hd)
        self.dQKV = e(T, self.qkv)
        self.dX = e(T, sh.H)
        self.dWqkv = e(*self.Wqkv.shape)
        self.dWo = e(*self.Wo.shape)
        self.dWgu = e(*self.Wgu.shape)
        self.dWd = e(*self.Wd.shape)
        self.ws_bytes = lt.lt_attn_bwd_workspace_size(sh.B, sh.S, sh.Hq, sh.Hkv, sh.D)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.dev)

    # ------------------------------------------------------------ steps
    def _attn_ptrs(self, base):
        p = base.data_ptr()
        return p, p + 2 * self.hd, p + 2 * (self.hd + self.sh.Hkv * self.sh.D)

    def forward(self, stream=None, hook=None):
        """Layer forward.  ``hook(name)`` (optional) is called after each launch."""
        sh, T = self.sh, self.T
        mark = hook or (lambda name: None)
        lt.lt_gemm_f16(0, 1, T, self.qkv, sh.H, 1.0, self.X, sh.H, self.Wqkv, sh.H, 0.0,
                       self.QKV, self.qkv, stream)
        mark("qkv_fwd")
        q, k, v = self._attn_ptrs(self.QKV)
        lt.lt_attn_fwd(q, k, v, self.qkv, self.qkv, self.O, self.hd, self.LSE, sh.B, sh.S, sh.Hq,
                       sh.Hkv, sh.D, self.scale, 1, stream)
        mark("attn_fwd")
        lt.lt_gemm_f16_res(0, 1, T, sh.H, self.hd, 1.0, self.O, self.hd, self.Wo, self.hd, 1.0,
                           self.X, sh.H, self.H1, sh.H, stream)
        mark("o_fwd")
        lt.lt_gemm_f16(0, 1, T, 2 * sh.F, sh.H, 1.0, self.H1, sh.H, self.Wgu, sh.H, 0.0, self.GU,
                       2 * sh.F, stream)
        mark("gu_fwd")
        lt.lt_swiglu_fwd(self.GU, self.A, T, sh.F, stream)
        mark("swiglu_fwd")
        lt.lt_gemm_f16_res(0, 1, T, sh.H, sh.F, 1.0, self.A, sh.F, self.Wd, sh.F, 1.0, self.H1,
                           sh.H, self.Y, sh.H, stream)
        mark("down_fwd")

    def backward(self, stream=None, hook=None):
        sh, T = self.sh, self.T
        mark = hook or (lambda name: None)
        # down projection
        lt.lt_gemm_f16(1, 0, sh.H, sh.F, T, 1.0, self.dY, sh.H, self.A, sh.F, 0.0, self.dWd, sh.F,
                       stream)
        mark("down_wgrad")
        lt.lt_gemm_f16(0, 0, T, sh.F, sh.H, 1.0, self.dY, sh.H, self.Wd, sh.F, 0.0, self.dA, sh.F,
                       stream)
        mark("down_dgrad")
        lt.lt_swiglu_bwd(self.dA, self.GU, self.dGU, T, sh.F, stream)
        mark("swiglu_bwd")
        # gate/up projection
        lt.lt_gemm_f16(1, 0, 2 * sh.F, sh.H, T, 1.0, self.dGU, 2 * sh.F, self.H1, sh.H, 0.0,
                       self.dWgu, sh.H, stream)
        mark("gu_wgrad")
        lt.lt_gemm_f16_res(0, 0, T, sh.H, 2 * sh.F, 1.0, self.dGU, 2 * sh.F, self.Wgu, sh.H, 1.0,
                           self.dY, sh.H, self.dH1, sh.H, stream)
        mark("gu_dgrad")
        # output projection
        lt.lt_gemm_f16(1, 0, sh.H, self.hd, T, 1.0, self.dH1, sh.H, self.O, self.hd, 0.0, self.dWo,
                       self.hd, stream)
        mark("o_wgrad")
        lt.lt_gemm_f16(0, 0, T, self.hd, sh.H, 1.0, self.dH1, sh.H, self.Wo, self.hd, 0.0, self.dO,
                       self.hd, stream)
        mark("o_dgrad")
        # attention
        q, k, v = self._attn_ptrs(self.QKV)
        dq, dk, dv = self._attn_ptrs(self.dQKV)
        lt.lt_attn_bwd(q, k, v, self.qkv, self.qkv, self.O, self.dO, self.hd, self.LSE, dq, dk, dv,
                       self.qkv, self.qkv, self.ws, self.ws_bytes, sh.B, sh.S, sh.Hq, sh.Hkv, sh.D,
                       self.scale, 1, stream)
        mark("attn_bwd")
        # QKV projection
        lt.lt_gemm_f16(1, 0, self.qkv, sh.H, T, 1.0, self.dQKV, self.qkv, self.X, sh.H, 0.0,
                       self.dWqkv, sh.H, stream)
        mark("qkv_wgrad")
        lt.lt_gemm_f16_res(0, 0, T, sh.H, self.qkv, 1.0, self.dQKV, self.qkv, self.Wqkv, sh.H, 1.0,
                           self.dH1, sh.H, self.dX, sh.H, stream)
        mark("qkv_dgrad")

    def step(self, stream=None, hook=None):
        self.forward(stream, hook)
        self.backward(stream, hook)

    # GEMM launches of one step, in call order, as (name, M, N, K)
    def gemm_shapes(self):
        sh, T = self.sh, self.T
        return [("qkv_fwd", T, self.qkv, sh.H), ("o_fwd", T, sh.H, self.hd),
                ("gu_fwd", T, 2 * sh.F, sh.H), ("down_fwd", T, sh.H, sh.F),
                ("down_wgrad", sh.H, sh.F, T), ("down_dgrad", T, sh.F, sh.H),
                ("gu_wgrad", 2 * sh.F, sh.H, T), ("gu_dgrad", T, sh.H, 2 * sh.F),
                ("o_wgrad", sh.H, self.hd, T), ("o_dgrad", T, self.hd, sh.H),
                ("qkv_wgrad", self.qkv, sh.H, T), ("qkv_dgrad", T, sh.H, self.qkv)]
