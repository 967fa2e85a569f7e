"""One pipeline stage of L decoder layers on one GPU (the planner's P = 1 case).

The stage runs non-interleaved 1F1B with a single stage: for each of the A
micro-batches, the forward through all L layers and then the backward back
through them (Sec. 3's 1F1B main schedule; with one stage there is no warm-up
and one micro-batch is in flight).  Weight gradients accumulate over the
micro-batches (the first writes, the others add through the GEMM's beta = 1
accumulation input, Sec. 4.1).

Activation policies (Sec. 4.3):
  * "full": every layer keeps its forward activations until its backward;
  * "ckpt": every layer keeps only its input (the previous layer's output) and
    one recovery buffer set is shared by all layers: the backward of layer l
    first recomputes layer l's forward into it.

Layers with RMSNorm / rotary embedding / QKV bias (``norm``) run single
micro-batches only (their norm and bias gradients are not accumulated).

Backward temporaries (dA, dGU, dH1, dO, dQKV and the attention workspace) are
shared by all layers; the input gradients alternate between two buffers.  With
``optimizer_state`` the stage also holds the FP32 master weights and two Adam
moments (12 bytes per parameter) that a training run keeps resident, so that
the measured peak memory covers the planner's state term.
"""

import torch

from .layer import DecoderLayer


class Stage:
    def __init__(self, shape, layers, act="full", seed=0, device="cuda", optimizer_state=False,
                 weights=None, norm=None):
        if act not in ("full", "ckpt"):
            raise ValueError("act must be 'full' or 'ckpt'")
        self.sh = sh = shape
        self.L = layers
        self.act = act
        self.dev = torch.device(device)
        T = sh.B * sh.S
        qkv = (sh.Hq + 2 * sh.Hkv) * sh.D
        gen = torch.Generator(device=self.dev)
        gen.manual_seed(seed)

        def rnd(*shape_, std=1.0):
            return (torch.randn(*shape_, generator=gen, device=self.dev) * std).half()

        self.layers = []
        for l in range(layers):
            if weights is not None:
                p = dict(weights[l])
            else:
                p = {"Wqkv": rnd(qkv, sh.H, std=0.02), "Wo": rnd(sh.H, sh.Hq * sh.D, std=0.02),
                     "Wgu": rnd(2 * sh.F, sh.H, std=0.02), "Wd": rnd(sh.H, sh.F, std=0.02)}
            p["X"] = None
            p["dY"] = None
            first = self.layers[0] if self.layers else None
            share_acts = first if (act == "ckpt" and first is not None) else None
            self.layers.append(DecoderLayer(sh, p, device=device, norm=norm, share_bwd=first,
                                            share_acts=share_acts))
        # input gradients alternate between two buffers (a layer reads the one
        # written by the layer above and writes the other)
        self.dx = [self.layers[0].dX, torch.empty(T, sh.H, dtype=torch.float16, device=self.dev)]
        self.opt = None
        if optimizer_state:
            n = sum(int(x.numel()) for L_ in self.layers for x in (L_.Wqkv, L_.Wo, L_.Wgu, L_.Wd))
            self.opt = torch.empty(3 * n, dtype=torch.float32, device=self.dev)

    def params(self):
        return sum(int(x.numel()) for L_ in self.layers for x in (L_.Wqkv, L_.Wo, L_.Wgu, L_.Wd))

    def _forward(self, l, x, stream):
        L_ = self.layers[l]
        L_.X = x
        L_.forward(stream)
        return L_.Y

    def forward(self, x, stream=None):
        """Forward of one micro-batch through the L layers; returns the output."""
        y = x
        for l in range(self.L):
            y = self._forward(l, y, stream)
        return y

    def backward(self, x, dy, first, stream=None):
        """Backward of the micro-batch whose forward ran last (input x, output
        gradient dy); returns the input gradient (a view of one of the stage's
        two gradient buffers).  ``first``: overwrite the weight gradients
        instead of accumulating."""
        g = dy
        for l in reversed(range(self.L)):
            L_ = self.layers[l]
            if self.act == "ckpt":
                inp = self.layers[l - 1].Y if l > 0 else x
                self._forward(l, inp, stream)            # recover the layer's activations
            L_.dY = g
            L_.dX = self.dx[l & 1]
            L_.accumulate = not first
            L_.backward(stream)
            g = L_.dX
        return g

    def micro_batch(self, x, dy, first, stream=None):
        """Forward and backward of one micro-batch; returns the input gradient."""
        self.forward(x, stream)
        return self.backward(x, dy, first, stream)

    def step(self, xs, dys, stream=None):
        """One step: len(xs) micro-batches, gradients accumulated.  The input
        gradient of the last micro-batch is returned (a view of one of the
        stage's two gradient buffers, overwritten by the next call)."""
        g = None
        for m, (x, dy) in enumerate(zip(xs, dys)):
            g = self.micro_batch(x, dy, first=(m == 0), stream=stream)
        return g
