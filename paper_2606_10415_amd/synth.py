"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module holds no arithmetic of the method: it only draws seeded random
float16 tensors of the workloads' shapes and distributions.  Both the HIP
path and the float64 oracle receive the very same float16 bytes.

Recipe (one ``numpy.random.Generator(PCG64(seed))`` per tensor):
    seed = 1000 * config_index + tensor_index
    tensor_index order: X=0, dY=1, Wqkv=2, Wo=3, Wgu=4, Wd=5, Q=6, K=7, V=8, dO=9
    weights ~ N(0, 0.02^2); activations and upstream gradients ~ N(0, 1)
    drawn as float32 standard normals, scaled, rounded once to float16 (RNE).

The workloads are the decoder-layer shapes of the paper's evaluated models
(Sec. 6.1: LLaMA-2-7B, Baichuan2-13B, Qwen2.5-32B, LLaMA-2-70B) at sequence
length 4096, plus a tiny layer that the float64 oracle finishes in seconds.
"""

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    index: int   # config index used in the seed
    B: int
    S: int
    H: int
    Hq: int
    Hkv: int
    D: int
    F: int

    @property
    def T(self):
        return self.B * self.S

    @property
    def qkv_cols(self):
        return (self.Hq + 2 * self.Hkv) * self.D


WORKLOADS = {
    "tiny": Workload("tiny", 0, B=1, S=256, H=256, Hq=4, Hkv=4, D=64, F=688),
    "llama2-7b": Workload("llama2-7b", 1, B=1, S=4096, H=4096, Hq=32, Hkv=32, D=128, F=11008),
    "baichuan2-13b": Workload("baichuan2-13b", 2, B=1, S=4096, H=5120, Hq=40, Hkv=40, D=128, F=13696),
    "qwen2.5-32b": Workload("qwen2.5-32b", 3, B=1, S=4096, H=5120, Hq=40, Hkv=8, D=128, F=27648),
    "llama2-70b": Workload("llama2-70b", 4, B=2, S=4096, H=8192, Hq=64, Hkv=8, D=128, F=28672),
}

TENSOR_INDEX = {"X": 0, "dY": 1, "Wqkv": 2, "Wo": 3, "Wgu": 4, "Wd": 5,
                "Q": 6, "K": 7, "V": 8, "dO": 9, "Wn1": 10, "Wn2": 11, "bqkv": 12}


@dataclass(frozen=True)
class NormInputs:
    """RMSNorm weights [H] of the attention and FFN inputs, eps, rotary base
    and the QKV projection bias [(Hq + 2 Hkv) d] (Qwen2.5; None for LLaMA-2)."""
    wn1: np.ndarray
    wn2: np.ndarray
    eps: float
    rope_base: float
    bqkv: object = None


# eps and rotary base of the evaluated model families (their published
# configurations): LLaMA-2 and Baichuan2 1e-5 / 1e4 ("llama"), Qwen2.5 1e-6 / 1e6.
NORM_CONSTANTS = {"llama": (1e-5, 10000.0), "qwen": (1e-6, 1000000.0)}


def normal_f16(seed, shape, std=1.0):
    """float16 array of N(0, std^2) samples, drawn as float32 then rounded (RNE)."""
    rng = np.random.Generator(np.random.PCG64(int(seed)))
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return x.astype(np.float16)


def uniform_int_f16(seed, shape, lo, hi):
    """float16 array of integers drawn uniformly from [lo, hi] (exactly representable)."""
    rng = np.random.Generator(np.random.PCG64(int(seed)))
    return rng.integers(lo, hi + 1, size=shape).astype(np.float16)


def layer_inputs(w):
    """X [T,H], dY [T,H] and the four weights ([out, in]) of workload ``w``."""
    base = 1000 * w.index
    t = TENSOR_INDEX
    return {
        "X": normal_f16(base + t["X"], (w.T, w.H)),
        "dY": normal_f16(base + t["dY"], (w.T, w.H)),
        "Wqkv": normal_f16(base + t["Wqkv"], (w.qkv_cols, w.H), 0.02),
        "Wo": normal_f16(base + t["Wo"], (w.H, w.Hq * w.D), 0.02),
        "Wgu": normal_f16(base + t["Wgu"], (2 * w.F, w.H), 0.02),
        "Wd": normal_f16(base + t["Wd"], (w.H, w.F), 0.02),
    }


def norm_inputs(w, family="llama"):
    """RMSNorm weights 1 + N(0, 0.1^2) (float16) for workload ``w``, the
    family's eps and rotary base, and for "qwen" a QKV bias N(0, 0.5^2)."""
    base = 1000 * w.index
    t = TENSOR_INDEX
    eps, rope_base = NORM_CONSTANTS[family]
    one = lambda seed: (1.0 + normal_f16(seed, (w.H,), 0.1).astype(np.float32)).astype(np.float16)
    bqkv = (normal_f16(base + t["bqkv"], ((w.Hq + 2 * w.Hkv) * w.D,), 0.5) if family == "qwen"
            else None)
    return NormInputs(one(base + t["Wn1"]), one(base + t["Wn2"]), eps, rope_base, bqkv)


def attention_inputs(B, S, Hq, Hkv, D, seed_base=0, qk_std=1.0):
    """Q [B,S,Hq,D], K, V [B,S,Hkv,D], dO [B,S,Hq,D] float16, N(0,1) (Q, K scaled by qk_std)."""
    t = TENSOR_INDEX
    return {
        "Q": normal_f16(seed_base + t["Q"], (B, S, Hq, D), qk_std),
        "K": normal_f16(seed_base + t["K"], (B, S, Hkv, D), qk_std),
        "V": normal_f16(seed_base + t["V"], (B, S, Hkv, D)),
        "dO": normal_f16(seed_base + t["dO"], (B, S, Hq, D)),
    }
