#!/usr/bin/env python3
"""Benchmark: one dense decoder layer forward + backward on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
the 12 layer GEMMs (fwd / dgrad / wgrad of QKV, O, gate/up and down), causal
attention forward and backward, and the SwiGLU gate -- every step a liblt
HIP launch on one stream, inputs resident in HBM before timing starts.

Prints ONE JSON line.  ``value`` is the layer's algorithmic FLOP rate (GEMM
FLOPs + attention forward over the causal triangle + the 4-contraction
attention backward) divided by the measured step time.

    python bench.py [--gpus 1] [--steps 10] [--warmup 3] [--workload llama2-7b]
"""

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2606_10415_amd.synth import WORKLOADS, layer_inputs, norm_inputs  # noqa: E402

PEAK_FP16_TFLOPS = 2516.6     # MI355X dense FP16 MFMA (256 CU x 2.4 GHz x 4096 FLOP/clk)
PEAK_HBM_GBS = 8000.0

# HBM traffic of the GEMM kernel at llama2-7b: mean bytes per GEMM call over the
# 12 GEMM calls of one layer step (the paper's layer, SwiGLU in the gate/up and
# down-dgrad epilogues; the gate/up forward runs as a 256x256 dispatch plus a
# half-tile tail dispatch, its weight gradient as a 256x256 dispatch, split-K
# partials of its last wave and their reduction, all counted as their call),
# from two rocprofv3 --pmc runs of this script
# (FETCH_SIZE, then WRITE_SIZE, with --copy-calibration-mib 1024) each scaled by
# what the same counter reads for the calibration copy of known size.  The
# figure holds only for the kernel sources it was measured on: any change to
# them makes bench report traffic as null until the counters are taken again.
GEMM_TRAFFIC = {
    "workload": "llama2-7b",
    "layer": "paper",
    "fuse_swiglu": True,
    "sources_sha256": "28b551bfcc85b63f527c7da3ddeff34891f1f5593ab9b9fe949b55c495b6b5ce",
    "fetch_bytes_per_launch": 675429221,
    "write_bytes_per_launch": 108471157,
}
GEMM_SOURCES = ("paper_2606_10415_amd/csrc/gemm_f16.hip", "paper_2606_10415_amd/csrc/common.hpp",
                "paper_2606_10415_amd/csrc/plan.cpp")


def gemm_sources_sha256():
    h = hashlib.sha256()
    for rel in GEMM_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def gemm_traffic(w, layer, fuse_swiglu):
    t = GEMM_TRAFFIC
    if (t["sources_sha256"] is None or t["workload"] != w.name or t["layer"] != layer
            or t["fuse_swiglu"] != fuse_swiglu or t["sources_sha256"] != gemm_sources_sha256()):
        return None
    return int(t["fetch_bytes_per_launch"] + t["write_bytes_per_launch"])


def layer_flops(w):
    T = w.T
    gemm_fwd = 2 * T * (w.qkv_cols * w.H + w.H * w.Hq * w.D + 2 * w.F * w.H + w.H * w.F)
    pairs = w.S * (w.S + 1) // 2
    attn_fwd = 2 * 2 * w.D * pairs * w.Hq * w.B
    attn_bwd = 4 * 2 * w.D * pairs * w.Hq * w.B
    return {"gemm": 3 * gemm_fwd, "attn_fwd": attn_fwd, "attn_bwd": attn_bwd,
            "total": 3 * gemm_fwd + attn_fwd + attn_bwd}


def host_cpu_model():
    """The host CPU's model name (first entry of /proc/cpuinfo) and logical CPU count."""
    name = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return f"{name} ({os.cpu_count()} logical CPUs visible)"


def cpu_baseline(w, budget_s=20.0):
    """Time the float64 oracle on a bounded sample of the same workload.

    Sample: the first R = min(4096, T) rows of every one of the 12 GEMMs (at
    LLaMA-2-7B every row except in the gate/up and QKV weight gradients,
    whose M is 22016 and 12288: 4.11 of the step's 4.97 TFLOP) and then whole causal
    attention heads, forward and backward at the workload's sequence length,
    one after another until the time passes `budget_s` or every query head
    is done (all of them = the whole layer step at T = 4096).  At least one
    head always runs; the GEMM loop also stops early past `budget_s`.
    Rate = algorithmic FLOPs of the sample / wall time.
    """
    import oracle
    from paper_2606_10415_amd.synth import normal_f16
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = os.cpu_count() or 1
    T = w.T
    R = min(4096, T)
    shapes = [(T, w.qkv_cols, w.H), (T, w.H, w.Hq * w.D), (T, 2 * w.F, w.H), (T, w.H, w.F),
              (w.H, w.F, T), (T, w.F, w.H), (2 * w.F, w.H, T), (T, w.H, 2 * w.F),
              (w.H, w.Hq * w.D, T), (T, w.Hq * w.D, w.H), (w.qkv_cols, w.H, T), (T, w.H, w.qkv_cols)]
    flops = 0
    t_total = 0.0
    for i, (M, N, K) in enumerate(shapes):
        a = normal_f16(90000 + i, (R, K))
        b = normal_f16(90100 + i, (K, N), 0.02)
        t0 = time.perf_counter()
        oracle.gemm(0, 0, 1.0, a, b)
        t_total += time.perf_counter() - t0
        flops += 2 * R * N * K
        if t_total > budget_s:
            break
    S, D = w.S, w.D
    pairs = S * (S + 1) // 2
    heads = 0
    for hh in range(w.Hq):
        q = normal_f16(90200 + 4 * hh, (S, D)); k = normal_f16(90201 + 4 * hh, (S, D))
        v = normal_f16(90202 + 4 * hh, (S, D)); do = normal_f16(90203 + 4 * hh, (S, D))
        t0 = time.perf_counter()
        oracle.attn_head_fwd(q, k, v, 1 / math.sqrt(D), True)
        oracle.attn_head_bwd(q, k, v, do, 1 / math.sqrt(D), True)
        t_total += time.perf_counter() - t0
        flops += 6 * 2 * D * pairs
        heads += 1
        if t_total > budget_s:
            break
    return {"value": flops / t_total / 1e12, "unit": "TFLOP/s", "cores": int(cores),
            "cpu": host_cpu_model(), "kind": "oracle",
            "sample": (f"{w.name}: first {R} rows of each of the 12 layer GEMMs + {heads} of "
                       f"{w.Hq} causal attention heads fwd+bwd (S={S}, d={D}); "
                       f"{flops / 1e9:.1f} GFLOP in {t_total:.1f} s, float64 numpy/OpenBLAS")}


def sweep():
    """Sweeps beside the headline step, one JSON line each (stdout):

    * attention forward / backward at the sequence lengths of the paper's
      attention-BP comparison (LLaMA-2-7B heads at S = 1024, 2048, 4096;
      Qwen2.5-32B heads at S = 2048), B = 1, causal: the default pair
      (lt_attn_fwd, then lt_attn_bwd recomputing P) beside the saved-P pair
      of Algorithm 1 (lt_attn_fwd_p stores P, lt_attn_bwd_p reads it);
    * the paper's representative GEMM shapes (Sec. 6.6, Table "Representative
      FP16 GEMM backend profile", sequence length 2048): M = 2048 tokens,
      K x N = 4096x4096, 4096x11008, 11008x4096, 6656x6656, 8192x8192, as the
      forward projection C = X W^T through lt_gemm_f16_ws with the split-K
      workspace the library asks for (the call the layer makes);
    * the whole LLaMA-2-7B-shaped layer step at S = 1024 and 2048.

    Inputs are seeded normal tensors made on the device (timing only).
    """
    import dataclasses
    import torch
    from paper_2606_10415_amd import lt
    from paper_2606_10415_amd.layer import DecoderLayer

    gen = torch.Generator(device="cuda")
    gen.manual_seed(12345)

    def rand(*shape, std=1.0):
        return (torch.randn(*shape, device="cuda", generator=gen) * std).half()

    def timed(fn, iters=10, warm=3):
        for _ in range(warm):
            fn()
        torch.cuda.synchronize()
        s = torch.cuda.Event(enable_timing=True)
        e = torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(iters):
            fn()
        e.record()
        torch.cuda.synchronize()
        return s.elapsed_time(e) / iters

    def emit(d):
        print(json.dumps(d), flush=True)

    for name, B, S, Hq, Hkv, D in [("llama2-7b", 1, 1024, 32, 32, 128),
                                   ("llama2-7b", 1, 2048, 32, 32, 128),
                                   ("llama2-7b", 1, 4096, 32, 32, 128),
                                   ("qwen2.5-32b", 1, 2048, 40, 8, 128)]:
        T, W = B * S, (Hq + 2 * Hkv) * D
        QKV, dO = rand(T, W), rand(T, Hq * D)
        O = torch.empty(T, Hq * D, dtype=torch.float16, device="cuda")
        dQKV = torch.empty_like(QKV)
        LSE = torch.empty(B, Hq, S, dtype=torch.float32, device="cuda")
        wsb = lt.lt_attn_bwd_workspace_size(B, S, Hq, Hkv, D, 1)
        ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
        p, dp, sc = QKV.data_ptr(), dQKV.data_ptr(), 1.0 / math.sqrt(D)
        q, k, v = p, p + 2 * Hq * D, p + 2 * (Hq + Hkv) * D
        dq, dk, dv = dp, dp + 2 * Hq * D, dp + 2 * (Hq + Hkv) * D
        fwd = lambda: lt.lt_attn_fwd(q, k, v, W, W, O, Hq * D, LSE, B, S, Hq, Hkv, D, sc, 1)
        bwd = lambda: lt.lt_attn_bwd(q, k, v, W, W, O, dO, Hq * D, LSE, dq, dk, dv, W, W, ws, wsb,
                                     B, S, Hq, Hkv, D, sc, 1)
        fwd()
        pairs = S * (S + 1) // 2 * Hq * B
        tf, tb = timed(fwd), timed(bwd)
        # saved P (its own workspace; P is 2 bytes per kept (query, key) pair)
        pbytes = lt.lt_attn_p_size(B, S, Hq, 1)
        P = torch.empty(pbytes, dtype=torch.uint8, device="cuda")
        wpb = lt.lt_attn_bwd_p_workspace_size(B, S, Hq, Hkv, D)
        wsp = torch.empty(wpb, dtype=torch.uint8, device="cuda")
        fwdp = lambda: lt.lt_attn_fwd_p(q, k, v, W, W, O, Hq * D, LSE, P, pbytes, B, S, Hq, Hkv, D,
                                        sc, 1)
        bwdp = lambda: lt.lt_attn_bwd_p(q, k, v, W, W, O, dO, Hq * D, LSE, P, pbytes, dq, dk, dv,
                                        W, W, wsp, wpb, B, S, Hq, Hkv, D, sc, 1)
        fwdp()
        tfp, tbp = timed(fwdp), timed(bwdp)
        emit({"sweep": "attention", "workload": name, "B": B, "S": S, "Hq": Hq, "Hkv": Hkv, "D": D,
              "fwd_ms": round(tf, 4), "fwd_tflops": round(4 * D * pairs / tf / 1e9, 1),
              "bwd_ms": round(tb, 4), "bwd_tflops": round(8 * D * pairs / tb / 1e9, 1),
              "bwd_frac_peak": round(8 * D * pairs / tb / 1e9 / PEAK_FP16_TFLOPS, 4),
              "saved_p": {"fwd_p_ms": round(tfp, 4), "bwd_p_ms": round(tbp, 4),
                          "p_mib": round(pbytes / 2**20, 1),
                          "fwd_bwd_ms": round(tfp + tbp, 4),
                          "recompute_fwd_bwd_ms": round(tf + tb, 4)}})
        del QKV, dO, O, dQKV, ws, P, wsp

    M = 2048
    for K, N in [(4096, 4096), (4096, 11008), (11008, 4096), (6656, 6656), (8192, 8192)]:
        A, Wt = rand(M, K), rand(N, K, std=0.02)
        C = torch.empty(M, N, dtype=torch.float16, device="cuda")
        gwb = lt.lt_gemm_f16_workspace_size(0, 1, M, N, K)
        gws = torch.empty(gwb, dtype=torch.uint8, device="cuda") if gwb else None
        t = timed(lambda: lt.lt_gemm_f16_ws(0, 1, M, N, K, 1.0, A, K, Wt, K, 0.0, None, N, None, C,
                                            N, gws, gwb), iters=20)
        tfl = 2 * M * N * K / t / 1e9
        emit({"sweep": "gemm", "M": M, "K": K, "N": N, "layout": "NT (X W^T)", "ms": round(t, 4),
              "tflops": round(tfl, 1), "frac_peak": round(tfl / PEAK_FP16_TFLOPS, 4),
              "split_k_workspace_mib": round(gwb / 2**20, 1)})
        del A, Wt, C, gws

    base = WORKLOADS["llama2-7b"]
    for S in (1024, 2048):
        w = dataclasses.replace(base, name=f"llama2-7b-s{S}", S=S)
        L = DecoderLayer(w, layer_inputs(w))
        t = timed(L.step, iters=10)
        fl = layer_flops(w)
        emit({"sweep": "layer", "workload": w.name, "B": w.B, "S": S, "ms_per_step": round(t, 4),
              "tflops": round(fl["total"] / t / 1e9, 1),
              "frac_peak": round(fl["total"] / t / 1e9 / PEAK_FP16_TFLOPS, 4)})
        del L


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama2-7b", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--layer", default="paper", choices=["paper", "full"],
                    help="paper: the layer of the paper's hot path (projections, attention, "
                         "SwiGLU, residuals); full: plus the evaluated models' RMSNorm and "
                         "rotary embedding (same FLOP count, longer step)")
    ap.add_argument("--fuse-swiglu", type=int, default=1, choices=[0, 1],
                    help="1: SwiGLU in the gate/up GEMM and down-dgrad GEMM epilogues; "
                         "0: separate SwiGLU kernels")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the headline step, print the sequence / GEMM-shape sweeps "
                         "(one JSON line each)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="before warmup, run a plain elementwise copy (negation) of this many "
                         "MiB of fp16 three times: the reference dispatch for scaling HBM "
                         "byte counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU (its layer at full shape); --gpus {args.gpus} is not "
              "supported: the data-parallel path needs no collective inside a layer step and "
              "this build runs on one MI355X only", file=sys.stderr)
        sys.exit(2)

    import torch
    assert torch.cuda.is_available(), "bench.py needs a ROCm GPU"
    from paper_2606_10415_amd.layer import DecoderLayer
    if args.sweep:
        sweep()
        return

    w = WORKLOADS[args.workload]
    print(f"[bench] workload {w.name}: generating inputs", file=sys.stderr, flush=True)
    full = args.layer == "full"
    norm = norm_inputs(w, "qwen" if w.name.startswith("qwen") else "llama") if full else None
    L = DecoderLayer(w, layer_inputs(w), norm=norm, fuse_swiglu=bool(args.fuse_swiglu))
    stream = torch.cuda.current_stream()
    fl = layer_flops(w)

    if args.copy_calibration_mib > 0:
        n = args.copy_calibration_mib * (1 << 20) // 2
        src = torch.empty(n, dtype=torch.float16, device="cuda").normal_()
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        print(f"[bench] calibration copy: {n * 2} bytes read and {n * 2} written per dispatch",
              file=sys.stderr, flush=True)
        del src, dst

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        L.step()
    torch.cuda.synchronize()

    # timed region: events around every launch, on the stream the kernels run on
    names_per_step = []
    events = []

    def hook(name):
        ev = torch.cuda.Event(enable_timing=True)
        ev.record(stream)
        events.append((name, ev))

    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        hook("__step__")
        L.step(hook=hook)
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_total = start.elapsed_time(end)
    ms_per_step = ms_total / args.steps

    step_ms = []
    step_start = None
    for name, ev in events + [("__step__", end)]:
        if name == "__step__":
            if step_start is not None:
                step_ms.append(step_start.elapsed_time(ev))
            step_start = ev

    per_op = {}
    prev = None
    for name, ev in events:
        if prev is not None and name != "__step__":
            per_op.setdefault(name, []).append(prev.elapsed_time(ev))
        prev = ev
    avg = {k: float(np.mean(v)) for k, v in per_op.items()}
    gemm_names = [n for n, *_ in L.gemm_shapes()]
    gemm_ms = sum(avg[n] for n in gemm_names)
    gemm_tflops = fl["gemm"] / (gemm_ms * 1e-3) / 1e12
    attn_bwd_tflops = fl["attn_bwd"] / (avg["attn_bwd"] * 1e-3) / 1e12
    attn_fwd_tflops = fl["attn_fwd"] / (avg["attn_fwd"] * 1e-3) / 1e12
    value = fl["total"] / (ms_per_step * 1e-3) / 1e12

    detail = {
        "gemm_ms": round(gemm_ms, 4), "gemm_tflops": round(gemm_tflops, 1),
        "gemm_frac_peak": round(gemm_tflops / PEAK_FP16_TFLOPS, 4),
        "attn_fwd_ms": round(avg["attn_fwd"], 4), "attn_fwd_tflops": round(attn_fwd_tflops, 1),
        "attn_bwd_ms": round(avg["attn_bwd"], 4), "attn_bwd_tflops": round(attn_bwd_tflops, 1),
        "attn_bwd_frac_peak": round(attn_bwd_tflops / PEAK_FP16_TFLOPS, 4),
        "swiglu": "fused into the gate/up and down-dgrad GEMM epilogues" if L.fuse_swiglu else
                  "separate kernels",
        **({} if L.fuse_swiglu else {
            "swiglu_fwd_ms": round(avg["swiglu_fwd"], 4),
            "swiglu_bwd_ms": round(avg["swiglu_bwd"], 4),
            "swiglu_fwd_gbs": round(6 * w.T * w.F / (avg["swiglu_fwd"] * 1e-3) / 1e9, 1),
            "swiglu_bwd_gbs": round(10 * w.T * w.F / (avg["swiglu_bwd"] * 1e-3) / 1e9, 1)}),
        "step_ms_median": round(float(np.median(step_ms)), 4),
        "step_ms_min": round(float(np.min(step_ms)), 4),
        "step_ms_max": round(float(np.max(step_ms)), 4),
        "per_op_ms": {k: round(v, 4) for k, v in avg.items()},
        **({"rmsnorm_fwd_gbs": round(2 * (4 * w.T * w.H) / ((avg["rmsnorm1_fwd"] + avg["rmsnorm2_fwd"]) * 1e-3) / 1e9, 1),
            "rmsnorm_bwd_gbs": round(2 * (8 * w.T * w.H) / ((avg["rmsnorm1_bwd"] + avg["rmsnorm2_bwd"]) * 1e-3) / 1e9, 1),
            "rope_gbs": round(2 * (4 * w.T * (w.Hq + w.Hkv) * w.D) / ((avg["rope_fwd"] + avg["rope_bwd"]) * 1e-3) / 1e9, 1)}
           if full else {}),
        **({"qkv_bias_grad_gbs": round(2 * w.T * w.qkv_cols / (avg["qkv_bias_grad"] * 1e-3) / 1e9, 1)}
           if "qkv_bias_grad" in avg else {}),
        "wall_s": round(wall, 3),
    }
    print("[bench] " + json.dumps(detail), file=sys.stderr, flush=True)

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (oracle sample)", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w)

    out = {
        "metric": "decoder-layer fwd+bwd TFLOP/s (GEMM, attn-bwd) and % of FP16 MFMA peak",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic (seeded N(0,1) activations/grads, N(0,0.02^2) weights, fp16)",
        "config": {"workload": f"{w.name} decoder layer fwd+bwd"
                               + ((" (with RMSNorm, rotary embedding and QKV bias)"
                                   if L.bqkv is not None else
                                   " (with RMSNorm and rotary embedding)") if full else ""),
                   "B": w.B, "S": w.S, "H": w.H,
                   "Hq": w.Hq, "Hkv": w.Hkv, "D": w.D, "F": w.F, "causal": True,
                   "flops_per_step": fl["total"], "parallelism": "single GPU"},
        "frac_of_peak": round(value / PEAK_FP16_TFLOPS, 4),
        "roofline": {"bound": "mfma", "kernel": "gemm_f16 (12 GEMM calls per step, two with the SwiGLU epilogues; achieved and traffic are per call; the gate/up forward adds a half-tile tail launch, the gate/up weight gradient a split-K last wave and its reduction)",
                     "achieved": round(gemm_tflops, 1), "peak": PEAK_FP16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(gemm_tflops / PEAK_FP16_TFLOPS, 4),
                     "traffic": gemm_traffic(w, args.layer, L.fuse_swiglu)},
        "attn_bwd": {"achieved": round(attn_bwd_tflops, 1), "peak": PEAK_FP16_TFLOPS,
                     "frac": round(attn_bwd_tflops / PEAK_FP16_TFLOPS, 4)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
