"""Resource-aware configuration planner for MI355X nodes (Sec. 4.4, Algorithm 2).

A candidate training configuration is c = (P, D, Z, b, A, act, pref)
(Sec. 4.4, Eq. config): pipeline degree P, data-parallel degree D, ZeRO stage
Z, micro-batch b, gradient-accumulation steps A, activation policy act
("full", "ckpt" or "fsr") and state-task policy pref ("layerwise": gradient
sync, update and parameter-view prefetch run per layer inside the windows of
Sec. 4.2; "bulk": at the accumulation boundary).  For each candidate the
planner

  1. partitions the layers into P contiguous stages,
  2. estimates each stage's peak memory M_p = M_state + M_act + M_buf
     (Eq. planner-memory) and drops the candidate if max_p M_p exceeds the
     budget (Eq. planner-memory-constraint),
  3. estimates the step time T_step = T_1F1B + E_comm + E_upd + E_pref +
     E_rec (Eq. planner-step-time), every exposure being
     E_x = max(0, T_x - W_x) (Eq. exposed-latency),

and returns the feasible candidate with the least T_step (Eq.
planner-objective).  The inputs are the three profiles of the paper: a model
profile (layer shapes), a platform profile (HBM capacity and bandwidth, link
and collective bandwidths of one MI355X node) and an execution profile (the
measured forward and backward time of one layer of this library at the
candidate's micro-batch and sequence length).

Terms the paper leaves open are fixed here (each is one line of the
design notes):
  * memory per parameter: FP16 weights (2 B), FP16 gradients (2 B), FP32
    master weights and two Adam moments (12 B); ZeRO stage Z >= 1 shards the
    optimizer states over D, Z >= 2 also the gradients, Z = 3 also the
    weights (whose layer views are then gathered into prefetch buffers);
  * N_act(p) = min(P - p, A) micro-batches resident at stage p under 1F1B;
    M_full = the tensors one layer keeps for its backward, M_ckpt = the
    layer input, M_rec = one layer's full activations (Eqs. act-full,
    act-fsr);
  * T_1F1B is the exact makespan of the non-interleaved 1F1B schedule with
    the stages' micro-batch times and one stage-boundary transfer per hop,
    evaluated as the longest path of the schedule's dependency graph;
  * checkpointing recovers in the backward slot (its recompute lengthens the
    stage's backward time); FSR recovers in the stage's idle time of the
    1F1B timeline, and only the part that does not fit is exposed (Eq.
    recovery-exposure);
  * "layerwise": a stage's gradient sync hides under the backward of its
    last micro-batch and the update/prefetch chain under that backward plus
    the stage's pipeline-fill wait of the next step; "bulk": no window.

Everything here is host arithmetic; the layer times come from running the
library's kernels (``measure_layer_profile``).
"""

from dataclasses import dataclass, field, replace
import functools
import math


# ----------------------------------------------------------------- profiles
@dataclass(frozen=True)
class ModelProfile:
    """Dense decoder-only model: layer shapes (Sec. 6.1's models)."""
    name: str
    layers: int
    H: int
    Hq: int
    Hkv: int
    D: int
    F: int
    vocab: int
    qkv_bias: bool = False
    norm: bool = True      # RMSNorm + rotary layer (False: the paper's bare layer)

    @property
    def qkv_cols(self):
        return (self.Hq + 2 * self.Hkv) * self.D

    @property
    def layer_params(self):
        p = (self.qkv_cols * self.H + self.H * self.Hq * self.D + 2 * self.F * self.H
             + self.H * self.F + (2 * self.H if self.norm else 0))
        return p + (self.qkv_cols if self.qkv_bias else 0)

    @property
    def embed_params(self):
        return self.vocab * self.H            # input embedding (stage 0)

    @property
    def head_params(self):
        return self.vocab * self.H + (self.H if self.norm else 0)   # final norm + output head

    @property
    def params(self):
        return self.layers * self.layer_params + self.embed_params + self.head_params

    def act_full(self, b, S):
        """Bytes one layer keeps for its backward, per micro-batch (FP16 unless
        noted): input X, QKV, O, LSE (FP32), H1, GU, A, and with norms the
        normed Xn, H1n and the two RMSNorm row factors (FP32)."""
        T = b * S
        half = T * (self.H + self.qkv_cols + self.Hq * self.D + self.H + 2 * self.F + self.F)
        extra = 2 * T * 2 * self.H + 4 * 2 * T if self.norm else 0
        return 2 * half + 4 * b * self.Hq * S + extra

    def act_ckpt(self, b, S):
        """Checkpoint of one layer: its input X."""
        return 2 * b * S * self.H

    def gemm_workspace(self, b, S):
        """FP32 split-K workspace of the layer's GEMMs (the largest any of its 10
        plain GEMM shapes asks the library for; one at a time on the stream; the
        gate/up forward and the down-projection input gradient run with the
        fused SwiGLU epilogues, which take none)."""
        from . import lt
        T, Hd = b * S, self.Hq * self.D
        shapes = [(T, self.qkv_cols, self.H), (T, self.H, Hd),
                  (T, self.H, self.F), (self.H, self.F, T),
                  (2 * self.F, self.H, T), (T, self.H, 2 * self.F), (self.H, Hd, T),
                  (T, Hd, self.H), (self.qkv_cols, self.H, T), (T, self.H, self.qkv_cols)]
        return max(lt.lt_gemm_f16_workspace_size(0, 0, M, N, K) for M, N, K in shapes)

    def bwd_work(self, b, S):
        """Short-lived buffers of one layer's backward, shared by a stage's
        layers: dA, dGU, dH1, dO, dQKV, two input-gradient buffers (a layer
        reads one and writes the other), with norms the two normed-input
        gradients, the attention workspace (D and the base-2 LSE, FP32, plus
        FP32 partial dK, dV when a GQA group's query heads are split over
        several workgroups) and the GEMMs' split-K workspace."""
        T = b * S
        half = T * (self.F + 2 * self.F + self.H + self.Hq * self.D + self.qkv_cols + 2 * self.H
                    + (2 * self.H if self.norm else 0))
        from . import lt
        attn_ws = lt.lt_attn_bwd_workspace_size(b, S, self.Hq, self.Hkv, self.D, 1)
        return 2 * half + attn_ws + self.gemm_workspace(b, S)


MODELS = {
    "llama2-7b": ModelProfile("llama2-7b", 32, 4096, 32, 32, 128, 11008, 32000),
    "baichuan2-13b": ModelProfile("baichuan2-13b", 40, 5120, 40, 40, 128, 13696, 125696),
    "qwen2.5-32b": ModelProfile("qwen2.5-32b", 64, 5120, 40, 8, 128, 27648, 152064, True),
    "llama2-70b": ModelProfile("llama2-70b", 80, 8192, 64, 8, 128, 28672, 32000),
}


@dataclass(frozen=True)
class PlatformProfile:
    """One node of MI355X GPUs.  Bandwidths in bytes/s."""
    name: str = "MI355X"
    gpus: int = 8
    hbm_bytes: float = 288e9
    reserve_bytes: float = 8e9       # runtime, code objects, allocator slack
    hbm_bw: float = 5.5e12           # achieved streaming rate (elementwise kernels)
    p2p_bw: float = 64e9             # one xGMI link, one direction (stage boundary)
    allreduce_busbw: float = 300e9   # collective bus bandwidth over the node

    @property
    def budget(self):
        return self.hbm_bytes - self.reserve_bytes


@dataclass(frozen=True)
class ExecProfile:
    """Measured per-layer times (seconds) keyed by (micro-batch, sequence)."""
    t_fwd: dict
    t_bwd: dict

    def layer(self, b, S):
        return self.t_fwd[(b, S)], self.t_bwd[(b, S)]


@dataclass(frozen=True)
class Config:
    P: int
    D: int
    Z: int
    b: int
    A: int
    act: str = "full"
    pref: str = "layerwise"


# ----------------------------------------------------------------- memory
def partition(layers, P):
    """Contiguous stages; the first L mod P stages take one extra layer."""
    base, extra = divmod(layers, P)
    return [base + (1 if p < extra else 0) for p in range(P)]


def stage_params(model, c, p):
    n = partition(model.layers, c.P)[p] * model.layer_params
    if p == 0:
        n += model.embed_params
    if p == c.P - 1:
        n += model.head_params
    return n


def n_act(c, p):
    """Micro-batches whose activations stage p holds under 1F1B."""
    return min(c.P - p, c.A)


def stage_memory(model, c, p, S):
    """M_p(c) = M_state + M_act + M_buf in bytes (Eq. planner-memory)."""
    n = stage_params(model, c, p)
    D = c.D
    w = 2.0 / D if c.Z >= 3 else 2.0
    g = 2.0 / D if c.Z >= 2 else 2.0
    o = 12.0 / D if c.Z >= 1 else 12.0
    m_state = n * (w + g + o)
    L_p = partition(model.layers, c.P)[p]
    if c.act == "full":
        m_act = n_act(c, p) * L_p * model.act_full(c.b, S)
    else:                                    # ckpt and FSR: checkpoints + one recovery buffer
        m_act = n_act(c, p) * L_p * model.act_ckpt(c.b, S) + model.act_full(c.b, S)
    m_buf = model.bwd_work(c.b, S)
    if c.P > 1:
        m_buf += 2 * 2 * c.b * S * model.H   # stage-boundary send / receive buffers
    if c.Z >= 3:                             # gathered working views of the weights
        views = 2 if c.pref == "layerwise" else L_p
        m_buf += views * 2 * model.layer_params
    if D > 1:                                # gradient-sync buckets (one layer, double-buffered)
        m_buf += 2 * 2 * model.layer_params
    return {"state": m_state, "act": m_act, "buf": m_buf, "total": m_state + m_act + m_buf}


# ----------------------------------------------------------------- time
def one_f_one_b_time(P, A, t_f, t_b, t_x):
    """Makespan of non-interleaved 1F1B: the longest path of the schedule's
    dependency graph.  Nodes are the tasks of each stage in 1F1B order; a task
    follows the previous task of its stage, a forward follows the previous
    stage's forward of its micro-batch (+ t_x), a backward follows its own
    forward and the next stage's backward of its micro-batch (+ t_x)."""
    orders = []
    for p in range(P):
        warm = min(P - 1 - p, A)
        seq = [("F", m) for m in range(warm)]
        f, bk = warm, 0
        while f < A:
            seq += [("F", f), ("B", bk)]
            f += 1
            bk += 1
        seq += [("B", m) for m in range(bk, A)]
        orders.append(seq)
    index = [{task: i for i, task in enumerate(o)} for o in orders]

    @functools.lru_cache(maxsize=None)
    def finish(p, i):
        kind, m = orders[p][i]
        ready = finish(p, i - 1) if i > 0 else 0.0
        if kind == "F":
            if p > 0:
                ready = max(ready, finish(p - 1, index[p - 1][("F", m)]) + t_x)
            return ready + t_f[p]
        ready = max(ready, finish(p, index[p][("F", m)]))
        if p < P - 1:
            ready = max(ready, finish(p + 1, index[p + 1][("B", m)]) + t_x)
        return ready + t_b[p]

    # evaluate in an order that keeps the recursion shallow
    for depth in range(2 * A):
        for p in range(P):
            if depth < len(orders[p]):
                finish(p, depth)
    return max(finish(p, len(orders[p]) - 1) for p in range(P))


def step_time(model, plat, prof, c, S):
    """T_step(c) and its terms in seconds (Eq. planner-step-time)."""
    tf1, tb1 = prof.layer(c.b, S)
    L = partition(model.layers, c.P)
    t_f = [L[p] * tf1 for p in range(c.P)]
    t_rec = [L[p] * tf1 for p in range(c.P)]            # recompute = the stage's forward
    t_b = [L[p] * tb1 + (t_rec[p] if c.act == "ckpt" else 0.0) for p in range(c.P)]
    t_x = 2 * c.b * S * model.H / plat.p2p_bw if c.P > 1 else 0.0
    t_1f1b = one_f_one_b_time(c.P, c.A, t_f, t_b, t_x)

    e_rec = 0.0
    if c.act == "fsr":
        for p in range(c.P):
            idle = t_1f1b - c.A * (t_f[p] + t_b[p])       # W_rec: the stage's idle time
            e_rec = max(e_rec, max(0.0, c.A * t_rec[p] - idle))

    e_comm = e_upd = e_pref = 0.0
    for p in range(c.P):
        n = stage_params(model, c, p)
        grad_bytes = 2.0 * n
        if c.D > 1:
            frac = (c.D - 1) / c.D
            t_comm = (1 if c.Z >= 2 else 2) * frac * grad_bytes / plat.allreduce_busbw
        else:
            t_comm = 0.0
        shard = n / c.D if c.Z >= 1 else n
        t_upd = shard * (2 + 24 + 2) / plat.hbm_bw     # read grad, r/w master+m+v, write weight
        t_pref = ((c.D - 1) / c.D * 2.0 * n / plat.allreduce_busbw
                  if (c.Z >= 3 and c.D > 1) else 0.0)
        if c.pref == "layerwise":
            w_comm = t_b[p]                               # the last micro-batch's backward
            w_chain = t_b[p] + p * t_f[p]                 # ... plus next step's fill wait
        else:
            w_comm = w_chain = 0.0
        e_c = max(0.0, t_comm - w_comm)
        e_comm = max(e_comm, e_c)
        left = max(0.0, w_chain - t_comm)                 # window the sync leaves over
        e_u = max(0.0, t_upd - left)
        e_upd = max(e_upd, e_u)
        e_pref = max(e_pref, max(0.0, t_pref - max(0.0, left - t_upd)))
    total = t_1f1b + e_comm + e_upd + e_pref + e_rec
    return {"T_1F1B": t_1f1b, "E_comm": e_comm, "E_upd": e_upd, "E_pref": e_pref, "E_rec": e_rec,
            "T_step": total}


# ----------------------------------------------------------------- search
def candidates(model, plat, gpus, global_batch, micro_batches=(1, 2, 4),
               acts=("full", "ckpt", "fsr"), prefs=("layerwise", "bulk")):
    """The search space C: every (P, D) with P * D = gpus and P <= layers,
    ZeRO 0-3, micro-batch b and A = global_batch / (b D) when integral."""
    for P in range(1, min(gpus, model.layers) + 1):
        if gpus % P:
            continue
        D = gpus // P
        for b in micro_batches:
            if global_batch % (b * D):
                continue
            A = global_batch // (b * D)
            for Z in range(4):
                if Z > 0 and D == 1:
                    continue
                for act in acts:
                    for pref in prefs:
                        yield Config(P, D, Z, b, A, act, pref)


def plan(model, plat, prof, S, gpus, global_batch, space=None):
    """Algorithm 2: prune by memory, estimate the step time, keep the best.
    Returns (best (config, T_step, terms, per-stage memory) or None, feasible list)."""
    feasible = []
    for c in (space if space is not None else candidates(model, plat, gpus, global_batch)):
        if (c.b, S) not in prof.t_fwd:
            continue
        mem = [stage_memory(model, c, p, S) for p in range(c.P)]
        if max(m["total"] for m in mem) > plat.budget:
            continue
        terms = step_time(model, plat, prof, c, S)
        feasible.append((c, terms["T_step"], terms, mem))
    if not feasible:
        return None, feasible
    return min(feasible, key=lambda r: r[1]), feasible


def min_feasible_gpus(model, plat, prof, S, global_batch, max_gpus=64):
    """Smallest GPU count with a memory-feasible configuration (the paper's
    minimum-resource search), and the best plan at that count."""
    for g in range(1, max_gpus + 1):
        best, _ = plan(model, replace(plat, gpus=g), prof, S, g, global_batch)
        if best is not None:
            return g, best
    return None, None


# ----------------------------------------------------------------- measurement
def measure_layer_profile(model, b, S, layers=8, reps=3, device="cuda"):
    """Forward and backward seconds of one layer of ``model`` at (b, S), run by
    this library's kernels inside a stage of ``layers`` layers (each with its
    own weights, one micro-batch, forward then backward) and averaged over
    them: the way the layers run in training.  With ``model.norm`` the layers
    are the full LLaMA/Qwen layers (RMSNorm, rotary embedding, the QKV bias
    where the model has one), else the paper's bare layer; SwiGLU fused in
    both."""
    import numpy as np
    import torch
    from .stage import Stage
    from .synth import Workload, norm_inputs
    w = Workload(f"{model.name}-b{b}-s{S}", 20 + b, B=b, S=S, H=model.H, Hq=model.Hq,
                 Hkv=model.Hkv, D=model.D, F=model.F)
    fam = "qwen" if model.qkv_bias else "llama"
    st = Stage(w, layers, act="full", device=device, seed=11,
               norm=norm_inputs(w, fam) if model.norm else None)
    gen = torch.Generator(device=device)
    gen.manual_seed(3)
    x = torch.randn(b * S, model.H, generator=gen, device=device).half()
    dy = torch.randn(b * S, model.H, generator=gen, device=device).half()
    stream = torch.cuda.current_stream()
    st.micro_batch(x, dy, first=True)                    # warm-up
    torch.cuda.synchronize()
    tf, tb = [], []
    for _ in range(reps):
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        e0.record(stream)
        st.forward(x)
        e1.record(stream)
        st.backward(x, dy, first=True)
        e2.record(stream)
        torch.cuda.synchronize()
        tf.append(e0.elapsed_time(e1) * 1e-3 / layers)
        tb.append(e1.elapsed_time(e2) * 1e-3 / layers)
    del st
    torch.cuda.empty_cache()
    return float(np.median(tf)), float(np.median(tb))


def validate(configs, reps=2, device="cuda", log=print):
    """Predicted against measured step time and peak memory of single-GPU
    stages (P = D = 1; Sec. 6's planner-accuracy check).  ``configs``: tuples
    (model name, layers L, b, S, A, act).  The stage runs the paper's bare
    layer (``stage.Stage``); the prediction uses the one-layer times measured
    here and the planner's memory model of L such layers with their optimizer
    states.  The optimizer update itself is not run, so the predicted time is
    T_1F1B (+ E_rec), without E_upd."""
    import json
    import time
    import torch
    from .stage import Stage
    from .synth import Workload
    out = []
    profiles = {}
    for name, L, b, S, A, act in configs:
        base = MODELS[name]
        m = replace(base, layers=L, vocab=0, norm=False, qkv_bias=False)
        key = (name, b, S)
        if key not in profiles:
            profiles[key] = measure_layer_profile(m, b, S, device=device)
        tf1, tb1 = profiles[key]
        prof = ExecProfile({(b, S): tf1}, {(b, S): tb1})
        c = Config(1, 1, 0, b, A, act)
        terms = step_time(m, PlatformProfile(), prof, c, S)
        pred_t = terms["T_1F1B"] + terms["E_rec"]
        pred_m = stage_memory(m, c, 0, S)["total"]

        w = Workload(f"{name}-stage", 40, B=b, S=S, H=m.H, Hq=m.Hq, Hkv=m.Hkv, D=m.D, F=m.F)
        T = b * S
        gen = torch.Generator(device=device)
        gen.manual_seed(7)
        xs = [torch.randn(T, m.H, generator=gen, device=device).half() for _ in range(A)]
        dys = [torch.randn(T, m.H, generator=gen, device=device).half() for _ in range(A)]
        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats()
        base_mem = torch.cuda.memory_allocated()
        t0 = time.perf_counter()
        st = Stage(w, L, act=act, device=device, optimizer_state=True)
        log(f"[planner] {name} L={L} b={b} S={S} A={A} {act}: stage built in "
            f"{time.perf_counter() - t0:.1f} s")
        st.step(xs, dys)                                  # warm-up step
        torch.cuda.synchronize()
        times = []
        stream = torch.cuda.current_stream()
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            st.step(xs, dys)
            e1.record(stream)
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1) * 1e-3)
        meas_t = min(times)
        meas_m = torch.cuda.max_memory_allocated() - base_mem
        rec = {"model": name, "layers": L, "b": b, "S": S, "A": A, "act": act,
               "layer_fwd_ms": round(tf1 * 1e3, 4), "layer_bwd_ms": round(tb1 * 1e3, 4),
               "pred_ms": round(pred_t * 1e3, 2), "meas_ms": round(meas_t * 1e3, 2),
               "time_err_pct": round(100 * (pred_t - meas_t) / meas_t, 2),
               "pred_mem_gb": round(pred_m / 1e9, 3), "meas_mem_gb": round(meas_m / 1e9, 3),
               "mem_err_pct": round(100 * (pred_m - meas_m) / meas_m, 2)}
        log(json.dumps(rec))
        out.append(rec)
        del st
        torch.cuda.empty_cache()
    return out


def _main():
    import argparse
    import json
    ap = argparse.ArgumentParser(description="resource-aware configuration planner")
    ap.add_argument("--validate", action="store_true",
                    help="measure single-GPU stages and compare with the planner's prediction")
    ap.add_argument("--plan", action="store_true",
                    help="plan every evaluated model on one node from measured layer times")
    ap.add_argument("--seq", type=int, default=2048)
    ap.add_argument("--global-batch", type=int, default=64)
    args = ap.parse_args()
    if args.validate:
        validate([("llama2-7b", 32, 1, 4096, 1, "full"), ("llama2-7b", 32, 1, 4096, 4, "full"),
                  ("llama2-7b", 32, 1, 4096, 4, "ckpt"), ("llama2-7b", 32, 2, 2048, 2, "full"),
                  ("qwen2.5-32b", 16, 1, 4096, 2, "full"), ("qwen2.5-32b", 16, 1, 4096, 2, "ckpt")])
    if args.plan:
        plat = PlatformProfile()
        for name, m in MODELS.items():
            prof_f, prof_b = {}, {}
            for b in (1, 2, 4):
                tf1, tb1 = measure_layer_profile(m, b, args.seq)
                prof_f[(b, args.seq)], prof_b[(b, args.seq)] = tf1, tb1
            prof = ExecProfile(prof_f, prof_b)
            best, feas = plan(m, plat, prof, args.seq, plat.gpus, args.global_batch)
            gmin, best_min = min_feasible_gpus(m, plat, prof, args.seq, args.global_batch, 8)
            rec = {"model": name, "gpus": plat.gpus, "seq": args.seq,
                   "global_batch": args.global_batch, "feasible": len(feas),
                   "min_gpus": gmin}
            if best is not None:
                c, t, terms, mem = best
                rec.update({"best": c.__dict__, "T_step_ms": round(t * 1e3, 2),
                            "tokens_per_s": round(args.global_batch * args.seq / t, 1),
                            "terms_ms": {k: round(v * 1e3, 3) for k, v in terms.items()},
                            "max_stage_mem_gb": round(max(x["total"] for x in mem) / 1e9, 2)})
            print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    _main()
