"""CPU checks of the resource-aware planner (Sec. 4.4, Algorithm 2).

* The model profiles reproduce the published parameter counts of the four
  evaluated models (LLaMA-2-7B/70B exactly, Baichuan2-13B and Qwen2.5-32B to
  the published totals).
* T_1F1B (the planner's longest path over the schedule graph) equals the
  oracle's discrete-event simulation on random stage times and transfers,
  and N_act(p) equals the simulated residency.
* Memory: closed forms of the state term per ZeRO stage; checkpointing never
  needs more activation memory than full-save; the budget prunes.
* Algorithm 2: plan() returns the least step time over exactly the feasible
  candidates of the space (brute force over the same space).
* Exposures are never negative; FSR recovery is free when the stage's idle
  time covers it and fully exposed on a single stage.
"""

import numpy as np
import pytest

import oracle
from paper_2606_10415_amd.planner import (MODELS, Config, ExecProfile, PlatformProfile, candidates,
                                          n_act, one_f_one_b_time, partition, plan, stage_memory,
                                          step_time)


def test_published_parameter_counts():
    assert MODELS["llama2-7b"].params == 6_738_415_616
    assert MODELS["llama2-70b"].params == 68_976_648_192
    assert MODELS["baichuan2-13b"].params == pytest.approx(13.9e9, rel=5e-3)
    assert MODELS["qwen2.5-32b"].params == pytest.approx(32.76e9, rel=5e-3)


@pytest.mark.parametrize("seed", range(12))
def test_1f1b_time_matches_simulation(seed):
    rng = np.random.default_rng(seed)
    P, A = int(rng.integers(1, 9)), int(rng.integers(1, 17))
    tf, tb = rng.uniform(0.2, 2, P), rng.uniform(0.4, 4, P)
    tx = float(rng.uniform(0, 0.6)) if P > 1 else 0.0
    sim = oracle.simulate_1f1b(P, A, tf, tb, tx)
    assert one_f_one_b_time(P, A, list(tf), list(tb), tx) == pytest.approx(sim["makespan"], rel=1e-12)
    c = Config(P, 1, 0, 1, A)
    assert [n_act(c, p) for p in range(P)] == sim["n_act"]


def test_partition():
    assert partition(32, 1) == [32]
    assert partition(80, 48) == [2] * 32 + [1] * 16
    assert sum(partition(64, 7)) == 64


@pytest.mark.parametrize("Z,D", [(0, 1), (1, 8), (2, 8), (3, 8)])
def test_state_memory_closed_form(Z, D):
    m = MODELS["llama2-7b"]
    c = Config(1, D, Z, 1, 8)
    per = {0: 16.0, 1: 2 + 2 + 12 / D, 2: 2 + 2 / D + 12 / D, 3: 16.0 / D}[Z]
    assert stage_memory(m, c, 0, 4096)["state"] == pytest.approx(per * m.params, rel=1e-12)


def test_checkpointing_needs_less_activation_memory():
    m = MODELS["qwen2.5-32b"]
    for P in (1, 4, 16):
        for p in range(P):
            full = stage_memory(m, Config(P, 1, 0, 1, 8, "full"), p, 2048)["act"]
            ck = stage_memory(m, Config(P, 1, 0, 1, 8, "ckpt"), p, 2048)["act"]
            assert ck <= full


def _toy_profile(b_list=(1, 2, 4), S=2048):
    # synthetic times (seconds) proportional to tokens, for CPU tests
    return ExecProfile({(b, S): 1e-3 * b for b in b_list}, {(b, S): 2.2e-3 * b for b in b_list})


def test_plan_is_the_argmin_over_the_feasible_space():
    m, plat, prof = MODELS["llama2-70b"], PlatformProfile(), _toy_profile()
    space = list(candidates(m, plat, 8, 64))
    best, feasible = plan(m, plat, prof, 2048, 8, 64, space=space)
    brute = []
    for c in space:
        mem = [stage_memory(m, c, p, 2048)["total"] for p in range(c.P)]
        if max(mem) <= plat.budget:
            brute.append((step_time(m, plat, prof, c, 2048)["T_step"], c))
    assert len(feasible) == len(brute) > 0
    assert best[1] == pytest.approx(min(t for t, _ in brute))
    assert all(max(x["total"] for x in r[3]) <= plat.budget for r in feasible)
    # a budget below the smallest stage memory prunes everything
    tiny = PlatformProfile(hbm_bytes=10e9, reserve_bytes=0)
    assert plan(m, tiny, prof, 2048, 8, 64, space=space)[0] is None


def test_exposures_and_recovery_windows():
    m, plat, prof = MODELS["llama2-7b"], PlatformProfile(), _toy_profile()
    for c in candidates(m, plat, 8, 32):
        t = step_time(m, plat, prof, c, 2048)
        assert min(t["E_comm"], t["E_upd"], t["E_pref"], t["E_rec"]) >= 0
        assert t["T_step"] >= t["T_1F1B"]
    # one stage has no idle time: FSR exposes the whole recompute
    c = Config(1, 1, 0, 1, 4, "fsr")
    t = step_time(m, plat, prof, c, 2048)
    assert t["E_rec"] == pytest.approx(4 * 32 * 1e-3)
    # long pipeline, few micro-batches: the bubbles cover the recompute of the last stage ...
    c = Config(8, 1, 0, 1, 8, "fsr")
    t8 = step_time(m, plat, prof, c, 2048)
    ck = step_time(m, plat, prof, Config(8, 1, 0, 1, 8, "ckpt"), 2048)
    assert t8["T_step"] <= ck["T_step"]
