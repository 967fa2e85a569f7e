"""Pins of the oracle's 1F1B schedule simulation (CPU).

Closed forms of non-interleaved 1F1B that do not depend on the simulation:
with equal stage times and free transfers the step takes (A + P - 1)(t_f +
t_b); one stage takes A (t_f + t_b); stage p holds min(P - p, A) micro-
batches' activations.  Brute-force checks of the simulated timeline: every
dependency is met, a stage never runs two tasks at once, every task runs
once.  Bounds: the makespan is at least the busiest stage's work and at
least one micro-batch's critical path.  A plausible slip (one warm-up
forward too many) fails the activation count.
"""

import itertools

import numpy as np
import pytest

import oracle.pipeline as pl
from oracle import simulate_1f1b, stage_order


@pytest.mark.parametrize("P,A", [(1, 1), (1, 7), (2, 1), (2, 2), (4, 8), (8, 3), (5, 16)])
def test_uniform_closed_form_and_resident_microbatches(P, A):
    r = simulate_1f1b(P, A, 1.0, 2.0)
    assert r["makespan"] == pytest.approx((A + P - 1) * 3.0, abs=1e-12)
    assert r["n_act"] == [min(P - p, A) for p in range(P)]


@pytest.mark.parametrize("P,A,seed", list(itertools.product([1, 2, 3, 5], [1, 2, 4, 9], [0, 1])))
def test_timeline_is_a_valid_1f1b_schedule(P, A, seed):
    rng = np.random.default_rng(seed)
    tf, tb, tx = rng.uniform(0.5, 2, P), rng.uniform(0.5, 3, P), float(rng.uniform(0, 0.5))
    r = simulate_1f1b(P, A, tf, tb, tx)
    s, e = r["start"], r["end"]
    assert len(s) == 2 * P * A
    for p in range(P):
        # one task at a time, in the stage's 1F1B order, each as long as its stage time
        prev_end = 0.0
        for kind, m in stage_order(P, A, p):
            k = (kind, p, m)
            assert s[k] >= prev_end - 1e-12
            assert e[k] - s[k] == pytest.approx(tf[p] if kind == "F" else tb[p])
            prev_end = e[k]
        for m in range(A):
            if p > 0:
                assert s[("F", p, m)] >= e[("F", p - 1, m)] + tx - 1e-12
            assert s[("B", p, m)] >= e[("F", p, m)] - 1e-12
            if p < P - 1:
                assert s[("B", p, m)] >= e[("B", p + 1, m)] + tx - 1e-12
    busiest = max(A * (tf[p] + tb[p]) for p in range(P))
    path = tf.sum() + tb.sum() + 2 * (P - 1) * tx
    assert r["makespan"] >= busiest - 1e-9 and r["makespan"] >= path - 1e-9


def test_stage_order_shape():
    assert stage_order(4, 8, 0)[:4] == [("F", 0), ("F", 1), ("F", 2), ("F", 3)]
    assert stage_order(4, 8, 3)[:2] == [("F", 0), ("B", 0)]
    for P, A in [(4, 8), (3, 2), (1, 5)]:
        for p in range(P):
            o = stage_order(P, A, p)
            assert sorted(o) == sorted([("F", m) for m in range(A)] + [("B", m) for m in range(A)])


def test_planted_extra_warmup_forward_fails_the_activation_count():
    saved = pl.stage_order
    try:
        def wrong(P, A, p):        # one warm-up forward too many (P - p instead of P - 1 - p)
            warm = min(P - p, A)
            order = [("F", m) for m in range(warm)]
            nf, nb = warm, 0
            while nf < A:
                order += [("F", nf), ("B", nb)]
                nf += 1
                nb += 1
            order += [("B", m) for m in range(nb, A)]
            return order
        pl.stage_order = wrong
        r = pl.simulate_1f1b(4, 8, 1.0, 2.0)
    finally:
        pl.stage_order = saved
    assert r["n_act"] != [4, 3, 2, 1]
