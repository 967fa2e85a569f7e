"""Oracle non-interleaved 1F1B pipeline schedule (test infrastructure only).

The paper keeps the standard non-interleaved 1F1B main schedule (Sec. 3 and
Sec. 4.3) and its planner needs the schedule's main execution time T_1F1B
and the number of micro-batches whose activations a stage holds, N_act(p)
(Sec. 4.3, Eq. act-full; Sec. 4.4, Eq. planner-step-time).  This module
does not use a formula for either: it runs the schedule as a discrete-event
simulation and reads both off the simulated timeline.

Schedule: P stages, A micro-batches.  Stage p (0 = input side) runs
    min(P - 1 - p, A) warm-up forwards,
    then alternates one forward and one backward while forwards remain,
    then the remaining backwards,
each in micro-batch order.  Forward (p, m) needs forward (p - 1, m) plus one
stage-boundary transfer; backward (p, m) needs backward (p + 1, m) plus one
transfer, and the stage's own forward (p, m).  A stage runs one task at a
time, in its list order, as soon as its inputs are there.
"""

import numpy as np


def stage_order(P, A, p):
    """Task list of stage p: [("F", m) or ("B", m), ...] in 1F1B order."""
    warm = min(P - 1 - p, A)
    order = [("F", m) for m in range(warm)]
    nf, nb = warm, 0
    while nf < A:
        order.append(("F", nf))
        nf += 1
        order.append(("B", nb))
        nb += 1
    while nb < A:
        order.append(("B", nb))
        nb += 1
    return order


def simulate_1f1b(P, A, t_f, t_b, t_x=0.0):
    """Simulate the schedule.  t_f[p], t_b[p]: forward / backward time of one
    micro-batch on stage p; t_x: one stage-boundary transfer.

    Returns a dict with
      'makespan'  : time at which the last task ends,
      'n_act'     : [P] the most micro-batches a stage holds activations for
                    at once (from its forward's start to its backward's end),
      'start', 'end' : {(kind, p, m): time}.
    """
    t_f = np.broadcast_to(np.asarray(t_f, dtype=np.float64), (P,))
    t_b = np.broadcast_to(np.asarray(t_b, dtype=np.float64), (P,))
    orders = [stage_order(P, A, p) for p in range(P)]
    pos = [0] * P                     # next task index per stage
    free = [0.0] * P                  # time the stage becomes idle
    start, end = {}, {}
    remaining = sum(len(o) for o in orders)
    while remaining:
        progressed = False
        for p in range(P):
            if pos[p] == len(orders[p]):
                continue
            kind, m = orders[p][pos[p]]
            if kind == "F":
                deps = [] if p == 0 else [("F", p - 1, m)]
                extra = 0.0 if p == 0 else t_x
                dur = t_f[p]
            else:
                deps = [("F", p, m)] + ([] if p == P - 1 else [("B", p + 1, m)])
                extra = 0.0 if p == P - 1 else t_x
                dur = t_b[p]
            if not all(d in end for d in deps):
                continue
            ready = max([free[p]] + [end[d] + (extra if d[0] == kind and d[1] != p else 0.0)
                                     for d in deps])
            start[(kind, p, m)] = ready
            end[(kind, p, m)] = ready + dur
            free[p] = ready + dur
            pos[p] += 1
            remaining -= 1
            progressed = True
        if not progressed:
            raise RuntimeError("1F1B schedule deadlocked")
    n_act = []
    for p in range(P):
        events = []
        for m in range(A):
            events.append((start[("F", p, m)], 1))
            events.append((end[("B", p, m)], -1))
        events.sort(key=lambda e: (e[0], e[1]))   # a release at t precedes an acquire at t
        cur = best = 0
        for _, d in events:
            cur += d
            best = max(best, cur)
        n_act.append(best)
    return {"makespan": max(end.values()), "n_act": n_act, "start": start, "end": end}
