"""Brute-force inter-stage planner: the plan of Eq. 1-3 by exhaustive enumeration.

TEST INFRASTRUCTURE ONLY (see oracle/oracle.py): plain Python loops for small spaces.

A plan for one hardware sample fixes the gradient-accumulation steps G, the number of stages
PP = S, the layer counts l_1..l_S (each in the space's layer set for PP, summing to the model's
L) and, for every stage i, one candidate configuration of the intra-stage group
(hw, G, PP, k = PP - i + 1, l_i): stage 1 runs PP microbatches in flight, the last stage one.
A group's candidates are the points sampled from its (t, d) frontier (Eq. 3): the
configurations that the weight-sampled argmins select (Eq. 4), and the group's best (the tuner's
own objective); a group without a feasible configuration has none.  The plan's value is the
objective of Eq. 2 with the inner sum read as the time of the stages before i:

    F = (G - 1) * max_i t_i + sum_i t_i + max_i (d_i - sum_{j<i} t_j),

evaluated in stage order: the sums left to right, F = ((G-1)*t_max + t_sum) + m.

The same objective regrouped, F = (G - 1) * max_i t_i + max_i (d_i + sum_{j>=i} t_j), is equal in
real arithmetic; evaluated with the sums taken from the last stage to the first it can differ in
the last bits.  plan_value_suffix is that form (the one in which a stage-by-stage search from the
last stage prunes exactly).
"""

from __future__ import annotations

import itertools

import numpy as np

from . import oracle as O


def plan_value(G: int, ts, ds) -> float:
    """Eq. 2 for one plan (stage order, left to right)."""
    t_max = ts[0]
    t_sum = 0.0
    m = None
    for t, d in zip(ts, ds):
        v = d - t_sum
        m = v if m is None else max(m, v)
        t_sum = t_sum + t
        t_max = max(t_max, t)
    return (float(G - 1) * t_max + t_sum) + m


def plan_value_suffix(G: int, ts, ds) -> float:
    """Eq. 2 as (G - 1) * max t + max_i (d_i + T_i), T_i = t_i + T_{i+1} summed from the last
    stage to the first."""
    T = 0.0
    h = None
    for t, d in zip(reversed(ts), reversed(ds)):
        T = t + T
        h = d + T if h is None else max(h, d + T)
    return float(G - 1) * max(ts) + h


def candidates(wl: dict, alphas=()) -> dict:
    """{hw: {(G, PP, k, l): [(t, d, id), ...]}} from the oracle's own results: each group's best
    configuration and the one each weight sample selects."""
    o = O.Oracle(wl)
    keys = o.group_keys()
    best = o.run()
    ids = [[int(i)] for i in best["best_id"]]
    if len(alphas):
        al = o.run_alpha(list(alphas))
        for g in range(o.n_groups):
            ids[g] += [int(i) for i in al["id"][g]]
    out = {}
    for g, k in enumerate(keys):
        uniq = sorted(set(i for i in ids[g] if i != int(O.NONE)))
        if not uniq:
            continue
        vals = o.eval_ids(np.array(uniq, dtype=np.uint64))
        out.setdefault(k["hw"], {})[(k["G"], k["PP"], k["k"], k["l"])] = [
            (float(v[0]), float(v[1]), i) for v, i in zip(vals, uniq)]
    return out


def candidates_groups(wl: dict, alphas, groups, procs: int = 1) -> dict:
    """candidates() restricted to the listed groups (process-parallel oracle runs):
    {hw: {(G, PP, k, l): [(t, d, id), ...]}}."""
    groups = sorted(int(g) for g in groups)
    o = O.Oracle(wl)
    keys = o.group_keys()
    best = O.run_groups(wl, groups, procs)
    ids = {g: [int(i)] for g, i in zip(groups, best["best_id"])}
    if len(alphas):
        al = O.run_alpha_groups(wl, alphas, groups, procs)
        for r, g in enumerate(groups):
            ids[g] += [int(i) for i in al["id"][r]]
    out = {}
    for g in groups:
        uniq = sorted(set(i for i in ids[g] if i != int(O.NONE)))
        if not uniq:
            continue
        k = keys[g]
        vals = o.eval_ids(np.array(uniq, dtype=np.uint64))
        out.setdefault(k["hw"], {})[(k["G"], k["PP"], k["k"], k["l"])] = [
            (float(v[0]), float(v[1]), i) for v, i in zip(vals, uniq)]
    return out


def best_plan(cand: dict, n_layers: int, pp: int = 0, value=plan_value):
    """Exhaustive minimum of Eq. 2 over (G, PP, layer counts, one point per stage) for one
    hardware sample's candidates {(G, PP, k, l): [(t, d, id)]}; stage i draws from group
    (G, PP, PP - i + 1, l_i).  `value` evaluates a plan (plan_value or plan_value_suffix).
    Returns (F, G, PP, [l_i], [id_i]) or None; the first minimum found on ties."""
    lsets = {}
    for (G, PP, k, l) in cand:
        lsets.setdefault((G, PP), set()).add(l)
    best = None
    for (G, PP), ls in sorted(lsets.items()):
        if pp and PP != pp:
            continue
        for parts in itertools.product(sorted(ls), repeat=PP):
            if sum(parts) != n_layers:
                continue
            pts = [cand.get((G, PP, PP - i, parts[i]), []) for i in range(PP)]
            if any(len(p) == 0 for p in pts):
                continue
            for choice in itertools.product(*pts):
                F = value(G, [c[0] for c in choice], [c[1] for c in choice])
                if best is None or F < best[0]:
                    best = (F, G, PP, list(parts), [c[2] for c in choice])
    return best
