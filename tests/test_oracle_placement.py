"""Pins of the placement oracle (Sec. 4.3 objective, Alg. 1), CPU only.

The oracle enumerates placements; these tests check it against a placement
worked by hand, against an independent exact solver (scipy's MILP, HiGHS) on
seeded instances, and against closed forms of special cases.
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import placement as pl

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _worked():
    with open(os.path.join(GOLD, "placement_worked.json")) as f:
        return json.load(f)


def test_worked_example_golden():
    w = _worked()
    g = w["granularity"]
    s = [m * g for m in w["sizes_mib"]]
    for case in w["cases"]:
        c = [0.0] * len(s) if case.get("c_zero") else w["c"]
        best, arg = pl.brute_force(s, w["r"], c, case["budget_mib"] * g, g, case.get("is_expert"))
        assert best == case["best"], case
        assert sorted(arg) == sorted(case["placements"]), case


def _milp(s, r, c, M, g, is_expert=None):
    """Exact optimum by mixed-integer programming: x_i = [b_i = GPU], z_i >= |x_i - x_{i-1}|
    (c >= 0 makes z_i equal it at the optimum), the quantised budget over the chosen tensors,
    and Alg. 1's fixed tensors as bounds."""
    from scipy.optimize import Bounds, LinearConstraint, milp
    n = len(s)
    forced, budget = pl.branch(s, M, is_expert)
    nv = n + (n - 1)
    cost = np.concatenate([-np.asarray(r, float), np.asarray(c[1:], float)])
    rows, lo, hi = [], [], []
    for i in range(1, n):
        for sign in (1, -1):
            a = np.zeros(nv)
            a[n + i - 1] = 1
            a[i] -= sign
            a[i - 1] += sign
            rows.append(a); lo.append(0); hi.append(np.inf)
    a = np.zeros(nv)
    for i in range(n):
        if forced[i] is None:
            a[i] = math.ceil(s[i] / g)
    rows.append(a); lo.append(-np.inf); hi.append(pl.budget_units(budget, g))
    lb = np.zeros(nv); ub = np.ones(nv)
    for i, f in enumerate(forced):
        if f is not None:
            lb[i] = ub[i] = f
    res = milp(cost, constraints=LinearConstraint(np.array(rows), lo, hi), integrality=np.ones(nv),
               bounds=Bounds(lb, ub))
    assert res.success
    return -res.fun


@pytest.mark.parametrize("seed", range(12))
def test_brute_force_matches_milp(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(3, 13))
    g = 1 << 20
    s = (rng.integers(1, 9, n) * g - rng.integers(0, g, n)).astype(float)  # not multiples of g
    r = rng.normal(1.0, 1.5, n)
    c = np.abs(rng.normal(0.0, 1.0, n))
    M = float(rng.uniform(0.2, 0.8) * s.sum())
    expert = None if seed % 3 == 0 else [int(v) for v in rng.integers(0, 2, n)]
    best, arg = pl.brute_force(list(s), list(r), list(c), M, g, expert)
    assert best == pytest.approx(_milp(list(s), list(r), list(c), M, g, expert), abs=1e-9)
    for b in arg:
        assert pl.feasible(b, list(s), M, g, expert)


def test_everything_fits_and_no_switch_cost():
    """With room for every tensor and c = 0, the optimum puts exactly the
    tensors with a positive gain on the GPU."""
    r = [2.0, -1.0, 0.5, -3.0, 4.0]
    s = [1.0] * 5
    best, arg = pl.brute_force(s, r, [0.0] * 5, 10.0, 1.0)
    assert best == 6.5 and arg == [[1, 0, 1, 0, 1]]


def test_zero_budget_keeps_everything_on_cpu():
    best, arg = pl.brute_force([3.0, 1.0], [5.0, 7.0], [0.0, 1.0], 0.0, 1.0)
    assert best == 0.0 and arg == [[0, 0]]


def test_switch_cost_prefers_one_contiguous_run():
    """Two equally useful tensors separated by a useless one: with costly
    switches, moving the middle one too (one run) beats two separate runs."""
    s, r, c = [1.0, 1.0, 1.0], [3.0, 0.0, 3.0], [0.0, 2.0, 2.0]
    best, arg = pl.brute_force(s, r, c, 3.0, 1.0)
    assert best == 6.0 and arg == [[1, 1, 1]]
    best, arg = pl.brute_force(s, r, c, 2.0, 1.0)  # no room for the bridge: 3 + 3 - 2 * 2 vs 3 - 2
    assert best == 2.0 and arg == [[1, 0, 1]]


def test_sizes_round_up_and_budget_rounds_down():
    g = 10.0
    # 11 bytes take 2 units; a 19-byte budget has 1 unit: the tensor does not fit
    assert pl.brute_force([11.0], [1.0], [0.0], 19.0, g)[1] == [[0]]
    assert pl.brute_force([11.0], [1.0], [0.0], 20.0, g)[1] == [[1]]
