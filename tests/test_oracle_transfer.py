"""Pins of the dynamic-transfer oracle (Sec. 4.4; Alg. 2 and 3), CPU only.

* a four-tensor round worked by hand (tests/golden/transfer_worked.json):
  every one of the eight assignments and the minimum;
* an event-timeline simulation of a round (a CPU/GPU executor and one
  host-to-GPU link, promoted weights issued from the first CPU-side endpoint
  after the previous promotion) that must give T(rb) for every assignment of
  random rounds: it never forms seg(j, i), so a dropped switch term, a wrong
  window index or the runtime backend in place of the default one in seg
  disagrees with it;
* closed forms: one- and two-tensor rounds, and an all-CPU chain with free
  transfers, where the optimum promotes every other tensor;
* special cases: transfers too slow to hide never pay; a CPU faster than the
  GPU is never left;
* Alg. 3's decision at and around eps and tau, with exact binary fractions.
"""
import json
import math
import os
import random

import pytest

from oracle import transfer as tr

HERE = os.path.dirname(os.path.abspath(__file__))
CPU, GPU = tr.CPU, tr.GPU


def _golden():
    with open(os.path.join(HERE, "golden", "transfer_worked.json")) as f:
        return json.load(f)


def test_worked_round_every_assignment():
    g = _golden()
    seen = set()
    for case in g["cases"]:
        t = tr.latency(case["rb"], g["b"], g["tg"], g["tc"], g["c"], g["w"])
        if case["T"] is None:
            assert t == math.inf, case
        else:
            assert t == pytest.approx(case["T"], abs=1e-12), case
        seen.add(tuple(case["rb"]))
    assert seen == {tuple(rb) for rb in tr.assignments(g["b"])}


def test_worked_round_minimum():
    g = _golden()
    best, arg = tr.best_by_enumeration(g["b"], g["tg"], g["tc"], g["c"], g["w"])
    assert best == pytest.approx(g["best"]["T"], abs=1e-12)
    assert [list(r) for r in arg] == g["best"]["rb"]


def _timeline(rb, b, tg, tc, c, w):
    """End time of a round on one CPU, one GPU and one host-to-GPU link.
    Each tensor starts once its predecessor has ended and, after a backend
    change, the activation has moved (c_i); a promoted tensor also waits for
    its weights, whose copy is issued at the round start or at the end of the
    first CPU-run tensor after the previous promotion."""
    end = 0.0
    issue_at = 0.0  # when the next promoted tensor's copy can be issued; None: not yet
    for i in range(len(b)):
        ready = end
        if b[i] == CPU and rb[i] == GPU:
            if issue_at is None:
                return math.inf
            ready = max(ready, issue_at + w[i])
            issue_at = None
        if i >= 1 and rb[i - 1] != rb[i]:
            ready += c[i]
        end = ready + (tg[i] if rb[i] == GPU else tc[i])
        if rb[i] == CPU and issue_at is None:
            issue_at = end
    return end


def _random_round(rng, n):
    b = [rng.choice((CPU, GPU)) for _ in range(n)]
    tg = [rng.uniform(0.1, 2.0) for _ in range(n)]
    tc = [rng.uniform(0.5, 6.0) for _ in range(n)]
    c = [rng.uniform(0.0, 0.8) for _ in range(n)]
    w = [rng.uniform(0.0, 12.0) for _ in range(n)]
    return b, tg, tc, c, w


@pytest.mark.parametrize("seed", range(12))
def test_latency_equals_timeline(seed):
    rng = random.Random(seed)
    n = rng.randint(1, 10)
    b, tg, tc, c, w = _random_round(rng, n)
    for rb in tr.assignments(b):
        t1 = tr.latency(rb, b, tg, tc, c, w)
        t2 = _timeline(rb, b, tg, tc, c, w)
        if t2 == math.inf:
            assert t1 == math.inf, rb
        else:
            assert t1 == pytest.approx(t2, rel=1e-12, abs=1e-12), rb


def test_gpu_placed_tensor_cannot_run_on_cpu():
    with pytest.raises(ValueError):
        tr.latency([CPU], [GPU], [1.0], [1.0], [0.0], [0.0])


def test_one_tensor_closed_form():
    for tg, tc, w in [(1.0, 3.0, 1.5), (1.0, 3.0, 2.5), (2.0, 1.0, 0.0), (0.5, 4.0, 9.0)]:
        best, _ = tr.best_by_enumeration([CPU], [tg], [tc], [0.0], [w])
        assert best == pytest.approx(min(tc, tg + w))


def test_two_tensor_closed_form():
    rng = random.Random(7)
    for _ in range(50):
        tg = [rng.uniform(0.1, 3) for _ in range(2)]
        tc = [rng.uniform(0.1, 3) for _ in range(2)]
        c = [0.0, rng.uniform(0, 1)]
        w = [rng.uniform(0, 5) for _ in range(2)]
        cc = tc[0] + tc[1]
        gc = w[0] + tg[0] + c[1] + tc[1]
        cg = tc[0] + c[1] + max(w[1] - tc[0], 0.0) + tg[1]
        best, _ = tr.best_by_enumeration([CPU, CPU], tg, tc, c, w)
        assert best == pytest.approx(min(cc, gc, cg), abs=1e-12)


@pytest.mark.parametrize("n", [1, 2, 3, 6, 9, 14])
def test_free_transfers_alternate(n):
    """All tensors CPU-placed, GPU faster, no switch or transfer cost: promotions
    need a CPU-run tensor between them, so the best round promotes ceil(n/2)."""
    g, h = 1.0, 3.0
    best, arg = tr.best_by_enumeration([CPU] * n, [g] * n, [h] * n, [0.0] * n, [0.0] * n)
    assert best == pytest.approx(n * h - math.ceil(n / 2) * (h - g))
    for rb in arg:
        assert sum(rb) == math.ceil(n / 2)


@pytest.mark.parametrize("seed", range(6))
def test_unhideable_transfers_never_pay(seed):
    rng = random.Random(100 + seed)
    b, tg, tc, c, _ = _random_round(rng, 9)
    w = [1e6] * 9
    best, arg = tr.best_by_enumeration(b, tg, tc, c, w)
    assert arg == [list(b)]
    assert best == pytest.approx(_timeline(b, b, tg, tc, c, w))


@pytest.mark.parametrize("seed", range(6))
def test_fast_cpu_is_kept(seed):
    rng = random.Random(200 + seed)
    b, tg, tc, c, w = _random_round(rng, 9)
    tc = [0.01] * 9
    tg = [5.0] * 9
    best, arg = tr.best_by_enumeration(b, tg, tc, c, w)
    assert arg == [list(b)]


@pytest.mark.parametrize("seed", range(6))
def test_optimum_is_monotone_in_costs(seed):
    rng = random.Random(300 + seed)
    b, tg, tc, c, w = _random_round(rng, 8)
    base, _ = tr.best_by_enumeration(b, tg, tc, c, w)
    slower_link, _ = tr.best_by_enumeration(b, tg, tc, c, [x * 1.5 for x in w])
    slower_cpu, _ = tr.best_by_enumeration(b, tg, [x * 1.5 for x in tc], c, w)
    assert slower_link >= base - 1e-12 and slower_cpu >= base - 1e-12


def _snap(tg, tc, c, w):
    return (tg, tc, c, w)


def test_deviation_by_hand():
    prev = _snap([1.0, 1.0], [2.0, 2.0], [0.5, 0.5], [3.0, 1.0])
    assert tr.deviation(prev, prev) == 0.0
    # CPU total 4 -> 4.625: 0.15625; link total 4 -> 3.5: 0.125; the larger counts
    cur = _snap([1.0, 1.0], [2.0, 2.625], [0.5, 0.5], [3.0, 0.5])
    assert tr.deviation(prev, cur) == 0.15625
    # a series growing from zero always deviates
    assert tr.deviation(_snap([1.0], [1.0], [0.0], [1.0]), _snap([1.0], [1.0], [0.25], [1.0])) == math.inf


def test_reschedule_thresholds():
    prev = _snap([1.0, 1.0], [2.0, 2.0], [0.5, 0.5], [3.0, 1.0])
    at_eps = _snap([1.0, 1.0], [2.0, 2.5], [0.5, 0.5], [3.0, 1.0])        # d = 0.125 exactly
    below = _snap([1.0, 1.0], [2.0, 2.4375], [0.5, 0.5], [3.0, 1.0])      # d = 0.109375
    tau = 5 * 0.03125
    last = 1.0
    assert tr.should_reschedule(None, prev, 0.125, 0.0, 0.0, tau)
    assert tr.should_reschedule(prev, at_eps, 0.125, last + tau, last, tau)
    assert not tr.should_reschedule(prev, below, 0.125, last + tau, last, tau)
    assert not tr.should_reschedule(prev, at_eps, 0.125, last + tau - 2.0 ** -10, last, tau)
    assert tr.should_reschedule(prev, at_eps, 0.125, last + 10 * tau, last, tau)
