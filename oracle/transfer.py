"""Oracle of the load-aware dynamic transfer (Sec. 4.4): the round latency
T(rb) of a runtime backend assignment, its minimum by enumeration, and the
re-scheduling decision of Alg. 3.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU baseline may import this module; it shares no code with the
library's scheduler.

Definitions (Sec. 4.4.1).  Tensors 1..n in execution order have a default
placement b_i in {CPU, GPU} (the static placement), GPU and CPU execution
times t^g_i, t^c_i, activation-transfer (backend-switch) costs c_i at the
boundary between tensors i-1 and i, and weight-transfer times w_i.  A runtime
assignment rb keeps every b_i = GPU tensor on the GPU; a b_i = CPU tensor
either runs on the CPU or is promoted (its weights are copied to the GPU and
it runs there).  The round latency is

  T(rb) = sum_i t_i^{rb_i} + sum_{i>=2} c_i [rb_{i-1} != rb_i]
          + sum over promoted i of delta_i,
  delta_i = max(w_i - seg(j, i), 0),
  seg(j, i) = sum_{k=j+1}^{i-1} t_k^{b_k} + sum_{k=j+1}^{i-1} c_k [b_{k-1} != b_k],

with j the CPU-side endpoint where the transfer of i starts.  Readings where
the paper leaves the definition open (the dynamic program of Alg. 2 fixes
them, and this module follows it so that its minimum is the program's):

 * j is the round start (j = 0, a virtual CPU-side point) or a tensor that
   runs on the CPU, and every tensor strictly between j and i runs on its
   default backend (which is what seg(j, i) sums).  For a given rb the window
   is widest at the earliest such j, and that is the j counted: the round
   start when no tensor before i is promoted, else the first CPU-run tensor
   after the last promoted tensor before i.  When no such j exists (two
   promotions with no CPU-run tensor between them) rb is not reachable and
   T(rb) is infinite.
 * A switch term needs a tensor before it: c_1 never counts, neither in T nor
   in seg(0, i).
 * The switch charged when i is promoted is c_i when the tensor before it
   runs on the CPU, which is the T(rb) switch term; the algorithm's printed
   condition (previous default backend GPU) contradicts T(rb) and is read as
   a slip.

Here CPU is 0 and GPU is 1 in every array, and indices are 0-based (the
virtual round start is -1).
"""
from __future__ import annotations

import itertools
import math

CPU, GPU = 0, 1
START = -1


def seg(j: int, i: int, b, tg, tc, c) -> float:
    """seg(j, i): the default path's time strictly between CPU-side endpoint
    j (START for the round start) and tensor i."""
    s = 0.0
    for k in range(j + 1, i):
        s += tg[k] if b[k] == GPU else tc[k]
        if k >= 1 and b[k - 1] != b[k]:
            s += c[k]
    return s


def transfer_starts(rb, b):
    """For each promoted tensor i, the CPU-side endpoint its transfer starts
    from (see the module readings), or None where rb is not reachable."""
    out = {}
    start = START        # earliest admissible endpoint; None right after a promotion
    for i in range(len(b)):
        if b[i] == CPU and rb[i] == GPU:
            out[i] = start
            start = None
        elif rb[i] == CPU and start is None:
            start = i
    return out


def latency(rb, b, tg, tc, c, w) -> float:
    """T(rb) of Sec. 4.4.1 (math.inf for an unreachable rb)."""
    n = len(b)
    if any(b[i] == GPU and rb[i] == CPU for i in range(n)):
        raise ValueError("a tensor placed on the GPU stays on the GPU")
    starts = transfer_starts(rb, b)
    if any(j is None for j in starts.values()):
        return math.inf
    total = 0.0
    for i in range(n):
        total += tg[i] if rb[i] == GPU else tc[i]
        if i >= 1 and rb[i - 1] != rb[i]:
            total += c[i]
    for i, j in starts.items():
        total += max(w[i] - seg(j, i, b, tg, tc, c), 0.0)
    return total


def assignments(b):
    """Every rb that keeps the GPU-placed tensors on the GPU."""
    free = [i for i in range(len(b)) if b[i] == CPU]
    for bits in itertools.product((CPU, GPU), repeat=len(free)):
        rb = [GPU] * len(b)
        for i, v in zip(free, bits):
            rb[i] = v
        yield rb


def best_by_enumeration(b, tg, tc, c, w, rtol: float = 1e-12):
    """(minimum T over all rb, the list of rb reaching it within rtol)."""
    if sum(1 for v in b if v == CPU) > 16:
        raise ValueError("enumeration is for rounds with at most 16 CPU-placed tensors")
    scored = [(latency(rb, b, tg, tc, c, w), rb) for rb in assignments(b)]
    best = min(t for t, _ in scored)
    tol = rtol * max(1.0, abs(best))
    return best, [rb for t, rb in scored if t <= best + tol]


def deviation(prev, cur) -> float:
    """ComputeDeviation of Alg. 3 (the paper leaves it open).  Reading: a
    snapshot is the four measured series (t^g, t^c, c, w); the deviation is the
    largest relative change of a series' total, max_s |sum cur_s - sum prev_s|
    / sum prev_s (infinite when a series grows from zero)."""
    d = 0.0
    for p, q in zip(prev, cur):
        sp, sq = math.fsum(p), math.fsum(q)
        if sp > 0.0:
            d = max(d, abs(sq - sp) / sp)
        elif sq > 0.0:
            d = math.inf
    return d


def should_reschedule(prev, cur, eps: float, now: float, last: float, tau: float,
                      placement_changed: bool = False) -> bool:
    """Alg. 3's test: keep the previous assignment when the deviation is below
    eps or less than tau has passed since the last re-scheduling.  Readings:
    with no previous snapshot (the first round) schedule; a new default
    placement b invalidates the previous assignment, so it schedules too."""
    if prev is None or placement_changed:
        return True
    return not (deviation(prev, cur) < eps or now - last < tau)
