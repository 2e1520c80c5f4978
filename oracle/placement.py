"""Static tensor placement by exhaustive enumeration (test infrastructure only).

Sec. 4.3 (Problem Formulation) places each tensor i of the execution order on
b_i in {CPU, GPU} to maximise

    sum_i r_i [b_i = GPU]  -  sum_{i >= 2} c_i [b_i != b_{i-1}]

subject to sum_i s_i [b_i = GPU] <= M, where r_i = t_i^c - t_i^g is the
latency saved by running tensor i on the GPU and c_i the activation-switch
cost at the boundary between tensors i-1 and i.  Sizes and the budget are
quantised at a granularity g (the paper uses MB): a tensor takes ceil(s_i / g)
units, the budget floor(M / g) units.

Alg. 1 (Static Tensor Placement) adds a branch for MoE models: when the budget
covers every non-expert tensor, those are placed on the GPU and only the
expert tensors are chosen, within what remains; otherwise every expert tensor
stays on the CPU and only the non-expert tensors are chosen.  Reading used
here (the algorithm does not say how adjacency is counted for a subset): the
chosen subset is optimised for the full objective over the whole execution
order, with the other tensors fixed to their branch's backend.

This module enumerates every placement of the free tensors (2^n of them), so
it is meant for n up to about 16.  Nothing here is imported by the library.
"""
from __future__ import annotations

import itertools
import math

CPU, GPU = 0, 1


def objective(b, r, c) -> float:
    """The Sec. 4.3 objective of placement b (0 = CPU, 1 = GPU); c[0] is unused."""
    n = len(b)
    gain = sum(float(r[i]) for i in range(n) if b[i] == GPU)
    switches = sum(float(c[i]) for i in range(1, n) if b[i] != b[i - 1])
    return gain - switches


def size_units(s: float, g: float) -> int:
    """Budget units a tensor of s bytes takes at granularity g (rounded up)."""
    return int(math.ceil(s / g))


def budget_units(m: float, g: float) -> int:
    """Budget units of m bytes at granularity g (rounded down)."""
    return int(math.floor(m / g)) if m > 0 else 0


def branch(s, M, is_expert=None):
    """Alg. 1's dense/MoE branch: (forced, budget) where forced[i] is None for
    a tensor the knapsack chooses, else its fixed backend, and budget is the
    bytes left for the chosen tensors."""
    n = len(s)
    if is_expert is None:
        return [None] * n, M
    s_nonexp = sum(float(s[i]) for i in range(n) if not is_expert[i])
    if M >= s_nonexp:
        return [None if is_expert[i] else GPU for i in range(n)], M - s_nonexp
    return [CPU if is_expert[i] else None for i in range(n)], M


def feasible(b, s, M, g, is_expert=None) -> bool:
    """b respects Alg. 1's branch and its chosen GPU tensors fit the quantised budget."""
    forced, budget = branch(s, M, is_expert)
    if any(f is not None and b[i] != f for i, f in enumerate(forced)):
        return False
    used = sum(size_units(s[i], g) for i in range(len(b)) if forced[i] is None and b[i] == GPU)
    return used <= budget_units(budget, g)


def brute_force(s, r, c, M, g, is_expert=None):
    """(best objective, every placement reaching it) over all feasible placements."""
    n = len(s)
    forced, _ = branch(s, M, is_expert)
    free = [i for i in range(n) if forced[i] is None]
    best, arg = -math.inf, []
    for bits in itertools.product((CPU, GPU), repeat=len(free)):
        b = [forced[i] if forced[i] is not None else CPU for i in range(n)]
        for i, v in zip(free, bits):
            b[i] = v
        if not feasible(b, s, M, g, is_expert):
            continue
        val = objective(b, r, c)
        if val > best:
            best, arg = val, [b]
        elif val == best:
            arg.append(b)
    return best, arg
