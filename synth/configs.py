"""Shapes, seeds and placement recipes of the five synthetic workloads.

Sizes are in x out ("K x N"); a quantised tensor stores N rows of K inputs.
Every weight is block-int4 with one fp16 scale per 32 consecutive inputs.

  linear4096   one 4096 x 4096 linear; decode batch 1 and batch 16; all in HBM.
  dense_layer  one 8B-shaped decoder layer (hidden 4096, 32 query / 8 KV heads
               of 128, SwiGLU 14336); decode batch 1 and prefill 512; three of
               the seven tensors, chosen by a seeded permutation, on host.
  dense_stack  32 such layers, decode loop of 256 steps over 8 sequences; the
               tensors with the lowest seeded access-cost scores go to host
               until 30 % of the int4 bytes are there.
  moe_layer    30B-A3B-shaped MoE layer (hidden 2048, 128 experts of SwiGLU
               768, top-8); prefill 512 and decode 1; 51 experts on host.
  moe_stack    94 235B-A22B-shaped layers (hidden 4096, 64 / 4 heads of 128,
               128 experts of SwiGLU 1536, top-8); prefill 2048 and decode 1;
               40 % of the expert matrices on host by seeded score.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import gen

ROLES = ("q", "k", "v", "o", "gate", "up", "down")


def qbytes(K: int, N: int) -> int:
    """Bytes of one block-int4 tensor: K*N/2 code bytes plus K*N/32 fp16 scales."""
    return K * N // 2 + 2 * (K * N // 32)


def dense_uid(layer: int, role: str) -> int:
    return layer * 1_000_000 + 999_000 + ROLES.index(role)


def expert_uid(layer: int, expert: int, proj: str) -> int:
    return layer * 1_000_000 + expert * 10 + ("gate", "up", "down").index(proj)


def router_uid(layer: int) -> int:
    return layer * 1_000_000 + 998_000


@dataclass(frozen=True)
class DenseShape:
    hidden: int = 4096
    n_heads: int = 32
    n_kv: int = 8
    head_dim: int = 128
    inter: int = 14336

    def kn(self, role: str) -> tuple[int, int]:
        h, q, kv, i = self.hidden, self.n_heads * self.head_dim, self.n_kv * self.head_dim, self.inter
        return {"q": (h, q), "k": (h, kv), "v": (h, kv), "o": (q, h),
                "gate": (h, i), "up": (h, i), "down": (i, h)}[role]

    def layer_bytes(self) -> int:
        return sum(qbytes(*self.kn(r)) for r in ROLES)


@dataclass(frozen=True)
class MoEShape:
    hidden: int = 2048
    n_experts: int = 128
    top_k: int = 8
    inter: int = 768

    def expert_bytes(self) -> int:
        return 3 * qbytes(self.hidden, self.inter)


@dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    dense: DenseShape | None = None
    moe: MoEShape | None = None
    n_layers: int = 1
    decode_m: int = 1
    prefill_m: int = 0
    steps: int = 1
    notes: dict = field(default_factory=dict)


LINEAR4096 = Workload("linear4096", 1001, decode_m=1, prefill_m=16,
                      notes={"K": 4096, "N": 4096})
DENSE_LAYER = Workload("dense_layer", 1002, dense=DenseShape(), decode_m=1, prefill_m=512)
DENSE_STACK = Workload("dense_stack", 1003, dense=DenseShape(), n_layers=32, decode_m=8, steps=256)
MOE_LAYER = Workload("moe_layer", 1004, moe=MoEShape(), decode_m=1, prefill_m=512)
MOE_STACK = Workload("moe_stack", 1005,
                     dense=DenseShape(hidden=4096, n_heads=64, n_kv=4, head_dim=128, inter=0),
                     moe=MoEShape(hidden=4096, n_experts=128, top_k=8, inter=1536),
                     n_layers=94, decode_m=1, prefill_m=2048)

WORKLOADS = {w.name: w for w in (LINEAR4096, DENSE_LAYER, DENSE_STACK, MOE_LAYER, MOE_STACK)}


# ---------------------------------------------------------------- placement recipes

def dense_layer_host_mask(seed: int = DENSE_LAYER.seed, n_host: int = 3) -> np.ndarray:
    """uint8[7] over ROLES; the first n_host roles of a seeded permutation are on host.

    Half of seven tensors is read as floor(3.5) = 3.
    """
    mask = np.zeros(len(ROLES), np.uint8)
    mask[gen.permutation(seed, 777, len(ROLES))[:n_host]] = 1
    return mask


def dense_stack_host_mask(shape: DenseShape = DENSE_STACK.dense, n_layers: int = 32,
                          seed: int = DENSE_STACK.seed, frac: float = 0.30) -> np.ndarray:
    """uint8[n_layers][7]: scan tensors by ascending seeded access-cost score and put
    each on host while the host share stays within frac of all int4 bytes."""
    n = n_layers * len(ROLES)
    sc = gen.scores(seed, 778, n)
    sizes = np.array([qbytes(*shape.kn(ROLES[i % len(ROLES)])) for i in range(n)], np.int64)
    budget = frac * sizes.sum()
    mask = np.zeros(n, np.uint8)
    used = 0
    for i in np.argsort(sc, kind="stable"):
        if used + sizes[i] <= budget:
            mask[i] = 1
            used += sizes[i]
    return mask.reshape(n_layers, len(ROLES))


def moe_host_experts(n_experts: int = 128, frac: float = 0.40, seed: int = MOE_LAYER.seed,
                     layer: int = 0) -> np.ndarray:
    """uint8[n_experts]: floor(frac * n_experts) experts, chosen by a seeded
    permutation that knows nothing of expert popularity, live on host."""
    mask = np.zeros(n_experts, np.uint8)
    mask[gen.permutation(seed, 779 + 1000 * layer, n_experts)[: int(frac * n_experts)]] = 1
    return mask
