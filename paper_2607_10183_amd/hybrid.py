"""Runtime backend selection for a stack of dense decoder layers (Sec. 4.3-4.4):
the execution units the schedulers see, per-unit measurements, the static
placement (Alg. 1) and dynamic transfer (Alg. 2) decisions, and the online
re-scheduling loop (Alg. 3).  Host-side plumbing only: the products run in
libatsi.so (GPU kernels or its CPU backend) and the decisions are the
library's atsi_solve_placement, atsi_schedule_transfers and atsi_rescheduler.

Units.  A decoder layer launches q, k and v together, o, the gate/up pair
(one fused SwiGLU launch, so the two share a backend) and down.  The unit
chain is q, k, v, o, gate+up, down per layer, in execution order; a unit's
times and size are the sums over its tensors.

Cost model of this engine.  Activations live in HBM; a CPU-run launch moves
its input to pinned memory and its output back by itself, so a CPU unit's
time t^c includes its own activation transfers and a fixed per-launch cost
(calibrated from a whole-stack run), and the backend-switch costs c are 0.
A promoted unit's weight-transfer time w is its size over the measured
host-to-device rate.
"""
from __future__ import annotations

import math
import statistics

import numpy as np

from . import atsi

ROLE_UNITS = (("q",), ("k",), ("v",), ("o",), ("gate", "up"), ("down",))


def dense_units(layers):
    """[(layer, role names, tensor ids)] in execution order; layers: list of
    {role: tid} dicts."""
    out = []
    for li, t in enumerate(layers):
        for roles in ROLE_UNITS:
            out.append((li, roles, [t[r] for r in roles]))
    return out


def unit_sum(units, per_tensor):
    return [sum(per_tensor[t] for t in tids) for _, _, tids in units]


def median_timings(samples, field, units):
    """Per-unit sum over its tensors of the median (over samples) of one
    atsi_get_timings field; NaN where a tensor has no measurement."""
    out = []
    for _, _, tids in units:
        s = 0.0
        for t in tids:
            vals = [smp[t][field] for smp in samples if not math.isnan(smp[t][field])]
            s += statistics.median(vals) if vals else math.nan
        out.append(s)
    return out


def host_mask(sess, units, unit_on_host):
    """Tensor host mask for per-unit placement (1 = host)."""
    mask = [0] * len(sess.shapes)
    for (_, _, tids), h in zip(units, unit_on_host):
        for t in tids:
            mask[t] = int(h)
    return mask


def cpu_mask(sess, units, unit_on_cpu):
    mask = [0] * len(sess.shapes)
    for (_, _, tids), h in zip(units, unit_on_cpu):
        for t in tids:
            mask[t] = int(h)
    return mask


def static_placement(unit_bytes, t_gpu, t_cpu, budget_bytes, granularity=float(64 << 10)):
    """Alg. 1 over the units: r = t^c - t^g, c = 0 (see the module's cost
    model); returns on_gpu per unit."""
    r = [tc - tg for tc, tg in zip(t_cpu, t_gpu)]
    on_gpu, _ = atsi.atsi_solve_placement(unit_bytes, r, [0.0] * len(r), budget_bytes, granularity)
    return on_gpu


def schedule(on_gpu, t_gpu, t_cpu, w):
    """Alg. 2 over the units: (rb per unit, 1 = GPU; predicted T)."""
    return atsi.atsi_schedule_transfers(on_gpu, t_gpu, t_cpu, [0.0] * len(on_gpu), w)


def cpu_unit_raw(units, tm):
    """Per-unit CPU figure of one timing read: compute plus the activation
    transfers of its launches (NaN where the unit did not run on the CPU)."""
    out = []
    for _, _, tids in units:
        out.append(sum(tm[t]["t_cpu"] + tm[t]["d2h"] + tm[t]["h2d"] for t in tids))
    return out


class Snapshotter:
    """Builds Alg. 3's measurement snapshot m = (t^g, t^c, c, w) of a round
    from the library's per-tensor timings.  `model` holds the per-unit figures
    the scheduler was profiled with and `reference` the raw timing figures
    measured in the same profiling runs; a unit measured in this round takes
    model * (fresh / reference), and a unit not measured (it ran on the other
    backend, or was not copied) the median of those ratios over its series:
    a load that slows the CPU slows every CPU unit, contention on the link
    every copy (the paper leaves unmeasured entries open).  Switch costs stay
    0 (see the module's cost model)."""

    SERIES = ("t_gpu", "t_cpu", "w")

    def __init__(self, units, model: dict, reference: dict, window: int = 4):
        self.units = units
        self.model = {k: list(model[k]) for k in self.SERIES}
        self.reference = {k: list(reference[k]) for k in self.SERIES}
        self.window = window
        self.reads = []

    def raw(self, reads):
        cpu = [cpu_unit_raw(self.units, tm) for tm in reads]
        return {"t_gpu": median_timings(reads, "t_gpu", self.units),
                "t_cpu": [float(np.nanmedian(v)) if not all(math.isnan(x) for x in v) else math.nan
                          for v in zip(*cpu)],
                "w": median_timings(reads, "w", self.units)}

    def record(self, tm):
        self.reads = (self.reads + [tm])[-self.window:]

    def __call__(self, tm):
        """Snapshot from the last `window` rounds' timing reads (per-unit
        medians, so one round disturbed by the scheduler of the host does not
        trigger a re-scheduling by itself)."""
        self.record(tm)
        fresh = self.raw(self.reads)
        out = {}
        for k in self.SERIES:
            f, ref, mod = fresh[k], self.reference[k], self.model[k]
            ratios = [fv / rv for fv, rv in zip(f, ref) if not math.isnan(fv) and rv > 0]
            scale = statistics.median(ratios) if ratios else 1.0
            out[k] = [m * (fv / rv if (not math.isnan(fv) and rv > 0) else scale) for m, fv, rv in zip(mod, f, ref)]
        return out["t_gpu"], out["t_cpu"], [0.0] * len(self.units), out["w"]


class Controller:
    """Alg. 3's loop over rounds: after each round, snapshot the measurements
    and let the library's rescheduler decide; BuildRuntime applies a new
    assignment with atsi_set_backends."""

    def __init__(self, sess, units, on_gpu, snapshotter, eps=0.15, tau_tpot=5.0):
        self.sess, self.units, self.on_gpu = sess, units, list(on_gpu)
        self.snap = snapshotter
        self.tau_tpot = tau_tpot
        self.r = atsi.atsi_rescheduler_create(len(units), eps, tau_tpot)
        self.rb = None
        self.t_last = None
        self.reschedules = 0

    def step(self, now_s, tpot_s, timings):
        """One round's decision: (re-scheduled, deviation or None).  Within
        tau of the last re-scheduling Alg. 3 keeps the assignment whatever the
        deviation, so the snapshot is only recorded then."""
        if self.t_last is not None and now_s - self.t_last < self.tau_tpot * tpot_s:
            self.snap.record(timings)
            return False, None
        tg, tc, c, w = self.snap(timings)
        rb, did, d = atsi.atsi_rescheduler_step(self.r, self.on_gpu, tg, tc, c, w, now_s, tpot_s)
        if did:
            self.reschedules += 1
            self.t_last = now_s
            self.apply(rb)
        return did, d

    def apply(self, rb):
        self.rb = list(rb)
        self.sess.set_backends(cpu_mask(self.sess, self.units, [1 - v for v in rb]))

    def close(self):
        if self.r:
            atsi.atsi_rescheduler_destroy(self.r)
            self.r = 0


def predicted(on_gpu, rb, t_gpu, t_cpu, w):
    """T(rb) of Sec. 4.4.1 for the units (atsi_transfer_latency)."""
    return atsi.atsi_transfer_latency(on_gpu, t_gpu, t_cpu, [0.0] * len(rb), w, rb)


def as_np(v):
    return np.asarray(v, dtype=np.float64)
