"""The profiling step of the static placement (Alg. 1's Profile, Sec. 4.3.1):
measure each tensor's resident GPU time and its streamed cost, turn them into
the solver's per-tensor gains r, and ask atsi_solve_placement for the mask.

On this path every tensor executes on the GPU whichever way it is stored, so
the latency a tensor saves by staying resident is its copy time over the host
link (bytes over the measured link rate, plus the fixed cost of one copy)
minus the time its resident kernel takes anyway (an over-estimate of the
cost where copies hide behind compute, which is what the solver's budget then
trades); there is no backend switch between tensors, so the switch costs c
are zero.  The empirical performance density of a tensor is r_i / s_i.
"""
from __future__ import annotations

import numpy as np
import torch

from . import atsi


def kernel_seconds(sess, tid: int, M: int, reps: int = 20) -> float:
    """Median time of one HBM-resident launch of tensor tid at M tokens (a
    graph of `reps` launches, replayed, timed with HIP events on the
    library's compute stream)."""
    K, N = sess.shapes[tid]
    x = torch.randn(M, K, device=sess.device).half()
    y = torch.empty(M, N, dtype=torch.float16, device=sess.device)
    sess.cs.wait_stream(torch.cuda.current_stream(sess.device))

    def run():
        for _ in range(reps):
            atsi.atsi_linear(sess.ctx, tid, x.data_ptr(), M, y.data_ptr())

    run()
    torch.cuda.synchronize(sess.device)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=sess.cs, capture_error_mode="relaxed"):
        run()
    ts = []
    for _ in range(7):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(sess.cs)
        g.replay()
        b.record(sess.cs)
        b.synchronize()
        ts.append(a.elapsed_time(b) * 1e-3 / reps)
    return float(np.median(ts))


def gains(sizes, t_gpu, h2d_bytes_per_s: float, per_copy_s: float = 0.0):
    """r_i = s_i / B_h2d + tau - t_gpu,i: the time tensor i saves by staying
    resident (tau: the fixed cost of one copy)."""
    s = np.asarray(sizes, dtype=np.float64)
    return s / h2d_bytes_per_s + per_copy_s - np.asarray(t_gpu, dtype=np.float64)


def solve(sizes, t_gpu, h2d_bytes_per_s: float, budget_bytes: float, granularity: float = float(1 << 20),
          is_expert=None, per_copy_s: float = 0.0):
    """Host mask (1 = streamed from pinned host memory) maximising the summed
    gains of the resident tensors within budget_bytes, and the objective."""
    r = gains(sizes, t_gpu, h2d_bytes_per_s, per_copy_s)
    on_gpu, obj = atsi.atsi_solve_placement([float(v) for v in sizes], list(r), [0.0] * len(sizes),
                                            float(budget_bytes), granularity, is_expert)
    return [1 - g for g in on_gpu], obj
