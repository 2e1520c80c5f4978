#!/usr/bin/env python3
"""Benchmark of the block-int4 quantised-linear hot path on one MI355X.

Workload: one 8B-shaped dense decoder layer (hidden 4096, 32 query / 8 KV heads
of 128, SwiGLU 14336; seven int4 g32 tensors, 122.7 MB), synthetic weights
and activations from the seeded generator.

  value            decode weight GB/s: layer bytes / decode-step time, batch 1,
                   all tensors HBM-resident (inputs resident before timing),
                   rotating over copies of the layer so the 256 MB MALL cannot
                   serve the weights; steps are replayed from a HIP graph.
  prefill          tokens/s of a 512-token prefill pass over the same layer.
  streamed         the same decode step with the seeded placement mask (three
                   of the seven tensors read from pinned host memory through
                   the streaming engine), PCIe-inclusive.
  roofline         dominant decode kernel (the 4096 x 14336 GEMV) against
                   8 TB/s; roofline_prefill: the 512 x 4096 x 14336 GEMM
                   against 2.5 PFLOP/s fp16 MFMA.
  cpu_baseline     the fp64 oracle on the host cores, on a bounded sample.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "quantized linear: decode weight GB/s (% HBM peak); prefill tokens/s (% MFMA)"
HBM_PEAK_GBS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--copies", type=int, default=5, help="layer copies rotated to defeat the MALL")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on exactly one GPU: this build has no multi-GPU path "
              "(sharding is described in DESIGN.md, not implemented)", file=sys.stderr)
        return 2

    import torch

    import synth
    from synth import configs
    from paper_2607_10183_amd.session import Session

    wl = configs.DENSE_LAYER
    shape = wl.dense
    roles = configs.ROLES
    dev = torch.device("cuda", 0)
    R = args.copies

    log("generating weights")
    host_np = {}
    for r in roles:
        K, N = shape.kn(r)
        uid = configs.dense_uid(0, r)
        host_np[r] = (synth.int4_codes(wl.seed, uid, N, K), synth.group_scales(wl.seed, uid, N, K))
    layer_bytes = shape.layer_bytes()

    sess = Session(workspace_bytes=1 << 30, n_slots=4)
    tids = []  # tids[copy][role]
    for c in range(R):
        row = {}
        for r in roles:
            codes, scales = host_np[r]
            row[r] = sess.register(codes, scales, hbm=True, host=(c == 0))
        tids.append(row)
    torch.cuda.synchronize()

    H, I = shape.hidden, shape.inter
    xs = {r: torch.from_numpy(synth.activations(wl.seed, 50 + i, 512, shape.kn(r)[0])).to(dev)
          for i, r in enumerate(roles)}
    ys = {r: torch.empty((512, shape.kn(r)[1]), dtype=torch.float16, device=dev) for r in roles}
    from paper_2607_10183_amd import atsi

    def step(copy: int, M: int) -> None:
        for r in roles:
            atsi.atsi_linear(sess.ctx, tids[copy][r], xs[r].data_ptr(), M, ys[r].data_ptr())

    cs = sess.cs
    cs.wait_stream(torch.cuda.current_stream())

    # ------------------------------------------------------------ decode, HBM-resident, graph
    log("decode: capturing graph")
    reps = 4
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=cs, capture_error_mode="relaxed"):
        for _ in range(reps):
            for c in range(R):
                step(c, 1)
    steps_per_replay = reps * R
    n_replay = max(1, args.steps // steps_per_replay)
    n_warm = max(1, args.warmup // steps_per_replay)
    with torch.cuda.stream(cs):
        for _ in range(n_warm):
            g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(cs):
        e0.record(cs)
        for _ in range(n_replay):
            g.replay()
        e1.record(cs)
    torch.cuda.synchronize()
    steps_timed = n_replay * steps_per_replay
    decode_ms = e0.elapsed_time(e1) / steps_timed
    decode_gbs = layer_bytes / (decode_ms * 1e-3) / 1e9
    log(f"decode step {decode_ms * 1e3:.2f} us  -> {decode_gbs:.1f} GB/s over {steps_timed} steps")

    # ------------------------------------------------------------ dominant decode kernel
    def time_kernel(role: str, M: int, launches_per_copy: int, n_outer: int):
        gk = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gk, stream=cs, capture_error_mode="relaxed"):
            for _ in range(launches_per_copy):
                for c in range(R):
                    atsi.atsi_linear(sess.ctx, tids[c][role], xs[role].data_ptr(), M, ys[role].data_ptr())
        with torch.cuda.stream(cs):
            gk.replay()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(cs):
            a.record(cs)
            for _ in range(n_outer):
                gk.replay()
            b.record(cs)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e-3 / (n_outer * launches_per_copy * R)

    K_g, N_g = shape.kn("gate")
    gemv_bytes = configs.qbytes(K_g, N_g)
    t_gemv = time_kernel("gate", 1, 8, 10)
    gemv_gbs = gemv_bytes / t_gemv / 1e9
    log(f"gate GEMV {t_gemv * 1e6:.2f} us -> {gemv_gbs:.1f} GB/s")

    # ------------------------------------------------------------ prefill 512
    Mp = wl.prefill_m
    with torch.cuda.stream(cs):
        step(0, Mp)
    torch.cuda.synchronize()
    n_pf = max(2, min(20, args.steps // 10))
    with torch.cuda.stream(cs):
        e0.record(cs)
        for i in range(n_pf):
            step(i % R, Mp)
        e1.record(cs)
    torch.cuda.synchronize()
    prefill_ms = e0.elapsed_time(e1) / n_pf
    prefill_tps = Mp / (prefill_ms * 1e-3)
    prefill_flops = sum(2.0 * Mp * shape.kn(r)[0] * shape.kn(r)[1] for r in roles)
    log(f"prefill step {prefill_ms:.3f} ms -> {prefill_tps:.0f} tok/s, "
        f"{prefill_flops / (prefill_ms * 1e-3) / 1e12:.1f} TFLOP/s")
    t_gemm = time_kernel("gate", Mp, 1, 4)
    gemm_flops = 2.0 * Mp * K_g * N_g
    gemm_tfs = gemm_flops / t_gemm / 1e12
    log(f"gate GEMM {t_gemm * 1e6:.1f} us -> {gemm_tfs:.1f} TFLOP/s")

    # ------------------------------------------------------------ streamed decode (placement mask)
    mask_roles = configs.dense_layer_host_mask()
    host_roles = [r for r, m in zip(roles, mask_roles) if m]
    full_mask = [0] * len(sess.shapes)
    for r in host_roles:
        full_mask[tids[0][r]] = 1
    sess.set_placement(full_mask)
    host_bytes = sum(configs.qbytes(*shape.kn(r)) for r in host_roles)
    with torch.cuda.stream(cs):
        for _ in range(3):
            step(0, 1)
    torch.cuda.synchronize()
    n_st = max(5, min(50, args.steps // 4))
    t0 = time.perf_counter()
    with torch.cuda.stream(cs):
        e0.record(cs)
        for _ in range(n_st):
            step(0, 1)
        e1.record(cs)
    sess.sync()
    torch.cuda.synchronize()
    streamed_ms = e0.elapsed_time(e1) / n_st
    wall_streamed = (time.perf_counter() - t0) / n_st
    sess.set_placement([0] * len(sess.shapes))
    log(f"streamed decode step {streamed_ms:.3f} ms ({host_roles} on host, {host_bytes / 1e6:.1f} MB) -> "
        f"PCIe {host_bytes / (streamed_ms * 1e-3) / 1e9:.1f} GB/s")

    # ------------------------------------------------------------ CPU baseline (the oracle)
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(host_np, shape, roles, args.cpu_seconds, layer_bytes)
        log(f"cpu baseline {cpu}")

    out = {
        "metric": METRIC,
        "value": round(decode_gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": steps_timed,
        "warmup": n_warm * steps_per_replay,
        "ms_per_step": round(decode_ms, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {
            "workload": "dense_layer: one 8B-shaped decoder layer's seven block-int4 g32 projections "
                        "(Q 4096x4096, K/V 4096x1024, O 4096x4096, gate/up 4096x14336, down 14336x4096)",
            "decode_batch": 1, "prefill_tokens": Mp, "layer_bytes": layer_bytes,
            "placement": "all HBM-resident for value; seeded mask with 3 host tensors for 'streamed'",
            "mall_rotation_copies": R,
        },
        "pct_hbm_peak": round(100 * decode_gbs / HBM_PEAK_GBS, 2),
        "prefill_tokens_per_s": round(prefill_tps, 1),
        "prefill_ms_per_step": round(prefill_ms, 4),
        "prefill_pct_mfma": round(100 * prefill_flops / (prefill_ms * 1e-3) / 1e12 / MFMA_F16_PEAK_TFLOPS, 2),
        "roofline": {"bound": "hbm", "achieved": round(gemv_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gemv_gbs / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": "q4_gemv_kernel<1,4> on the 4096x14336 gate tensor, batch 1",
                     "bytes_per_launch": gemv_bytes, "avg_us": round(t_gemv * 1e6, 3)},
        "roofline_prefill": {"bound": "mfma", "achieved": round(gemm_tfs, 1), "peak": MFMA_F16_PEAK_TFLOPS,
                             "unit": "TFLOP/s", "frac": round(gemm_tfs / MFMA_F16_PEAK_TFLOPS, 4), "traffic": None,
                             "kernel": "q4_gemm_kernel<128,128> on the 4096x14336 gate tensor, 512 tokens",
                             "flops_per_launch": gemm_flops, "avg_us": round(t_gemm * 1e6, 2)},
        "streamed": {"host_tensors": host_roles, "host_bytes": host_bytes, "ms_per_step": round(streamed_ms, 4),
                     "weight_GBps_pcie_inclusive": round(layer_bytes / (streamed_ms * 1e-3) / 1e9, 2),
                     "pcie_GBps": round(host_bytes / (streamed_ms * 1e-3) / 1e9, 2),
                     "host_wall_ms_per_step": round(wall_streamed * 1e3, 4)},
        "cpu_baseline": cpu,
    }
    sess.close()
    print(json.dumps(out), flush=True)
    return 0


def cpu_baseline(host_np, shape, roles, budget_s, layer_bytes):
    """Time the fp64 oracle on the same decode step (7 tensors, batch 1)."""
    import oracle
    import synth
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover
        blas_threads = 1
    x = {r: synth.activations(1002, 90 + i, 1, shape.kn(r)[0]) for i, r in enumerate(roles)}
    n = 0
    t0 = time.perf_counter()
    while True:
        for r in roles:
            oracle.linear(x[r], *host_np[r])
        n += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = (time.perf_counter() - t0) / n
    return {"value": round(layer_bytes / dt / 1e9, 4), "unit": "GB/s", "cores": int(blas_threads),
            "kind": "oracle",
            "sample": f"{n} decode steps of the dense layer (7 tensors, batch 1, fp64 dequant + matmul), "
                      f"{dt:.2f} s per step",
            "host_cpus": len(os.sched_getaffinity(0))}


if __name__ == "__main__":
    sys.exit(main())
