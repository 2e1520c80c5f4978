#!/usr/bin/env python3
"""Benchmark of the block-int4 quantised-linear hot path on one MI355X.

Headline workload: one 8B-shaped dense decoder layer (hidden 4096, 32 query /
8 KV heads of 128, SwiGLU 14336; seven int4 g32 tensors, 122.7 MB), seeded
synthetic weights and activations.

  value             decode weight GB/s = layer bytes / decode-step time for a
                    batch-1 pass of the whole layer (4 fused launches), all
                    tensors HBM-resident before timing, replayed from a HIP
                    graph over rotating copies of the layer (so the 256 MB
                    MALL cannot serve the weights).
  prefill           tokens/s of a 512-token pass of the same layer.
  streamed          decode and prefill with the seeded placement mask (3 of 7
                    tensors in pinned host memory, copied on the transfer
                    stream); PCIe-inclusive, never the headline value.
  moe               30B-A3B-shaped MoE layer (128 experts, top-8, capped-Zipf
                    routing): decode and 512-token prefill, all-HBM and with
                    51 experts on host.
  roofline          the dominant decode kernel, the fused SwiGLU gate/up GEMV
                    (two 4096 x 14336 tensors, 66.1 MB per launch), against
                    8 TB/s; roofline_prefill: the fused gate/up GEMM at 512
                    tokens against 2.5 PFLOP/s fp16 MFMA.  Both are timed
                    alone (atsi_swiglu_gate_up) with HIP events; their HBM
                    traffic comes from the committed counter profile when the
                    kernel sources still match it.
  stacks            dense_stack: 32 such layers as a decode loop of 8
                    sequences (hidden state renormalised after every layer),
                    all-HBM and with 30 % of the bytes streamed; moe_stack:
                    one 235B-A22B-shaped MoE decoder layer at decode and
                    2048-token prefill, all-HBM and with 40 % of its experts
                    streamed (94-layer figures = 94 x the layer).
  placement_solver  host time of the static placement solver (Alg. 1) on the
                    94-layer 235B-A22B-shaped model at 1 MiB granularity.
  cpu_baseline      the fp64 oracle's decode step on the host cores.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
       python bench.py --roofline-only   (the two roofline kernels and a
                                          256 MiB copy; for counter runs)
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


class Timer:
    """HIP-event timing on the compute stream the library launches on."""

    def __init__(self, stream):
        import torch
        self.s = stream
        self.a = torch.cuda.Event(enable_timing=True)
        self.b = torch.cuda.Event(enable_timing=True)

    def run(self, fn, n: int) -> float:
        """Seconds per call of fn over n calls."""
        import torch
        torch.cuda.synchronize()
        with torch.cuda.stream(self.s):
            self.a.record(self.s)
            for _ in range(n):
                fn()
            self.b.record(self.s)
        torch.cuda.synchronize()
        return self.a.elapsed_time(self.b) * 1e-3 / n


def h2d_timed(sess, timer, fn, n: int):
    """(seconds per call, host-to-device bytes the engine copied per call) of
    fn over n timed calls; the bytes come from the library's own counters."""
    sess.stats(reset=True)
    t = timer.run(fn, n)
    return t, sess.stats(reset=True)["h2d_bytes"] / n


def kernel_hash(kind: str) -> str:
    """sha256 of the sources a roofline kernel is built from."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2607_10183_amd", "csrc")
    files = {"q4_gemv": ("common.h", "q4_gemv_core.h", "q4_gemv.hip"),
             "q4_gemm": ("common.h", "q4_gemm_wide.hip")}[kind]
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(key: str, kind: str):
    """HBM bytes per launch from the committed FETCH_SIZE / WRITE_SIZE profile
    (profiles/traffic.json), or None when the kernel sources changed since."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as fh:
            rec = json.load(fh)[key]
    except (OSError, KeyError, ValueError):
        return None
    if rec.get("source_sha256_16") != kernel_hash(kind):
        return None
    return rec.get("hbm_bytes_per_launch")


def graph_of(stream, fn):
    import torch
    fn()  # warm (allocations, table writes) outside capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream, capture_error_mode="relaxed"):
        fn()
    return g


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--copies", type=int, default=5, help="dense-layer copies rotated to defeat the MALL")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-moe", action="store_true")
    ap.add_argument("--no-stacks", action="store_true", help="skip the dense-stack and MoE-stack lines")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--roofline-only", action="store_true",
                    help="run only the roofline kernels and a 256 MiB copy (for rocprofv3 --pmc)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path", file=sys.stderr)
        return 2

    import torch

    import synth
    from synth import configs
    from paper_2607_10183_amd import atsi
    from paper_2607_10183_amd.session import Session

    wl = configs.DENSE_LAYER
    shape = wl.dense
    roles = configs.ROLES
    dev = torch.device("cuda", 0)
    R = args.copies
    sess = Session(workspace_bytes=3 << 30, n_slots=32)
    cs = sess.cs
    timer = Timer(cs)

    # ------------------------------------------------------------ dense layer weights
    log("generating dense-layer weights")
    W = {}
    for r in roles:
        K, N = shape.kn(r)
        uid = configs.dense_uid(0, r)
        W[r] = (synth.int4_codes(wl.seed, uid, N, K), synth.group_scales(wl.seed, uid, N, K))
    layer_bytes = shape.layer_bytes()
    tids = [{r: sess.register(*W[r], hbm=True, host=(c == 0)) for r in roles} for c in range(R)]
    descs = [atsi.atsi_dense_layer(shape.n_heads, shape.n_kv, shape.head_dim, 1e-6,
                                   *[t[r] for r in ("q", "k", "v", "o", "gate", "up", "down")]) for t in tids]
    Mp = wl.prefill_m
    h1 = torch.from_numpy(synth.activations(wl.seed, 1, 1, shape.hidden)).to(dev)
    hp = torch.from_numpy(synth.activations(wl.seed, 2, Mp, shape.hidden)).to(dev)
    cs.wait_stream(torch.cuda.current_stream())

    # a dense layer does the same work whatever h holds, so timed calls keep
    # updating h in place (the MoE stack below restores its inputs instead)
    def layer(c, h, M):
        atsi.atsi_decoder_layer(sess.ctx, descs[c], h.data_ptr(), M, 0, 0, None)

    # ------------------------------------------------------------ decode, HBM-resident (value)
    decode_s = steps_timed = n_warm = per_replay = decode_gbs = 0
    if not args.roofline_only:
        reps = 4

        def decode_round():
            for _ in range(reps):
                for c in range(R):
                    layer(c, h1, 1)

        g = graph_of(cs, decode_round)
        per_replay = reps * R
        n_replay = max(1, args.steps // per_replay)
        n_warm = max(1, args.warmup // per_replay)
        timer.run(g.replay, n_warm)
        decode_s = timer.run(g.replay, n_replay) / per_replay
        steps_timed = n_replay * per_replay
        decode_gbs = layer_bytes / decode_s / 1e9
        log(f"decode layer {decode_s * 1e6:.2f} us -> {decode_gbs:.1f} GB/s ({steps_timed} steps)")

    # ------------------------------------------------------------ dominant kernels
    xs = {r: torch.from_numpy(synth.activations(wl.seed, 50 + i, Mp, shape.kn(r)[0])).to(dev)
          for i, r in enumerate(roles)}
    hg = torch.empty((Mp, shape.inter), dtype=torch.float16, device=dev)
    yg = torch.empty((Mp, shape.inter), dtype=torch.float16, device=dev)
    cs.wait_stream(torch.cuda.current_stream())
    K_g, N_g = shape.kn("gate")

    def gate_up_round(M, n):
        def f():
            for _ in range(n):
                for c in range(R):
                    atsi.atsi_swiglu_gate_up(sess.ctx, tids[c]["gate"], tids[c]["up"], xs["gate"].data_ptr(), M,
                                             hg.data_ptr())
        return f

    gk = graph_of(cs, gate_up_round(1, 8))
    t_gemv = timer.run(gk.replay, 10) / (8 * R)
    gemv_bytes = 2 * configs.qbytes(K_g, N_g)
    gemv_gbs = gemv_bytes / t_gemv / 1e9
    log(f"gate/up GEMV {t_gemv * 1e6:.2f} us -> {gemv_gbs:.1f} GB/s")
    gm = graph_of(cs, gate_up_round(Mp, 1))
    t_gemm = timer.run(gm.replay, 4) / R
    gemm_flops = 2.0 * 2.0 * Mp * K_g * N_g
    gemm_tfs = gemm_flops / t_gemm / 1e12
    log(f"gate/up GEMM {t_gemm * 1e6:.1f} us -> {gemm_tfs:.1f} TFLOP/s")
    if args.roofline_only:
        # copy of known size: calibrates the FETCH_SIZE / WRITE_SIZE counters
        src = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        sess.close()
        print(json.dumps({"roofline_only": True, "gate_up_gemv_us": round(t_gemv * 1e6, 3),
                          "gate_up_gemm_us": round(t_gemm * 1e6, 2), "copy_bytes": 256 << 20}), flush=True)
        return 0

    # the standalone gate GEMV / GEMM (same kernels as the q, k, v, o launches)
    def gate_round(M, n):
        def f():
            for _ in range(n):
                for c in range(R):
                    atsi.atsi_linear(sess.ctx, tids[c]["gate"], xs["gate"].data_ptr(), M, yg.data_ptr())
        return f

    g1 = graph_of(cs, gate_round(1, 8))
    t_gate1 = timer.run(g1.replay, 10) / (8 * R)
    log(f"gate GEMV {t_gate1 * 1e6:.2f} us -> {configs.qbytes(K_g, N_g) / t_gate1 / 1e9:.1f} GB/s")

    # ------------------------------------------------------------ prefill 512, HBM-resident
    pf_state = {"i": 0}

    def prefill_once():
        layer(pf_state["i"] % R, hp, Mp)
        pf_state["i"] += 1

    timer.run(prefill_once, 2)
    prefill_s = timer.run(prefill_once, max(4, min(20, args.steps // 10)))
    prefill_flops = sum(2.0 * Mp * shape.kn(r)[0] * shape.kn(r)[1] for r in roles)
    prefill_tps = Mp / prefill_s
    log(f"prefill layer {prefill_s * 1e3:.3f} ms -> {prefill_tps:.0f} tok/s, "
        f"{prefill_flops / prefill_s / 1e12:.1f} TFLOP/s")

    # ------------------------------------------------------------ PCIe ceiling: one large pinned H2D copy
    pin = torch.empty(256 << 20, dtype=torch.uint8).pin_memory()
    dst = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
    cs.wait_stream(torch.cuda.current_stream())
    timer.run(lambda: dst.copy_(pin, non_blocking=True), 1)
    h2d_gbs = (256 << 20) / timer.run(lambda: dst.copy_(pin, non_blocking=True), 4) / 1e9
    del pin, dst
    log(f"pinned H2D ceiling {h2d_gbs:.1f} GB/s")

    # ------------------------------------------------------------ streamed placement (PCIe-inclusive)
    # Timing starts right after the placement is set (slots empty), over many
    # calls, so copies issued ahead of the timed window cannot hide in it.
    host_roles = [r for r, m in zip(roles, configs.dense_layer_host_mask()) if m]
    mask = [0] * len(sess.shapes)
    for r in host_roles:
        mask[tids[0][r]] = 1
    host_bytes = sum(configs.qbytes(*shape.kn(r)) for r in host_roles)
    order = [tids[0][r] for r in ("q", "k", "v", "o", "gate", "up", "down")]
    sess.set_placement(mask)
    sess.set_schedule(order)
    n_sd = 40
    st_dec, h2d_dec = h2d_timed(sess, timer, lambda: layer(0, h1, 1), n_sd)
    sess.set_placement(mask)
    sess.set_schedule(order)
    st_pf, h2d_pf = h2d_timed(sess, timer, lambda: layer(0, hp, Mp), 10)
    sess.set_schedule([])
    sess.set_placement([0] * len(sess.shapes))
    log(f"streamed decode {st_dec * 1e3:.3f} ms, prefill {st_pf * 1e3:.3f} ms ({host_roles} on host, "
        f"{host_bytes / 1e6:.1f} MB; copied per call {h2d_dec / 1e6:.1f} / {h2d_pf / 1e6:.1f} MB) -> PCIe "
        f"{h2d_dec / st_dec / 1e9:.1f} GB/s")

    moe = None if args.no_moe else bench_moe(sess, timer, args)
    stacks = None
    if not args.no_stacks:
        sess.close()
        stacks = {"dense_stack": bench_dense_stack(timer_cls=Timer, h2d_gbs=h2d_gbs),
                  "moe_stack": bench_moe_stack(timer_cls=Timer)}

    placement = bench_placement_solver()
    log(f"placement solver: {placement}")

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(W, shape, args.cpu_seconds, layer_bytes)
        log(f"cpu baseline {cpu}")

    out = {
        "metric": METRIC,
        "value": round(decode_gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": steps_timed,
        "warmup": n_warm * per_replay,
        "ms_per_step": round(decode_s * 1e3, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {
            "workload": "dense_layer: one 8B-shaped decoder layer, block-int4 g32 weights (Q 4096x4096, "
                        "K/V 4096x1024, O 4096x4096, gate/up 4096x14336, down 14336x4096; 122.7 MB), "
                        "RMS-norm, context-length-1 GQA, SwiGLU, residuals",
            "decode_batch": 1, "prefill_tokens": Mp, "layer_bytes": layer_bytes,
            "placement": "all HBM-resident for value; seeded mask (3 of 7 tensors on host) under 'streamed'",
            "mall_rotation_copies": R,
        },
        "pct_hbm_peak": round(100 * decode_gbs / HBM_PEAK_GBS, 2),
        "prefill_tokens_per_s": round(prefill_tps, 1),
        "prefill_ms_per_step": round(prefill_s * 1e3, 4),
        "prefill_pct_mfma": round(100 * prefill_flops / prefill_s / 1e12 / MFMA_F16_PEAK_TFLOPS, 2),
        "roofline": {"bound": "hbm", "achieved": round(gemv_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gemv_gbs / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic("gemv_gate_up", "q4_gemv"),
                     "kernel": "q4_gemv1_kernel<7,true,4>: SwiGLU gate/up, two 4096x14336 tensors, batch 1",
                     "bytes_per_launch": gemv_bytes, "avg_us": round(t_gemv * 1e6, 3)},
        "roofline_prefill": {"bound": "mfma", "achieved": round(gemm_tfs, 1), "peak": MFMA_F16_PEAK_TFLOPS,
                             "unit": "TFLOP/s", "frac": round(gemm_tfs / MFMA_F16_PEAK_TFLOPS, 4),
                             "traffic": measured_traffic("gemm_gate_up", "q4_gemm"),
                             "kernel": "q4_gemm_wide_kernel<true,false,false>: SwiGLU gate/up, two 4096x14336 "
                                       "tensors, 512 tokens",
                             "flops_per_launch": gemm_flops, "avg_us": round(t_gemm * 1e6, 2)},
        "gate_gemv_us": round(t_gate1 * 1e6, 3),
        "pcie_h2d_ceiling_GBps": round(h2d_gbs, 2),
        "streamed": {"host_tensors": host_roles, "host_bytes": host_bytes,
                     "decode_ms": round(st_dec * 1e3, 4), "prefill_ms": round(st_pf * 1e3, 4),
                     "decode_weight_GBps_pcie_inclusive": round(layer_bytes / st_dec / 1e9, 2),
                     "decode_h2d_bytes_per_call": int(h2d_dec), "prefill_h2d_bytes_per_call": int(h2d_pf),
                     "decode_pcie_GBps": round(h2d_dec / st_dec / 1e9, 2),
                     "decode_pct_of_h2d_ceiling": round(100 * h2d_dec / st_dec / 1e9 / h2d_gbs, 1),
                     "prefill_exposed_ms": round(max(0.0, st_pf - prefill_s) * 1e3, 4),
                     "prefill_tokens_per_s": round(Mp / st_pf, 1)},
        "moe": moe,
        "stacks": stacks,
        "placement_solver": placement,
        "cpu_baseline": cpu,
    }
    if args.no_stacks:
        sess.close()
    print(json.dumps(out), flush=True)
    return 0


def bench_moe(sess, timer, args):
    """30B-A3B-shaped MoE layer: decode (batch 1) and 512-token prefill."""
    import torch

    import synth
    from synth import configs
    from synth.calibrate_router_bias import load_bias
    from paper_2607_10183_amd import atsi

    wl = configs.MOE_LAYER
    shp = wl.moe
    E, H, I, k = shp.n_experts, shp.hidden, shp.inter, shp.top_k
    dev = torch.device("cuda", 0)
    log("generating MoE weights")
    tids = [[], [], []]
    for e in range(E):
        group = []
        for j, (n, kk) in enumerate(((I, H), (I, H), (H, I))):
            uid = configs.expert_uid(0, e, ("gate", "up", "down")[j])
            group.append((synth.int4_codes(wl.seed, uid, n, kk), synth.group_scales(wl.seed, uid, n, kk)))
        for j, t in enumerate(sess.register_group(group, hbm=True, host=True)):
            tids[j].append(t)
    wr = torch.from_numpy(synth.router_weights(wl.seed, configs.router_uid(0), H, E)).to(dev)
    bias = torch.from_numpy(load_bias()).to(dev)
    moe_l = sess.moe_layer(wr, *tids, top_k=k, router_bias=bias)

    def layer(x, y):
        atsi.atsi_moe_ffn(sess.ctx, moe_l.desc, x.data_ptr(), x.shape[0], y.data_ptr(), None)

    n_tok = 64
    xd = torch.from_numpy(synth.activations(wl.seed, 7, n_tok, H)).to(dev)
    xp = torch.from_numpy(synth.activations(wl.seed, 8, wl.prefill_m, H)).to(dev)
    yd = torch.empty((n_tok, H), dtype=torch.float16, device=dev)
    yp = torch.empty((wl.prefill_m, H), dtype=torch.float16, device=dev)
    sess.cs.wait_stream(torch.cuda.current_stream())
    expert_bytes = shp.expert_bytes()

    def decode_all():  # 64 different tokens, one at a time
        for t in range(n_tok):
            layer(xd[t:t + 1], yd[t:t + 1])

    # routed bytes actually touched per decode token (8 distinct experts)
    routed_bytes = k * expert_bytes
    g = graph_of(sess.cs, decode_all)
    timer.run(g.replay, 2)
    dec_s = timer.run(g.replay, 5) / n_tok
    timer.run(lambda: layer(xp, yp), 2)
    pf_s = timer.run(lambda: layer(xp, yp), 10)
    pf_flops = 2.0 * wl.prefill_m * k * 3 * H * I
    log(f"moe decode {dec_s * 1e6:.1f} us/token ({routed_bytes / dec_s / 1e9:.0f} GB/s routed), "
        f"prefill {pf_s * 1e3:.3f} ms -> {wl.prefill_m / pf_s:.0f} tok/s, {pf_flops / pf_s / 1e12:.1f} TFLOP/s")

    host_exp = configs.moe_host_experts()
    mask = list(sess.placement)
    for j in range(3):
        for e in range(E):
            mask[tids[j][e]] = int(host_exp[e])
    sess.set_placement(mask)
    st_dec, h2d_dec = h2d_timed(sess, timer, lambda: [layer(xd[t:t + 1], yd[t:t + 1]) for t in range(32)], 1)
    st_dec, h2d_dec = st_dec / 32, h2d_dec / 32
    st_pf, h2d_pf = h2d_timed(sess, timer, lambda: layer(xp, yp), 3)
    # the same placement with the routed host experts read in place (zero-copy):
    # nothing is copied, the PCIe bytes are those the copy path moves
    sess.set_zero_copy(True)
    timer.run(lambda: [layer(xd[t:t + 1], yd[t:t + 1]) for t in range(32)], 1)
    zc_dec = timer.run(lambda: [layer(xd[t:t + 1], yd[t:t + 1]) for t in range(32)], 1) / 32
    gz = graph_of(sess.cs, decode_all)
    timer.run(gz.replay, 1)
    zc_graph = timer.run(gz.replay, 3) / n_tok
    sess.set_zero_copy(False)
    for j in range(3):
        for e in range(E):
            mask[tids[j][e]] = 0
    sess.set_placement(mask)
    log(f"moe streamed decode {st_dec * 1e3:.3f} ms/token ({h2d_dec / 1e6:.1f} MB copied), prefill "
        f"{st_pf * 1e3:.2f} ms ({h2d_pf / 1e6:.1f} MB copied, {h2d_pf / st_pf / 1e9:.1f} GB/s PCIe); "
        f"zero-copy decode {zc_dec * 1e3:.3f} ms/token ({zc_graph * 1e3:.3f} graph-replayed)")
    return {"workload": "moe_layer: 128 experts of SwiGLU 768 over hidden 2048, top-8, capped Zipf(1.1) loads",
            "decode_us_per_token": round(dec_s * 1e6, 2),
            "decode_routed_GBps": round(routed_bytes / dec_s / 1e9, 1),
            "prefill_tokens_per_s": round(wl.prefill_m / pf_s, 1),
            "prefill_ms": round(pf_s * 1e3, 4),
            "prefill_TFLOPs": round(pf_flops / pf_s / 1e12, 2),
            "streamed_40pct_host": {"decode_ms_per_token": round(st_dec * 1e3, 4),
                                    "decode_h2d_bytes_per_token": int(h2d_dec),
                                    "decode_pcie_GBps": round(h2d_dec / st_dec / 1e9, 2),
                                    "prefill_ms": round(st_pf * 1e3, 3),
                                    "prefill_h2d_bytes": int(h2d_pf),
                                    "prefill_pcie_GBps": round(h2d_pf / st_pf / 1e9, 2),
                                    "zero_copy_decode_ms_per_token": round(zc_dec * 1e3, 4),
                                    "zero_copy_decode_ms_per_token_graph": round(zc_graph * 1e3, 4),
                                    "zero_copy_decode_pcie_GBps": round(h2d_dec / zc_graph / 1e9, 2)}}


def bench_dense_stack(timer_cls, h2d_gbs, steps=6):
    """32 8B-shaped layers, a decode loop over 8 sequences (hidden state
    renormalised after every layer), 30 % of the int4 bytes on host by
    seeded score, streamed each step with schedule-driven prefetch."""
    import torch

    import synth
    from synth import configs
    from paper_2607_10183_amd.session import Session

    wl = configs.DENSE_STACK
    shape = wl.dense
    mask = configs.dense_stack_host_mask()
    log("generating dense-stack weights (32 layers)")
    sess = Session(workspace_bytes=2 << 30, n_slots=24)
    timer = timer_cls(sess.cs)
    tids = []
    for layer in range(wl.n_layers):
        t = {}
        for j, r in enumerate(configs.ROLES):
            K, N = shape.kn(r)
            uid = configs.dense_uid(layer, r)
            t[r] = sess.register(synth.int4_codes(wl.seed, uid, N, K), synth.group_scales(wl.seed, uid, N, K),
                                 hbm=True, host=bool(mask[layer, j]))
        tids.append(t)
    total_bytes = wl.n_layers * shape.layer_bytes()
    host_bytes = sum(configs.qbytes(*shape.kn(configs.ROLES[j])) for layer in range(wl.n_layers)
                     for j in range(len(configs.ROLES)) if mask[layer, j])
    h = torch.from_numpy(synth.activations(wl.seed, 1, wl.decode_m, shape.hidden)).cuda()
    sess.cs.wait_stream(torch.cuda.current_stream())

    def step():
        for layer in range(wl.n_layers):
            sess.decoder_layer(tids[layer], h, shape.n_heads, shape.n_kv, shape.head_dim, 1e-6, renorm_out=True)

    # all weights in HBM
    timer.run(step, 1)
    t_hbm = timer.run(step, steps)
    # the seeded 30 % mask, streamed with the schedule (execution order)
    pl = [0] * len(sess.shapes)
    for layer in range(wl.n_layers):
        for j, r in enumerate(configs.ROLES):
            pl[tids[layer][r]] = int(mask[layer, j])
    sess.set_placement(pl)
    sess.set_schedule([tids[layer][r] for layer in range(wl.n_layers) for r in configs.ROLES])
    timer.run(step, 1)
    t_st, h2d_st = h2d_timed(sess, timer, step, steps)
    sess.close()
    m = wl.decode_m
    log(f"dense stack: decode step {t_hbm * 1e3:.2f} ms all-HBM ({total_bytes / t_hbm / 1e9:.0f} GB/s), "
        f"{t_st * 1e3:.2f} ms with {host_bytes / 1e9:.2f} GB on host ({h2d_st / 1e9:.2f} GB copied per step, "
        f"{h2d_st / t_st / 1e9:.1f} GB/s PCIe)")
    return {"workload": "dense_stack: 32 8B-shaped layers, decode loop of 8 sequences, hidden state renormalised "
                        "after every layer, 30 % of the int4 bytes on host by seeded score",
            "layers": wl.n_layers, "sequences": m, "steps_timed": steps,
            "total_bytes": total_bytes, "host_bytes": host_bytes,
            "all_hbm": {"ms_per_step": round(t_hbm * 1e3, 3), "tokens_per_s": round(m / t_hbm, 1),
                        "weight_GBps": round(total_bytes / t_hbm / 1e9, 1)},
            "streamed": {"ms_per_step": round(t_st * 1e3, 3), "tokens_per_s": round(m / t_st, 1),
                         "weight_GBps_pcie_inclusive": round(total_bytes / t_st / 1e9, 1),
                         "h2d_bytes_per_step": int(h2d_st),
                         "pcie_GBps": round(h2d_st / t_st / 1e9, 2),
                         "pct_of_h2d_ceiling": round(100 * h2d_st / t_st / 1e9 / h2d_gbs, 1),
                         "tokens_per_s_256_steps": round(m / t_st, 1)}}


def bench_moe_stack(timer_cls):
    """One 235B-A22B-shaped layer (attention 64 / 4 heads of 128 over hidden
    4096, 128 experts of SwiGLU 1536, top-8), timed at decode (batch 1) and
    prefill (2048 tokens), all-HBM and with 40 % of its experts on host;
    the 94-layer figures are 94 x one layer."""
    import torch

    import synth
    from synth import configs
    from synth.calibrate_router_bias import load_bias
    from paper_2607_10183_amd.session import MoEDecoderLayer, Session

    wl = configs.MOE_STACK
    ds, ms = wl.dense, wl.moe
    H, E, I, k = ms.hidden, ms.n_experts, ms.inter, ms.top_k
    layer = 0
    log("generating one MoE-stack layer")
    sess = Session(workspace_bytes=3 << 30, n_slots=24)
    timer = timer_cls(sess.cs)
    a = {r: sess.register(synth.int4_codes(wl.seed, configs.dense_uid(layer, r), ds.kn(r)[1], ds.kn(r)[0]),
                          synth.group_scales(wl.seed, configs.dense_uid(layer, r), ds.kn(r)[1], ds.kn(r)[0]))
         for r in ("q", "k", "v", "o")}
    tids = [[], [], []]
    for e in range(E):
        group = []
        for p, (n, kk) in zip(("gate", "up", "down"), ((I, H), (I, H), (H, I))):
            uid = configs.expert_uid(layer, e, p)
            group.append((synth.int4_codes(wl.seed, uid, n, kk), synth.group_scales(wl.seed, uid, n, kk)))
        for j, t in enumerate(sess.register_group(group, hbm=True, host=True)):
            tids[j].append(t)
    wr = torch.from_numpy(synth.router_weights(wl.seed, configs.router_uid(layer), H, E)).cuda()
    moe = sess.moe_layer(wr, *tids, top_k=k, router_bias=torch.from_numpy(load_bias()).cuda())
    L = MoEDecoderLayer(moe, a["q"], a["k"], a["v"], a["o"], ds.n_heads, ds.n_kv, ds.head_dim, 1e-6)
    # The layer updates h in place (h += attention + MoE) and routing depends
    # on h, so every timed call starts from the same hidden states: restored
    # from a pristine copy inside the call, with the copy's own time taken off.
    hd0 = torch.from_numpy(synth.activations(wl.seed, 1, 32, H)).cuda()
    hp0 = torch.from_numpy(synth.activations(wl.seed, 2, wl.prefill_m, H)).cuda()
    hd, hp = hd0.clone(), hp0.clone()
    sess.cs.wait_stream(torch.cuda.current_stream())
    attn_bytes = sum(configs.qbytes(*ds.kn(r)) for r in ("q", "k", "v", "o"))
    expert_bytes = 3 * configs.qbytes(H, I)
    t_cd = timer.run(lambda: hd.copy_(hd0), 20)
    t_cp = timer.run(lambda: hp.copy_(hp0), 20)

    def dec():
        hd.copy_(hd0)
        for t in range(32):
            L(hd[t:t + 1])

    def pf():
        hp.copy_(hp0)
        L(hp)

    def measure():
        timer.run(dec, 1)
        t_dec, b_dec = h2d_timed(sess, timer, dec, 2)
        timer.run(pf, 1)
        t_pf, b_pf = h2d_timed(sess, timer, pf, 3)
        return (t_dec - t_cd) / 32, t_pf - t_cp, b_dec / 32, b_pf

    d_hbm, p_hbm, _, _ = measure()
    host_exp = configs.moe_host_experts(frac=0.40, seed=wl.seed, layer=layer)
    pl = list(sess.placement)
    for j in range(3):
        for e in range(E):
            pl[tids[j][e]] = int(host_exp[e])
    sess.set_placement(pl)
    d_st, p_st, d_h2d, p_h2d = measure()
    sess.set_zero_copy(True)
    timer.run(dec, 1)
    d_zc = (timer.run(dec, 2) - t_cd) / 32
    sess.set_zero_copy(False)
    # experts the prefill actually routes to, and how many of those are on host
    dbg = L(hp0.clone(), debug=True)
    sess.sync()
    counts = dbg["counts"].cpu().numpy()
    n_act = int((counts > 0).sum())
    n_host_act = int(((counts > 0) & (host_exp > 0)).sum())
    sess.close()
    pf_flops = 2.0 * wl.prefill_m * (attn_bytes * 16 / 9 + k * expert_bytes * 16 / 9)  # 2 M K N per weight
    log(f"moe stack layer: decode {d_hbm * 1e3:.3f} ms ({d_st * 1e3:.3f} streamed), prefill {p_hbm * 1e3:.2f} ms "
        f"({p_st * 1e3:.2f} streamed, {n_host_act} of {n_act} active experts on host, {p_h2d / 1e6:.0f} MB "
        f"copied -> {p_h2d / p_st / 1e9:.1f} GB/s PCIe); decode copies {d_h2d / 1e6:.1f} MB/token "
        f"({d_zc * 1e3:.3f} ms with zero-copy reads); "
        f"x94: {94 * d_hbm * 1e3:.1f} ms/token all-HBM")
    return {"workload": "moe_stack: one 235B-A22B-shaped layer (attention 64/4 heads of 128, hidden 4096, "
                        "128 experts of SwiGLU 1536, top-8, capped-Zipf routing); 94-layer figures are 94 x the layer",
            "all_hbm": {"decode_ms_per_layer": round(d_hbm * 1e3, 4), "prefill_ms_per_layer": round(p_hbm * 1e3, 3),
                        "decode_tokens_per_s_94_layers": round(1.0 / (94 * d_hbm), 2),
                        "prefill_tokens_per_s_94_layers": round(wl.prefill_m / (94 * p_hbm), 1),
                        "prefill_TFLOPs": round(pf_flops / p_hbm / 1e12, 1)},
            "prefill_active_experts": n_act, "prefill_active_host_experts": n_host_act,
            "streamed_40pct_experts": {"decode_ms_per_layer": round(d_st * 1e3, 4),
                                       "prefill_ms_per_layer": round(p_st * 1e3, 3),
                                       "decode_h2d_bytes_per_layer": int(d_h2d),
                                       "decode_pcie_GBps": round(d_h2d / d_st / 1e9, 2),
                                       "prefill_h2d_bytes_per_layer": int(p_h2d),
                                       "prefill_pcie_GBps": round(p_h2d / p_st / 1e9, 2),
                                       "decode_tokens_per_s_94_layers": round(1.0 / (94 * d_st), 2),
                                       "prefill_tokens_per_s_94_layers": round(wl.prefill_m / (94 * p_st), 1),
                                       "zero_copy_decode_ms_per_layer": round(d_zc * 1e3, 4),
                                       "zero_copy_decode_pcie_GBps": round(d_h2d / d_zc / 1e9, 2),
                                       "zero_copy_decode_tokens_per_s_94_layers": round(1.0 / (94 * d_zc), 2)}}


def bench_placement_solver(reps: int = 3):
    """Host time of atsi_solve_placement on the 94-layer 235B-A22B-shaped
    model: per layer q, k, v, o, the router and the gate / up / down expert
    operators (128 experts each, one tensor per operator), 1 MiB granularity,
    a budget of half the model's 131.5 GB.  Gains are seeded (each tensor's
    size over 20 GB/s, times U(0.5, 1.5)); switch costs 20 us."""
    from paper_2607_10183_amd import atsi
    layer = [18874368, 1179648, 1179648, 18874368, 1048576, 128 * 3538944, 128 * 3538944, 128 * 3538944]
    expert_role = [0, 0, 0, 0, 0, 1, 1, 1]
    s = [float(v) for _ in range(94) for v in layer]
    expert = [e for _ in range(94) for e in expert_role]
    rng = np.random.default_rng(2607)
    r = list(np.array(s) / 2e10 * rng.uniform(0.5, 1.5, len(s)))
    c = [2e-5] * len(s)
    budget = 0.5 * sum(s)
    best = float("inf")
    for _ in range(reps):
        t0 = time.perf_counter()
        b, obj = atsi.atsi_solve_placement(s, r, c, budget, float(1 << 20), expert)
        best = min(best, time.perf_counter() - t0)
    units = int((budget - sum(x for x, e in zip(s, expert) if not e)) // (1 << 20))
    return {"workload": "static placement of the 94-layer 235B-A22B-shaped model (752 tensors), 1 MiB "
                        "granularity, budget half the model", "tensors": len(s), "budget_units": units,
            "gpu_resident_bytes": int(sum(x for x, g in zip(s, b) if g)), "objective_s": round(obj, 6),
            "host_ms": round(best * 1e3, 2)}


def cpu_baseline(W, shape, budget_s, layer_bytes):
    """The fp64 oracle's decode step of the same layer (batch 1), timed on the host."""
    import oracle
    import synth
    try:
        from threadpoolctl import threadpool_info
        blas = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover
        blas = 1
    h = synth.activations(1002, 1, 1, shape.hidden)
    n = 0
    t0 = time.perf_counter()
    while True:
        oracle.decoder_layer(h, W, shape.n_heads, shape.n_kv, shape.head_dim, 1e-6)
        n += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = (time.perf_counter() - t0) / n
    return {"value": round(layer_bytes / dt / 1e9, 4), "unit": "GB/s", "cores": int(blas), "kind": "oracle",
            "sample": f"{n} batch-1 decode steps of the dense layer (fp64 dequant + BLAS matmul), "
                      f"{dt:.2f} s per step",
            "host_cpus": len(os.sched_getaffinity(0))}


def summarize(trace_dir: str, fetch_dir: str, write_dir: str, commands: dict) -> None:
    """Write profiles/kernels_dense_layer_moe_layer.md (per-kernel durations of a
    full bench run) and profiles/traffic.json + .md (HBM bytes per launch of
    the two roofline kernels from FETCH_SIZE / WRITE_SIZE, scaled by what the
    same counters read for a 256 MiB device copy) from rocprofv3 CSV output."""
    import csv
    import glob

    def one(pattern):
        hits = glob.glob(os.path.join(pattern))
        if not hits:
            raise FileNotFoundError(pattern)
        return hits[0]

    prof = os.path.join(ROOT, "profiles")
    stats = list(csv.DictReader(open(one(os.path.join(trace_dir, "*kernel_stats.csv")))))
    lines = ["# Kernel durations: dense_layer + moe_layer bench run", "",
             "Command (from the repository root, on one MI355X):", "",
             "    " + commands["trace"], "",
             "| kernel | calls | avg us | min us | max us | share |", "|---|---|---|---|---|---|"]
    for r in sorted(stats, key=lambda r: -float(r["TotalDurationNs"]))[:24]:
        lines.append(f"| `{r['Name'][:110]}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.1f}% |")
    with open(os.path.join(prof, "kernels_dense_layer_moe_layer.md"), "w") as fh:
        fh.write("\n".join(lines) + "\n")

    def counter(dirname, name):
        per = {}
        for r in csv.DictReader(open(one(os.path.join(dirname, "*counter_collection.csv")))):
            if r["Counter_Name"] != name:
                continue
            per.setdefault(r["Kernel_Name"], {}).setdefault(r["Dispatch_Id"], 0.0)
            per[r["Kernel_Name"]][r["Dispatch_Id"]] += float(r["Counter_Value"])
        return {k: sorted(v.values()) for k, v in per.items()}

    def pick(per, needle):
        ks = [k for k in per if needle in k]
        if not ks:
            raise KeyError(needle)
        vals = per[ks[0]]
        return ks[0], vals[len(vals) // 2]  # median over dispatches, KiB

    fetch, write = counter(fetch_dir, "FETCH_SIZE"), counter(write_dir, "WRITE_SIZE")
    copy_bytes = 256 << 20
    # the device-to-device copy runs as the runtime's copy kernel; its three
    # 256 MiB dispatches are the largest ones
    f_copy = sorted(fetch["__amd_rocclr_copyBuffer"])[-2]
    w_copy = sorted(write["__amd_rocclr_copyBuffer"])[-2]
    f_scale, w_scale = copy_bytes / (f_copy * 1024), copy_bytes / (w_copy * 1024)
    out = {"calibration": {"copy_bytes": copy_bytes, "fetch_kib": f_copy, "write_kib": w_copy,
                           "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4)}}
    md = ["# HBM traffic of the roofline kernels (FETCH_SIZE, WRITE_SIZE)", "",
          "Commands (from the repository root, one counter per run):", "",
          "    " + commands["fetch"], "    " + commands["write"], "",
          f"Calibration: a {copy_bytes >> 20} MiB device copy reads {f_copy:.0f} KiB (FETCH_SIZE) and writes "
          f"{w_copy:.0f} KiB (WRITE_SIZE) per dispatch; scale factors {f_scale:.4f} and {w_scale:.4f}.", "",
          "| kernel | FETCH KiB | WRITE KiB | HBM bytes per launch (scaled) | algorithmic bytes |",
          "|---|---|---|---|---|"]
    for key, needle, kind, algo in (("gemv_gate_up", "q4_gemv1_kernel<7, true, 4>", "q4_gemv", 66060288),
                                    ("gemm_gate_up", "q4_gemm_wide_kernel<true, false, false>", "q4_gemm",
                                     66060288 + 2 * 512 * 4096 + 2 * 512 * 14336)):
        kname, f = pick(fetch, needle)
        _, w = pick(write, needle)
        bytes_ = int(round(f * 1024 * f_scale + w * 1024 * w_scale))
        out[key] = {"kernel": kname, "fetch_kib": f, "write_kib": w, "hbm_bytes_per_launch": bytes_,
                    "algorithmic_bytes": algo, "source_sha256_16": kernel_hash(kind)}
        md.append(f"| `{kname[:90]}` | {f:.0f} | {w:.0f} | {bytes_} | {algo} |")
    with open(os.path.join(prof, "traffic.json"), "w") as fh:
        json.dump(out, fh, indent=1)
    with open(os.path.join(prof, "traffic.md"), "w") as fh:
        fh.write("\n".join(md) + "\n")


if __name__ == "__main__":
    if len(sys.argv) > 1 and sys.argv[1] == "--summarize":
        # bench.py --summarize TRACE_DIR FETCH_DIR WRITE_DIR
        summarize(sys.argv[2], sys.argv[3], sys.argv[4], {
            "trace": "rocprofv3 --kernel-trace --stats -f csv -d gpurun_out/prof_trace -o bench -- "
                     "python -u bench.py --no-cpu-baseline",
            "fetch": "rocprofv3 --pmc FETCH_SIZE -f csv -d gpurun_out/prof_fetch -o f -- "
                     "python -u bench.py --roofline-only",
            "write": "rocprofv3 --pmc WRITE_SIZE -f csv -d gpurun_out/prof_write -o w -- "
                     "python -u bench.py --roofline-only"})
        sys.exit(0)
    sys.exit(main())
