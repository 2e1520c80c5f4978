"""Device-memory and stream plumbing around the C ABI, using PyTorch.

PyTorch only allocates (HBM tensors, pinned host tensors, the workspace) and
creates the two streams; all compute goes through libatsi.so.
"""
from __future__ import annotations

import numpy as np
import torch

from . import atsi


class Session:
    """One atsi context on one GPU with its own compute and transfer streams."""

    def __init__(self, workspace_bytes: int = 1 << 30, n_slots: int = 4, device: int = 0,
                 two_transfer_streams: bool = True):
        if not torch.cuda.is_available():
            raise RuntimeError("no GPU visible to torch; the atsi library has no CPU path")
        self.device = torch.device("cuda", device)
        self.cs = torch.cuda.Stream(device=self.device)
        self.ts = torch.cuda.Stream(device=self.device)
        self.ts2 = torch.cuda.Stream(device=self.device) if two_transfer_streams else None
        self.ws = torch.empty(workspace_bytes, dtype=torch.uint8, device=self.device)
        # pinned host buffer for the per-expert counts of MoE calls with streamed experts
        self.counts_host = torch.empty(128, dtype=torch.int32).pin_memory()
        self.ctx = atsi.atsi_create(device, self.cs.cuda_stream, self.ts.cuda_stream,
                                    self.ts2.cuda_stream if self.ts2 is not None else 0, self.ws.data_ptr(),
                                    workspace_bytes, self.counts_host.data_ptr(), n_slots)
        self._keep: list = []
        self.shapes: list[tuple[int, int]] = []
        self.placement: list[int] = []  # current host mask, mirrors the library's
        self.backends: list[int] = []   # current runtime assignment, 1 = CPU
        self.pool = 0
        self.staging = None

    # ---------------------------------------------------------------- tensors
    def register(self, codes: np.ndarray, scales: np.ndarray, hbm: bool = True, host: bool = False) -> int:
        """Register a block-int4 tensor (codes uint8[N][K/2], scales fp16[N][K/32])
        with an HBM copy and/or a pinned host copy."""
        N, kb = codes.shape
        K = 2 * kb
        sbits = np.ascontiguousarray(scales, dtype=np.float16).view(np.uint16)
        dc = ds = hc = hs = 0
        if hbm:
            tc = torch.from_numpy(np.ascontiguousarray(codes)).to(self.device)
            tsc = torch.from_numpy(sbits.view(np.int16)).to(self.device)
            self._keep += [tc, tsc]
            dc, ds = tc.data_ptr(), tsc.data_ptr()
        if host:
            # codes then scales in one pinned buffer: the engine moves it with one copy
            buf = torch.empty(codes.nbytes + sbits.nbytes, dtype=torch.uint8).pin_memory()
            self._fill_host(buf, 0, codes, sbits)
            self._keep.append(buf)
            hc, hs = buf.data_ptr(), buf.data_ptr() + codes.nbytes
        torch.cuda.synchronize(self.device)
        tid = atsi.atsi_tensor_register(self.ctx, K, N, dc, ds, hc, hs)
        self.shapes.append((K, N))
        self.placement.append(0 if hbm else 1)
        self.backends.append(0)
        return tid

    @staticmethod
    def _fill_host(buf: torch.Tensor, off: int, codes: np.ndarray, sbits: np.ndarray) -> None:
        nb = buf.numpy()
        nb[off:off + codes.nbytes] = np.ascontiguousarray(codes).reshape(-1).view(np.uint8)
        nb[off + codes.nbytes:off + codes.nbytes + sbits.nbytes] = np.ascontiguousarray(sbits).reshape(-1).view(np.uint8)

    def register_group(self, tensors, hbm: bool = True, host: bool = True) -> list[int]:
        """Register several tensors whose host copies sit back to back in one
        pinned buffer (e.g. an expert's gate, up and down), so a streamed group
        can move with a single copy."""
        sb = [np.ascontiguousarray(sc, dtype=np.float16).view(np.uint16) for _, sc in tensors]
        sizes = [c.nbytes + s.nbytes for (c, _), s in zip(tensors, sb)]
        buf = torch.empty(sum(sizes), dtype=torch.uint8).pin_memory() if host else None
        tids, off = [], 0
        for (codes, _), sbits, size in zip(tensors, sb, sizes):
            N, kb = codes.shape
            dc = ds = hc = hs = 0
            if hbm:
                tc = torch.from_numpy(np.ascontiguousarray(codes)).to(self.device)
                tsc = torch.from_numpy(sbits.view(np.int16)).to(self.device)
                self._keep += [tc, tsc]
                dc, ds = tc.data_ptr(), tsc.data_ptr()
            if host:
                self._fill_host(buf, off, codes, sbits)
                hc, hs = buf.data_ptr() + off, buf.data_ptr() + off + codes.nbytes
            off += size
            tids.append((2 * kb, N, dc, ds, hc, hs))
        if buf is not None:
            self._keep.append(buf)
        torch.cuda.synchronize(self.device)
        out = []
        for K, N, dc, ds, hc, hs in tids:
            out.append(atsi.atsi_tensor_register(self.ctx, K, N, dc, ds, hc, hs))
            self.shapes.append((K, N))
            self.placement.append(0 if hbm else 1)
            self.backends.append(0)
        return out

    def register_device(self, codes_t: torch.Tensor, scales_t: torch.Tensor,
                        host_codes: torch.Tensor | None = None, host_scales: torch.Tensor | None = None) -> int:
        """Register tensors already in memory (device uint8/int16, optional pinned host copies)."""
        N, kb = codes_t.shape
        self._keep += [codes_t, scales_t] + [t for t in (host_codes, host_scales) if t is not None]
        tid = atsi.atsi_tensor_register(self.ctx, 2 * kb, N, codes_t.data_ptr(), scales_t.data_ptr(),
                                        host_codes.data_ptr() if host_codes is not None else 0,
                                        host_scales.data_ptr() if host_scales is not None else 0)
        self.shapes.append((2 * kb, N))
        self.placement.append(0)
        self.backends.append(0)
        return tid

    def register_host(self, K: int, N: int, host_codes: int, host_scales: int) -> int:
        """Register a tensor with only a pinned host copy at raw addresses (codes
        [N][K/2] then fp16 scales [N][K/32]); the caller keeps that memory alive."""
        tid = atsi.atsi_tensor_register(self.ctx, K, N, 0, 0, host_codes, host_scales)
        self.shapes.append((K, N))
        self.placement.append(1)
        self.backends.append(0)
        return tid

    def set_debug(self, poison: bool = False, serialize: bool = False) -> None:
        """Checking modes of the streaming engine (atsi_set_debug)."""
        atsi.atsi_set_debug(self.ctx, (atsi.DEBUG_POISON if poison else 0) | (atsi.DEBUG_SERIALIZE if serialize else 0))

    def set_zero_copy(self, enable: bool = True) -> None:
        """Decode MoE calls read host-resident experts in place (atsi_set_zero_copy)."""
        atsi.atsi_set_zero_copy(self.ctx, enable)

    def set_moe_light_rows(self, rows: int) -> None:
        """Prefill experts routed at most `rows` pairs take the light-expert
        kernels, the others the grouped GEMM (atsi_set_moe_light_rows)."""
        atsi.atsi_set_moe_light_rows(self.ctx, rows)

    def set_placement(self, host_mask) -> None:
        mask = [int(v) for v in host_mask]
        atsi.atsi_set_placement(self.ctx, mask)
        self.placement = mask
        self.backends = [b if m else 0 for b, m in zip(self.backends, mask)]

    # ---------------------------------------------------------------- hybrid CPU-GPU
    def attach_cpu(self, threads: int, staging_bytes: int = 64 << 20) -> None:
        """Attach the host-CPU backend: a pool of `threads` workers and a pinned
        staging buffer for the activations of CPU-run launches."""
        if self.pool:
            raise RuntimeError("a CPU backend is already attached")
        self.pool = atsi.atsi_cpu_pool_create(threads)
        self.staging = torch.empty(staging_bytes, dtype=torch.uint8).pin_memory()
        atsi.atsi_set_cpu_backend(self.ctx, self.pool, self.staging.data_ptr(), staging_bytes)

    def set_backends(self, on_cpu) -> None:
        """Runtime backend assignment (1 = the CPU backend; host-placed tensors only)."""
        a = [int(v) for v in on_cpu]
        atsi.atsi_set_backends(self.ctx, a)
        self.backends = a

    def set_timing(self, enable: bool = True) -> None:
        atsi.atsi_set_timing(self.ctx, enable)

    def timings(self) -> list:
        """Latest per-tensor measurements (t_gpu, t_cpu, d2h, h2d, w in seconds; NaN where none)."""
        return atsi.atsi_get_timings(self.ctx, len(self.shapes))

    def place(self, tid: int, host: bool) -> None:
        """Move one tensor between HBM and host, keeping the others where they are."""
        mask = list(self.placement)
        mask[tid] = int(host)
        self.set_placement(mask)

    # ---------------------------------------------------------------- compute
    def linear(self, tid: int, x: torch.Tensor, y: torch.Tensor | None = None) -> torch.Tensor:
        K, N = self.shapes[tid]
        assert x.dtype == torch.float16 and x.is_contiguous() and x.shape[-1] == K
        M = x.numel() // K
        if y is None:
            with torch.cuda.stream(self.cs):
                y = torch.empty((M, N), dtype=torch.float16, device=self.device)
        self._wait_torch()
        atsi.atsi_linear(self.ctx, tid, x.data_ptr(), M, y.data_ptr())
        self._torch_waits()
        return y

    def ffn(self, gate: int, up: int, down: int, x: torch.Tensor, y: torch.Tensor | None = None) -> torch.Tensor:
        H, I = self.shapes[gate]
        M = x.numel() // H
        if y is None:
            with torch.cuda.stream(self.cs):
                y = torch.empty((M, H), dtype=torch.float16, device=self.device)
        self._wait_torch()
        atsi.atsi_ffn_swiglu(self.ctx, gate, up, down, x.data_ptr(), M, y.data_ptr())
        self._torch_waits()
        return y

    def rmsnorm(self, x: torch.Tensor, eps: float = 1e-6, y: torch.Tensor | None = None) -> torch.Tensor:
        """y = x / rms(x) per row (unit gain); in place when y is x."""
        M, H = x.shape
        if y is None:
            with torch.cuda.stream(self.cs):
                y = torch.empty_like(x)
        self._wait_torch()
        atsi.atsi_rmsnorm(self.ctx, x.data_ptr(), M, H, eps, y.data_ptr())
        self._torch_waits()
        return y

    def gate_up(self, gate: int, up: int, x: torch.Tensor, h: torch.Tensor | None = None) -> torch.Tensor:
        """h = silu(x Wg) * (x Wu), one launch."""
        H, I = self.shapes[gate]
        M = x.numel() // H
        if h is None:
            with torch.cuda.stream(self.cs):
                h = torch.empty((M, I), dtype=torch.float16, device=self.device)
        self._wait_torch()
        atsi.atsi_swiglu_gate_up(self.ctx, gate, up, x.data_ptr(), M, h.data_ptr())
        self._torch_waits()
        return h

    def decoder_layer(self, tids: dict, h: torch.Tensor, n_heads: int, n_kv: int, head_dim: int,
                      eps: float = 1e-6, q_out: torch.Tensor | None = None, k_out: torch.Tensor | None = None,
                      renorm_out: bool = False, debug: bool = False):
        """In-place pre-norm decoder layer on h[M][H]; tids maps q,k,v,o,gate,up,down to tensor ids.
        renorm_out: the output is renormalised (h <- rms(h + FFN)), as between the layers of a stack.
        debug: also returns the intermediate activations {attn, h_attn, act[, sum32]}."""
        L = atsi.atsi_dense_layer(n_heads, n_kv, head_dim, eps, *[tids[r] for r in
                                                                  ("q", "k", "v", "o", "gate", "up", "down")],
                                  int(renorm_out))
        M, H = h.shape
        inter = self.shapes[tids["gate"]][1]
        out, dbg = self._layer_debug(M, H, n_heads * head_dim, inter, renorm_out) if debug else ({}, None)
        self._wait_torch()
        atsi.atsi_decoder_layer(self.ctx, L, h.data_ptr(), M, q_out.data_ptr() if q_out is not None else 0,
                                k_out.data_ptr() if k_out is not None else 0, dbg)
        self._torch_waits()
        return (h, out) if debug else h

    def _layer_debug(self, M: int, H: int, Hq: int, inter: int, sum32: bool):
        with torch.cuda.stream(self.cs):
            out = {"attn": torch.empty((M, Hq), dtype=torch.float16, device=self.device),
                   "h_attn": torch.empty((M, H), dtype=torch.float16, device=self.device)}
            if inter:
                out["act"] = torch.empty((M, inter), dtype=torch.float16, device=self.device)
            if sum32:
                out["sum32"] = torch.empty((M, H), dtype=torch.float32, device=self.device)
        dbg = atsi.atsi_layer_debug(*[out[n].data_ptr() if n in out else None for n in atsi.LAYER_DEBUG_FIELDS])
        return out, dbg

    def moe_layer(self, router_w: torch.Tensor, gate, up, down, top_k: int,
                  router_bias: torch.Tensor | None = None) -> "MoELayer":
        return MoELayer(self, router_w, gate, up, down, top_k, router_bias)

    def moe_bucket(self, idx: torch.Tensor, n_experts: int):
        """Bucket device idx int32 [M][k]; returns (counts, offsets, perm, inv_perm)."""
        M, k = idx.shape
        with torch.cuda.stream(self.cs):
            counts = torch.empty(n_experts, dtype=torch.int32, device=self.device)
            offsets = torch.empty(n_experts + 1, dtype=torch.int32, device=self.device)
            perm = torch.empty(M * k, dtype=torch.int32, device=self.device)
            inv = torch.empty(M * k, dtype=torch.int32, device=self.device)
        self._wait_torch()
        atsi.atsi_moe_bucket(self.ctx, idx.data_ptr(), M, k, n_experts, counts.data_ptr(), offsets.data_ptr(),
                             perm.data_ptr(), inv.data_ptr())
        self._torch_waits()
        return counts, offsets, perm, inv

    def stats(self, reset: bool = False) -> dict:
        """Transfer counters: h2d_bytes, h2d_copies, h2d_tensors, host_reads (see atsi_get_stats)."""
        return atsi.atsi_get_stats(self.ctx, reset)

    def set_schedule(self, order) -> None:
        atsi.atsi_set_schedule(self.ctx, list(order))

    def unpack(self, tid: int) -> torch.Tensor:
        K, N = self.shapes[tid]
        with torch.cuda.stream(self.cs):
            q = torch.empty((N, K), dtype=torch.int8, device=self.device)
        self._wait_torch()
        atsi.atsi_debug_unpack(self.ctx, tid, q.data_ptr())
        self._torch_waits()
        return q

    def _wait_torch(self) -> None:
        # work torch queued on its current stream (uploads, allocations) precedes ours
        self.cs.wait_stream(torch.cuda.current_stream(self.device))

    def _torch_waits(self) -> None:
        # results are safe to consume on torch's current stream
        torch.cuda.current_stream(self.device).wait_stream(self.cs)

    def sync(self) -> None:
        atsi.atsi_sync(self.ctx)

    def close(self) -> None:
        if self.ctx:
            atsi.atsi_destroy(self.ctx)
            self.ctx = 0
        if self.pool:
            atsi.atsi_cpu_pool_destroy(self.pool)
            self.pool = 0

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


class MoELayer:
    """Keeps an atsi_moe descriptor (and what it points at) alive."""

    def __init__(self, sess: Session, router_w: torch.Tensor, gate, up, down, top_k: int,
                 router_bias: torch.Tensor | None = None):
        import ctypes
        E = len(gate)
        H, I = sess.shapes[gate[0]]
        assert router_w.dtype == torch.float16 and tuple(router_w.shape) == (H, E)
        self.sess = sess
        self.E, self.H, self.I, self.k = E, H, I, top_k
        self._ids = [(ctypes.c_int32 * E)(*[int(t) for t in ids]) for ids in (gate, up, down)]
        self._keep = [router_w, router_bias]
        self.desc = atsi.atsi_moe(E, top_k, H, I, router_w.data_ptr(),
                                  router_bias.data_ptr() if router_bias is not None else None,
                                  ctypes.cast(self._ids[0], ctypes.POINTER(ctypes.c_int32)),
                                  ctypes.cast(self._ids[1], ctypes.POINTER(ctypes.c_int32)),
                                  ctypes.cast(self._ids[2], ctypes.POINTER(ctypes.c_int32)))

    def __call__(self, x: torch.Tensor, y: torch.Tensor | None = None, debug: bool = False):
        s = self.sess
        M = x.shape[0]
        dbg = None
        out = {}
        with torch.cuda.stream(s.cs):
            if y is None:
                y = torch.empty((M, self.H), dtype=torch.float16, device=s.device)
        if debug:
            out, dbg = self._debug_buffers(M)
        s._wait_torch()
        atsi.atsi_moe_ffn(s.ctx, self.desc, x.data_ptr(), M, y.data_ptr(), dbg)
        s._torch_waits()
        return (y, out) if debug else y

    def _debug_buffers(self, M: int):
        s = self.sess
        with torch.cuda.stream(s.cs):
            out = {"logits": torch.empty((M, self.E), dtype=torch.float32, device=s.device),
                   "idx": torch.empty((M, self.k), dtype=torch.int32, device=s.device),
                   "p": torch.empty((M, self.k), dtype=torch.float32, device=s.device),
                   "counts": torch.empty(self.E, dtype=torch.int32, device=s.device),
                   "offsets": torch.empty(self.E + 1, dtype=torch.int32, device=s.device),
                   "perm": torch.empty(M * self.k, dtype=torch.int32, device=s.device),
                   "inv_perm": torch.empty(M * self.k, dtype=torch.int32, device=s.device),
                   "expert_h": torch.empty((M * self.k, self.I), dtype=torch.float16, device=s.device),
                   "expert_out": torch.empty((M * self.k, self.H), dtype=torch.float16, device=s.device)}
        dbg = atsi.atsi_moe_debug(*[out[n].data_ptr() for n in atsi.MOE_DEBUG_FIELDS])
        return out, dbg


class MoEDecoderLayer:
    """Attention (q, k, v, o tensor ids) plus an MoELayer as the FFN."""

    def __init__(self, moe: MoELayer, q: int, k: int, v: int, o: int, n_heads: int, n_kv: int, head_dim: int,
                 eps: float = 1e-6):
        self.moe = moe
        self.n_heads, self.head_dim = n_heads, head_dim
        self.desc = atsi.atsi_moe_layer(n_heads, n_kv, head_dim, eps, q, k, v, o,
                                        __import__("ctypes").pointer(moe.desc))

    def __call__(self, h: torch.Tensor, q_out: torch.Tensor | None = None, k_out: torch.Tensor | None = None,
                 debug: bool = False):
        """Updates h (fp16 [M][hidden]) in place; returns the routing buffers and
        the intermediate activations (attn, h_attn, expert_h, expert_out) when debug."""
        s = self.moe.sess
        M, H = h.shape
        out, dbg, ldbg = {}, None, None
        if debug:
            out, dbg = self.moe._debug_buffers(M)
            lo, ldbg = s._layer_debug(M, H, self.n_heads * self.head_dim, 0, False)
            out.update(lo)
        s._wait_torch()
        atsi.atsi_moe_decoder_layer(s.ctx, self.desc, h.data_ptr(), M, q_out.data_ptr() if q_out is not None else 0,
                                    k_out.data_ptr() if k_out is not None else 0, dbg, ldbg)
        s._torch_waits()
        return out if debug else None
