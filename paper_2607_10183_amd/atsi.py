"""Thin ctypes binding of libatsi.so: the C ABI in include/atsi.h, same names.

Argument marshalling only: every step of the hot path runs in the library's
HIP kernels.  Functions raise AtsiError when the library returns a non-OK
status.  Pointers are plain integers (torch: ``tensor.data_ptr()``; streams:
``torch.cuda.Stream().cuda_stream``).
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libatsi.so")

DEBUG_POISON = 1
DEBUG_SERIALIZE = 2

STATUS = {0: "ATSI_OK", 1: "ATSI_E_INVALID", 2: "ATSI_E_SHAPE", 3: "ATSI_E_UNKNOWN_TENSOR",
          4: "ATSI_E_NO_COPY", 5: "ATSI_E_WORKSPACE", 6: "ATSI_E_HIP", 7: "ATSI_E_STATE"}


class AtsiError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


class atsi_qtensor(ctypes.Structure):
    _fields_ = [("K", ctypes.c_int64), ("N", ctypes.c_int64), ("group", ctypes.c_int32),
                ("dev_codes", ctypes.c_void_p), ("dev_scales", ctypes.c_void_p),
                ("host_codes", ctypes.c_void_p), ("host_scales", ctypes.c_void_p)]


class atsi_dense_layer(ctypes.Structure):
    _fields_ = [("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("eps", ctypes.c_float), ("q", ctypes.c_int32), ("k", ctypes.c_int32), ("v", ctypes.c_int32),
                ("o", ctypes.c_int32), ("gate", ctypes.c_int32), ("up", ctypes.c_int32), ("down", ctypes.c_int32),
                ("renorm_out", ctypes.c_int32)]


class atsi_moe(ctypes.Structure):
    _fields_ = [("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32), ("hidden", ctypes.c_int64),
                ("inter", ctypes.c_int64), ("router_w_f16", ctypes.c_void_p), ("router_bias", ctypes.c_void_p),
                ("gate", ctypes.POINTER(ctypes.c_int32)), ("up", ctypes.POINTER(ctypes.c_int32)),
                ("down", ctypes.POINTER(ctypes.c_int32))]


MOE_DEBUG_FIELDS = ("logits", "idx", "p", "counts", "offsets", "perm", "inv_perm", "expert_h", "expert_out")
LAYER_DEBUG_FIELDS = ("attn", "h_attn", "act", "sum32")


class atsi_moe_debug(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in MOE_DEBUG_FIELDS]


class atsi_layer_debug(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in LAYER_DEBUG_FIELDS]


class atsi_moe_layer(ctypes.Structure):
    _fields_ = [("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("eps", ctypes.c_float), ("q", ctypes.c_int32), ("k", ctypes.c_int32), ("v", ctypes.c_int32),
                ("o", ctypes.c_int32), ("moe", ctypes.POINTER(atsi_moe))]


class atsi_placement_problem(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("size_bytes", ctypes.c_void_p), ("r", ctypes.c_void_p),
                ("c", ctypes.c_void_p), ("is_expert", ctypes.c_void_p), ("budget_bytes", ctypes.c_double),
                ("granularity_bytes", ctypes.c_double)]


class atsi_transfer_problem(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("on_gpu", ctypes.c_void_p), ("t_gpu", ctypes.c_void_p),
                ("t_cpu", ctypes.c_void_p), ("c", ctypes.c_void_p), ("w", ctypes.c_void_p)]


TIMING_FIELDS = ("t_gpu", "t_cpu", "d2h", "h2d", "w")


class atsi_tensor_timing(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in TIMING_FIELDS]


_P = ctypes.c_void_p
class atsi_stats(ctypes.Structure):
    _fields_ = [("h2d_bytes", ctypes.c_uint64), ("h2d_copies", ctypes.c_uint64), ("h2d_tensors", ctypes.c_uint64),
                ("host_reads", ctypes.c_uint64), ("host_read_bytes", ctypes.c_uint64)]


_SIGS = {
    "atsi_create": ([ctypes.c_int, _P, _P, _P, _P, ctypes.c_size_t, _P, ctypes.c_int, ctypes.POINTER(_P)],
                    ctypes.c_int),
    "atsi_destroy": ([_P], ctypes.c_int),
    "atsi_last_error": ([_P], ctypes.c_char_p),
    "atsi_tensor_register": ([_P, ctypes.POINTER(atsi_qtensor), ctypes.POINTER(ctypes.c_int32)], ctypes.c_int),
    "atsi_set_placement": ([_P, _P, ctypes.c_int32], ctypes.c_int),
    "atsi_linear": ([_P, ctypes.c_int32, _P, ctypes.c_int64, _P], ctypes.c_int),
    "atsi_ffn_swiglu": ([_P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _P, ctypes.c_int64, _P], ctypes.c_int),
    "atsi_ffn_swiglu_noalloc": ([_P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _P, ctypes.c_int64, _P],
                                ctypes.c_int),
    "atsi_swiglu_gate_up": ([_P, ctypes.c_int32, ctypes.c_int32, _P, ctypes.c_int64, _P], ctypes.c_int),
    "atsi_rmsnorm": ([_P, _P, ctypes.c_int64, ctypes.c_int64, ctypes.c_float, _P], ctypes.c_int),
    "atsi_decoder_layer": ([_P, ctypes.POINTER(atsi_dense_layer), _P, ctypes.c_int64, _P, _P,
                            ctypes.POINTER(atsi_layer_debug)], ctypes.c_int),
    "atsi_moe_ffn": ([_P, ctypes.POINTER(atsi_moe), _P, ctypes.c_int64, _P, ctypes.POINTER(atsi_moe_debug)],
                     ctypes.c_int),
    "atsi_moe_decoder_layer": ([_P, ctypes.POINTER(atsi_moe_layer), _P, ctypes.c_int64, _P, _P,
                                ctypes.POINTER(atsi_moe_debug), ctypes.POINTER(atsi_layer_debug)], ctypes.c_int),
    "atsi_moe_bucket": ([_P, _P, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, _P, _P, _P, _P], ctypes.c_int),
    "atsi_set_schedule": ([_P, _P, ctypes.c_int32], ctypes.c_int),
    "atsi_prefetch": ([_P, ctypes.c_int32], ctypes.c_int),
    "atsi_sync": ([_P], ctypes.c_int),
    "atsi_get_stats": ([_P, ctypes.POINTER(atsi_stats), ctypes.c_int32], ctypes.c_int),
    "atsi_debug_unpack": ([_P, ctypes.c_int32, _P], ctypes.c_int),
    "atsi_set_debug": ([_P, ctypes.c_uint32], ctypes.c_int),
    "atsi_set_zero_copy": ([_P, ctypes.c_int32], ctypes.c_int),
    "atsi_set_moe_light_rows": ([_P, ctypes.c_int32], ctypes.c_int),
    "atsi_solve_placement": ([ctypes.POINTER(atsi_placement_problem), _P, ctypes.POINTER(ctypes.c_double)],
                             ctypes.c_int),
    "atsi_schedule_transfers": ([ctypes.POINTER(atsi_transfer_problem), _P, ctypes.POINTER(ctypes.c_double)],
                                ctypes.c_int),
    "atsi_transfer_latency": ([ctypes.POINTER(atsi_transfer_problem), _P, ctypes.POINTER(ctypes.c_double)],
                              ctypes.c_int),
    "atsi_rescheduler_create": ([ctypes.c_int32, ctypes.c_double, ctypes.c_double, ctypes.POINTER(_P)],
                                ctypes.c_int),
    "atsi_rescheduler_step": ([_P, ctypes.POINTER(atsi_transfer_problem), ctypes.c_double, ctypes.c_double, _P,
                               ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_double)], ctypes.c_int),
    "atsi_rescheduler_destroy": ([_P], ctypes.c_int),
    "atsi_cpu_pool_create": ([ctypes.c_int32, ctypes.POINTER(_P)], ctypes.c_int),
    "atsi_cpu_pool_destroy": ([_P], ctypes.c_int),
    "atsi_cpu_linear": ([_P, _P, _P, ctypes.c_int64, ctypes.c_int64, _P, ctypes.c_int64, _P], ctypes.c_int),
    "atsi_set_cpu_backend": ([_P, _P, _P, ctypes.c_size_t], ctypes.c_int),
    "atsi_set_backends": ([_P, _P, ctypes.c_int32], ctypes.c_int),
    "atsi_set_timing": ([_P, ctypes.c_int32], ctypes.c_int),
    "atsi_get_timings": ([_P, ctypes.c_int32, ctypes.POINTER(atsi_tensor_timing)], ctypes.c_int),
    "atsi_debug_cpu_f16": ([_P, ctypes.c_int64, _P, _P], ctypes.c_int),
    "atsi_debug_read_probe": ([_P, _P, ctypes.c_size_t], ctypes.c_int),
}

_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises ImportError (never falls back) when it is not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built: run `python -m paper_2607_10183_amd.build` "
                              "(there is no CPU fallback)")
        l = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            f = getattr(l, name)
            f.argtypes = args
            f.restype = res
        _lib = l
    return _lib


def _check(ctx, status: int) -> None:
    if status != 0:
        msg = lib().atsi_last_error(ctx)
        raise AtsiError(status, msg.decode() if msg else "")


def atsi_create(device: int, compute_stream: int, transfer_stream: int, transfer_stream2: int, workspace: int,
                workspace_bytes: int, host_counts: int, n_slots: int) -> int:
    out = _P()
    _check(None, lib().atsi_create(device, compute_stream, transfer_stream, transfer_stream2 or None, workspace,
                                   workspace_bytes, host_counts or None, n_slots, ctypes.byref(out)))
    return out.value


def atsi_destroy(ctx: int) -> None:
    _check(ctx, lib().atsi_destroy(ctx))


def atsi_last_error(ctx: int | None) -> str:
    m = lib().atsi_last_error(ctx)
    return m.decode() if m else ""


def atsi_tensor_register(ctx: int, K: int, N: int, dev_codes: int = 0, dev_scales: int = 0,
                         host_codes: int = 0, host_scales: int = 0, group: int = 32) -> int:
    d = atsi_qtensor(K, N, group, dev_codes or None, dev_scales or None, host_codes or None, host_scales or None)
    out = ctypes.c_int32()
    _check(ctx, lib().atsi_tensor_register(ctx, ctypes.byref(d), ctypes.byref(out)))
    return out.value


def atsi_set_placement(ctx: int, host_mask) -> None:
    arr = (ctypes.c_uint8 * len(host_mask))(*[int(v) for v in host_mask])
    _check(ctx, lib().atsi_set_placement(ctx, ctypes.cast(arr, _P), len(host_mask)))


def atsi_linear(ctx: int, w: int, x: int, M: int, y: int) -> None:
    _check(ctx, lib().atsi_linear(ctx, w, x, M, y))


def atsi_ffn_swiglu(ctx: int, gate: int, up: int, down: int, x: int, M: int, y: int) -> None:
    _check(ctx, lib().atsi_ffn_swiglu(ctx, gate, up, down, x, M, y))


def atsi_ffn_swiglu_noalloc(ctx: int, gate: int, up: int, down: int, x: int, M: int, y: int) -> None:
    _check(ctx, lib().atsi_ffn_swiglu_noalloc(ctx, gate, up, down, x, M, y))


def atsi_rmsnorm(ctx: int, x: int, M: int, H: int, eps: float, y: int) -> None:
    _check(ctx, lib().atsi_rmsnorm(ctx, x, M, H, eps, y))


def atsi_swiglu_gate_up(ctx: int, gate: int, up: int, x: int, M: int, h: int) -> None:
    _check(ctx, lib().atsi_swiglu_gate_up(ctx, gate, up, x, M, h))


def _ref(d):
    return ctypes.byref(d) if d is not None else None


def atsi_decoder_layer(ctx: int, layer: atsi_dense_layer, h: int, M: int, q_out: int = 0, k_out: int = 0,
                       dbg: atsi_layer_debug | None = None) -> None:
    _check(ctx, lib().atsi_decoder_layer(ctx, ctypes.byref(layer), h, M, q_out or None, k_out or None, _ref(dbg)))


def atsi_moe_ffn(ctx: int, moe: atsi_moe, x: int, M: int, y: int, dbg: atsi_moe_debug | None = None) -> None:
    _check(ctx, lib().atsi_moe_ffn(ctx, ctypes.byref(moe), x, M, y, ctypes.byref(dbg) if dbg is not None else None))


def atsi_moe_decoder_layer(ctx: int, layer: atsi_moe_layer, h: int, M: int, q_out: int = 0, k_out: int = 0,
                           dbg: atsi_moe_debug | None = None, ldbg: atsi_layer_debug | None = None) -> None:
    _check(ctx, lib().atsi_moe_decoder_layer(ctx, ctypes.byref(layer), h, M, q_out or None, k_out or None,
                                              _ref(dbg), _ref(ldbg)))


def atsi_moe_bucket(ctx: int, idx: int, M: int, k: int, n_experts: int, counts: int, offsets: int, perm: int,
                    inv_perm: int) -> None:
    _check(ctx, lib().atsi_moe_bucket(ctx, idx, M, k, n_experts, counts, offsets, perm, inv_perm))


def atsi_set_schedule(ctx: int, order) -> None:
    arr = (ctypes.c_int32 * max(1, len(order)))(*[int(t) for t in order])
    _check(ctx, lib().atsi_set_schedule(ctx, ctypes.cast(arr, _P), len(order)))


def atsi_prefetch(ctx: int, w: int) -> None:
    _check(ctx, lib().atsi_prefetch(ctx, w))


def atsi_sync(ctx: int) -> None:
    _check(ctx, lib().atsi_sync(ctx))


def atsi_get_stats(ctx: int, reset: bool = False) -> dict:
    st = atsi_stats()
    _check(ctx, lib().atsi_get_stats(ctx, ctypes.byref(st), int(reset)))
    return {f: int(getattr(st, f)) for f, _ in atsi_stats._fields_}


def atsi_debug_unpack(ctx: int, w: int, q_out: int) -> None:
    _check(ctx, lib().atsi_debug_unpack(ctx, w, q_out))


def atsi_solve_placement(size_bytes, r, c, budget_bytes: float, granularity_bytes: float = float(1 << 20),
                         is_expert=None):
    """(on_gpu list of 0/1, objective) of the static placement (host computation)."""
    n = len(size_bytes)
    D = ctypes.c_double * n
    sa, ra, ca = D(*map(float, size_bytes)), D(*map(float, r)), D(*map(float, c))
    ea = (ctypes.c_uint8 * n)(*[int(v) for v in is_expert]) if is_expert is not None else None
    prob = atsi_placement_problem(n, ctypes.cast(sa, _P), ctypes.cast(ra, _P), ctypes.cast(ca, _P),
                                  ctypes.cast(ea, _P) if ea is not None else None, float(budget_bytes),
                                  float(granularity_bytes))
    out = (ctypes.c_uint8 * max(n, 1))()
    obj = ctypes.c_double()
    _check(None, lib().atsi_solve_placement(ctypes.byref(prob), ctypes.cast(out, _P), ctypes.byref(obj)))
    return [int(out[i]) for i in range(n)], obj.value


def atsi_set_debug(ctx: int, flags: int) -> None:
    _check(ctx, lib().atsi_set_debug(ctx, int(flags)))


def atsi_set_zero_copy(ctx: int, enable: bool) -> None:
    _check(ctx, lib().atsi_set_zero_copy(ctx, 1 if enable else 0))


def atsi_set_moe_light_rows(ctx: int, rows: int) -> None:
    _check(ctx, lib().atsi_set_moe_light_rows(ctx, int(rows)))


class _TransferArrays:
    """An atsi_transfer_problem and the arrays it points at (kept alive together)."""

    def __init__(self, on_gpu, t_gpu, t_cpu, c, w):
        n = len(on_gpu)
        if not (len(t_gpu) == len(t_cpu) == len(c) == len(w) == n):
            raise ValueError("the five series of a transfer problem must have one length")
        D = ctypes.c_double * max(n, 1)
        self.b = (ctypes.c_uint8 * max(n, 1))(*[int(v) for v in on_gpu])
        self.tg, self.tc = D(*map(float, t_gpu)), D(*map(float, t_cpu))
        self.c, self.w = D(*map(float, c)), D(*map(float, w))
        self.p = atsi_transfer_problem(n, ctypes.cast(self.b, _P), ctypes.cast(self.tg, _P),
                                       ctypes.cast(self.tc, _P), ctypes.cast(self.c, _P), ctypes.cast(self.w, _P))
        self.n = n


def atsi_schedule_transfers(on_gpu, t_gpu, t_cpu, c, w):
    """(rb list, 1 = GPU; T) of Alg. 2 (host computation)."""
    a = _TransferArrays(on_gpu, t_gpu, t_cpu, c, w)
    out = (ctypes.c_uint8 * max(a.n, 1))()
    T = ctypes.c_double()
    _check(None, lib().atsi_schedule_transfers(ctypes.byref(a.p), ctypes.cast(out, _P), ctypes.byref(T)))
    return [int(out[i]) for i in range(a.n)], T.value


def atsi_transfer_latency(on_gpu, t_gpu, t_cpu, c, w, rb) -> float:
    """T(rb) of Sec. 4.4.1 (inf for an unreachable rb)."""
    a = _TransferArrays(on_gpu, t_gpu, t_cpu, c, w)
    arr = (ctypes.c_uint8 * max(a.n, 1))(*[int(v) for v in rb])
    T = ctypes.c_double()
    _check(None, lib().atsi_transfer_latency(ctypes.byref(a.p), ctypes.cast(arr, _P), ctypes.byref(T)))
    return T.value


def atsi_rescheduler_create(n: int, eps: float, tau_tpot: float) -> int:
    out = _P()
    _check(None, lib().atsi_rescheduler_create(n, eps, tau_tpot, ctypes.byref(out)))
    return out.value


def atsi_rescheduler_step(r: int, on_gpu, t_gpu, t_cpu, c, w, now_s: float, tpot_s: float):
    """(rb list, rescheduled bool, deviation) of one Alg. 3 step."""
    a = _TransferArrays(on_gpu, t_gpu, t_cpu, c, w)
    out = (ctypes.c_uint8 * max(a.n, 1))()
    did = ctypes.c_int32()
    d = ctypes.c_double()
    _check(None, lib().atsi_rescheduler_step(r, ctypes.byref(a.p), float(now_s), float(tpot_s),
                                             ctypes.cast(out, _P), ctypes.byref(did), ctypes.byref(d)))
    return [int(out[i]) for i in range(a.n)], bool(did.value), d.value


def atsi_rescheduler_destroy(r: int) -> None:
    _check(None, lib().atsi_rescheduler_destroy(r))


def atsi_cpu_pool_create(threads: int) -> int:
    out = _P()
    _check(None, lib().atsi_cpu_pool_create(int(threads), ctypes.byref(out)))
    return out.value


def atsi_cpu_pool_destroy(pool: int) -> None:
    _check(None, lib().atsi_cpu_pool_destroy(pool))


def atsi_cpu_linear(pool: int, codes: int, scales: int, N: int, K: int, x: int, M: int, y: int) -> None:
    _check(None, lib().atsi_cpu_linear(pool, codes, scales, N, K, x, M, y))


def atsi_set_cpu_backend(ctx: int, pool: int, staging: int, staging_bytes: int) -> None:
    _check(ctx, lib().atsi_set_cpu_backend(ctx, pool or None, staging or None, staging_bytes))


def atsi_set_backends(ctx: int, on_cpu) -> None:
    arr = (ctypes.c_uint8 * max(1, len(on_cpu)))(*[int(v) for v in on_cpu])
    _check(ctx, lib().atsi_set_backends(ctx, ctypes.cast(arr, _P), len(on_cpu)))


def atsi_set_timing(ctx: int, enable: bool) -> None:
    _check(ctx, lib().atsi_set_timing(ctx, 1 if enable else 0))


def atsi_get_timings(ctx: int, n: int) -> list:
    """Per-tensor dicts of the latest measured times (seconds; NaN where none)."""
    arr = (atsi_tensor_timing * max(1, n))()
    _check(ctx, lib().atsi_get_timings(ctx, n, arr))
    return [{f: getattr(arr[i], f) for f in TIMING_FIELDS} for i in range(n)]


def atsi_debug_cpu_f16(values):
    """(fp16 bit patterns, their fp32 values) of the CPU backend's rounding."""
    n = len(values)
    src = (ctypes.c_float * max(1, n))(*map(float, values))
    out = (ctypes.c_uint16 * max(1, n))()
    back = (ctypes.c_float * max(1, n))()
    _check(None, lib().atsi_debug_cpu_f16(ctypes.cast(src, _P), n, ctypes.cast(out, _P), ctypes.cast(back, _P)))
    return [int(out[i]) for i in range(n)], [back[i] for i in range(n)]


def atsi_debug_read_probe(ctx: int, dev_ptr: int, nbytes: int) -> None:
    """One read-only streaming pass over device memory (HBM read ceiling)."""
    _check(ctx, lib().atsi_debug_read_probe(ctx, dev_ptr, nbytes))
