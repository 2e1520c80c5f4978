"""Acceptance checks shared by the GPU parity tests.

required gate : |y - y_ref| <= 1e-2 * zeta elementwise, zeta = |W| . |x| for one
                  linear layer (x the stage's own input) and its propagated form
                  for composite stages.
tight gate      : the same with a smaller factor.  For one linear it follows the
                  arithmetic of the kernel that ran (tight_eps): fp32 accumulation
                  over K inputs (K 2^-24), the fp16 output rounding (2^-11) and,
                  on the MFMA prefill path, the fp16 rounding of each dequantised
                  weight (another 2^-11).  Composite stages default to 2.5e-3.
row rel-L2 gate : ||y_r - y_ref_r|| / ||y_ref_r|| <= 1e-3 for every row r (token)
                  separately (fp16 output rounding alone is about 2.8e-4), so an
                  error confined to one token's row cannot hide in the norm of
                  the whole batch.
"""
import numpy as np

REQUIRED = 1e-2
TIGHT = 2.5e-3
REL_L2 = 1e-3


def tight_eps(K, mfma=False, norm=False):
    """Tight factor for one quantised linear over K inputs: exact products with
    fp32 accumulation (GEMV, batched decode), plus the fp16 rounding of the
    dequantised weights on the MFMA GEMM, plus a few fp32 ulps of a folded
    RMS-norm factor."""
    return K * 2.0 ** -24 + 2.0 ** -11 * (2 if mfma else 1) + (2.0 ** -20 if norm else 0.0)


def as_np(t):
    return t.detach().cpu().numpy() if hasattr(t, "detach") else np.asarray(t)


def check(y, y_ref, zeta, name="", tight=TIGHT, rel_l2=REL_L2):
    y = as_np(y).astype(np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    zeta = np.broadcast_to(np.asarray(zeta, dtype=np.float64), y_ref.shape)
    assert y.shape == y_ref.shape, f"{name}: shape {y.shape} != {y_ref.shape}"
    err = np.abs(y - y_ref)
    assert np.all(np.isfinite(y)), f"{name}: non-finite output"
    worst = float(np.max(err / np.maximum(zeta, 1e-30))) if err.size else 0.0
    assert np.all(err <= REQUIRED * zeta), f"{name}: required 1e-2 bound violated (max err/zeta {worst:.3e})"
    assert np.all(err <= tight * zeta), f"{name}: tight bound violated (max err/zeta {worst:.3e} > {tight:.3e})"
    rows_y = (y - y_ref).reshape(-1, y_ref.shape[-1]) if y_ref.ndim else (y - y_ref).reshape(1, 1)
    rows_r = y_ref.reshape(rows_y.shape)
    num = np.linalg.norm(rows_y, axis=1)
    den = np.maximum(np.linalg.norm(rows_r, axis=1), 1e-30)
    rl2 = float(np.max(num / den)) if num.size else 0.0
    bad = int(np.argmax(num / den)) if num.size else 0
    assert rl2 <= rel_l2, f"{name}: row {bad} relative L2 {rl2:.3e}"
    return worst, rl2


def bits16(a):
    return np.ascontiguousarray(as_np(a)).astype(np.float16).view(np.uint16)


def ulp16(v):
    """Spacing of fp16 at |v| (the subnormal spacing 2^-24 near zero)."""
    a = np.abs(np.asarray(v, dtype=np.float64))
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -14)))
    return 2.0 ** (e - 10)


def assert_within_one_ulp16(y, exact, name=""):
    """Each fp16 output is the nearest-even rounding of the exact value or one
    of its fp16 neighbours (the kernel's last fp32 step, e.g. SiLU, may move
    the value by a few fp32 ulps before the rounding)."""
    y = as_np(y).astype(np.float64)
    r = np.asarray(exact, dtype=np.float64).astype(np.float16).astype(np.float64)
    d = np.abs(y - r)
    ok = d <= ulp16(r) * 1.0000001
    assert np.all(ok), f"{name}: {int((~ok).sum())} outputs more than one fp16 ulp from the rounded exact value"
