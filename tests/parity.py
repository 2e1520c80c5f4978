"""Acceptance checks shared by the GPU parity tests.

spec gate : |y - y_ref| <= 1e-2 * zeta elementwise, zeta = |W| . |x| for one
                  linear layer and its propagated form for composite stages.
tight gate      : the same with 2.5e-3, which covers fp32 accumulation over
                  K <= 14336 (K * 2^-24 <= 8.6e-4), the fp16 output rounding
                  (2^-11) and the fp16 rounding of dequantised weights on the
                  MFMA path (2^-11).
rel-L2 gate     : ||y - y_ref|| / ||y_ref|| <= 1e-3 (fp16 output rounding alone is
                  about 2.8e-4); catches errors concentrated in a few outputs.
"""
import numpy as np

NORTH_STAR = 1e-2
TIGHT = 2.5e-3
REL_L2 = 1e-3


def as_np(t):
    return t.detach().cpu().numpy() if hasattr(t, "detach") else np.asarray(t)


def check(y, y_ref, zeta, name="", tight=TIGHT, rel_l2=REL_L2):
    y = as_np(y).astype(np.float64)
    err = np.abs(y - y_ref)
    assert np.all(np.isfinite(y)), f"{name}: non-finite output"
    worst = float(np.max(err / np.maximum(zeta, 1e-30)))
    assert np.all(err <= NORTH_STAR * zeta), f"{name}: north-star bound violated (max err/zeta {worst:.3e})"
    assert np.all(err <= tight * zeta), f"{name}: tight bound violated (max err/zeta {worst:.3e})"
    rl2 = float(np.linalg.norm(y - y_ref) / max(np.linalg.norm(y_ref), 1e-30))
    assert rl2 <= rel_l2, f"{name}: relative L2 {rl2:.3e}"
    return worst, rl2


def bits16(a):
    return np.ascontiguousarray(as_np(a)).astype(np.float16).view(np.uint16)
