"""The acceptance checks of the GPU tests, checked on the CPU: a correctly
rounded result passes; one 32-input group dropped from one output of one
token is rejected; an error confined to one token's row is caught by the
per-row norm even where the norm of the whole batch would let it pass."""
import numpy as np
import pytest

import oracle
import synth
from tests.parity import check, tight_eps


def _case(M=512, N=64, K=4096):
    codes = synth.int4_codes(5, 1, N, K)
    scales = synth.group_scales(5, 1, N, K)
    x = synth.activations(5, 2, M, K)
    y, zeta = oracle.linear(x, codes, scales)
    return codes, scales, x, y, zeta


def test_rounded_result_passes():
    _, _, _, y, zeta = _case()
    check(y.astype(np.float16), y, zeta, name="rounded", tight=tight_eps(4096))


def test_dropped_group_is_rejected():
    codes, scales, x, y, zeta = _case()
    q = oracle.unpack_codes(codes).astype(np.float64)
    s = scales.astype(np.float64)
    bound = tight_eps(4096) * zeta
    rng = np.random.default_rng(0)
    caught = tested = 0
    for _ in range(40):
        m, n, g = int(rng.integers(512)), int(rng.integers(64)), int(rng.integers(128))
        contrib = s[n, g] * (q[n, 32 * g:32 * g + 32] @ x[m, 32 * g:32 * g + 32].astype(np.float64))
        bad = y.copy()
        bad[m, n] -= contrib
        bad = bad.astype(np.float16)
        tested += 1
        try:
            check(bad, y, zeta, name="dropped group", tight=tight_eps(4096))
        except AssertionError:
            caught += 1
        else:
            # passing is only allowed where the group's sum is within the bound
            assert abs(contrib) <= bound[m, n] + 2.0 ** -10 * abs(y[m, n]), (m, n, g, contrib, bound[m, n])
    assert caught >= 0.6 * tested, (caught, tested)


def test_row_norm_catches_an_error_confined_to_one_row():
    _, _, _, y, zeta = _case()
    bad = y.copy()
    bad[17] *= 1.003  # one token off by 0.3 %: the batch norm moves by about 1.3e-4
    glob = np.linalg.norm(bad - y) / np.linalg.norm(y)
    assert glob < 1e-3
    with pytest.raises(AssertionError, match="row 17 relative L2"):
        check(bad, y, zeta * 1e6, name="one row", tight=1.0)
