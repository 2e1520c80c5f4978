"""The library's host-CPU backend (atsi_cpu_linear, the CPU side of the hybrid
execution of Sec. 4.3-4.4) against the oracle, CPU only: the product needs no
GPU.  Its arithmetic is fp32 sums of exact products, so it meets the same
tight gate as the GPU's GEMV (K 2^-24 for the sums plus the fp16 output
rounding); the fp16 conversions it uses are checked exhaustively against
numpy's IEEE conversions."""
import ctypes

import numpy as np
import pytest

import oracle
import synth
from paper_2607_10183_amd import atsi
from tests import parity


@pytest.fixture(scope="module")
def pools():
    made = {}

    def get(threads):
        if threads not in made:
            made[threads] = atsi.atsi_cpu_pool_create(threads)
        return made[threads]
    yield get
    for p in made.values():
        atsi.atsi_cpu_pool_destroy(p)


def _run(pool, codes, scales, x):
    M, K = x.shape
    N = codes.shape[0]
    codes = np.ascontiguousarray(codes, np.uint8)
    sc = np.ascontiguousarray(scales, np.float16).view(np.uint16)
    xs = np.ascontiguousarray(x, np.float16).view(np.uint16)
    y = np.zeros((M, N), np.uint16)
    atsi.atsi_cpu_linear(pool, codes.ctypes.data, sc.ctypes.data, N, K, xs.ctypes.data, M, y.ctypes.data)
    return y.view(np.float16)


@pytest.mark.parametrize("M,K,N,threads", [(1, 32, 1, 1), (1, 4096, 1031, 8), (3, 640, 77, 3), (4, 1024, 256, 5),
                                           (7, 2048, 130, 8), (16, 4096, 64, 16), (5, 96, 9, 12)])
def test_matches_oracle(pools, M, K, N, threads):
    seed, uid = 11, 1000 + K + N
    codes = synth.int4_codes(seed, uid, N, K)
    scales = synth.group_scales(seed, uid, N, K)
    x = synth.activations(seed, uid + 1, M, K)
    y = _run(pools(threads), codes, scales, x)
    ref, zeta = oracle.linear(x.astype(np.float64), codes, scales)
    parity.check(y, ref, zeta, f"cpu linear {M}x{K}x{N}", tight=parity.tight_eps(K))


def test_thread_count_does_not_change_bits(pools):
    K, N, M = 1024, 203, 6
    codes = synth.int4_codes(5, 77, N, K)
    scales = synth.group_scales(5, 77, N, K)
    x = synth.activations(5, 78, M, K)
    ys = [_run(pools(t), codes, scales, x).view(np.uint16) for t in (1, 2, 7, 16)]
    for y in ys[1:]:
        assert np.array_equal(y, ys[0])


def test_exact_inputs_are_exact(pools):
    """Power-of-two scales and +-1 inputs: every partial sum is a small
    integer multiple of the scale, so the result is the exact value."""
    K, N, M = 512, 40, 3
    codes = synth.int4_codes(3, 9, N, K)
    scales = synth.exact_scales(N, K)
    x = synth.sign_activations(3, 10, M, K)
    y = _run(pools(4), codes, scales, x)
    ref, _ = oracle.linear(x.astype(np.float64), codes, scales)
    assert np.array_equal(y.astype(np.float64), ref.astype(np.float16).astype(np.float64))


def test_plain_loop_matches_oracle():
    """The loop CPUs without AVX2/FMA/F16C take (forced by ATSI_CPU_PLAIN=1 in
    a child process, since the choice is made once per process)."""
    import os
    import subprocess
    import sys
    code = ("import numpy as np, oracle, synth; from tests import parity; from tests.test_cpu_backend import _run; "
            "from paper_2607_10183_amd import atsi; p = atsi.atsi_cpu_pool_create(3); "
            "c = synth.int4_codes(2, 5, 37, 640); s = synth.group_scales(2, 5, 37, 640); "
            "x = synth.activations(2, 6, 5, 640); y = _run(p, c, s, x); r, z = oracle.linear(x.astype(np.float64), c, s); "
            "parity.check(y, r, z, 'plain', tight=parity.tight_eps(640)); print('ok')")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, "-c", code], cwd=root, env=dict(os.environ, ATSI_CPU_PLAIN="1"),
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stderr[-2000:]


def test_every_half_converts_exactly():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    vals = bits.view(np.float16).astype(np.float32)
    finite = np.isfinite(vals)
    out, back = atsi.atsi_debug_cpu_f16(list(vals[finite]))
    assert np.array_equal(np.array(out, np.uint16), bits[finite])
    assert np.array_equal(np.array(back, np.float32), vals[finite])


def test_rounding_matches_ieee():
    rng = np.random.default_rng(4)
    f = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * np.float32(2.0) ** rng.integers(-30, 17, 20000),
        np.array([65504.0, 65519.996, 65520.0, 65536.0, 1e9, -65520.0, 2.0 ** -24, 2.0 ** -25, 1.5 * 2.0 ** -25,
                  2.0 ** -14, 2.0 ** -14 - 2.0 ** -25, 0.0, -0.0, 1.0 + 2.0 ** -11, 1.0 + 3 * 2.0 ** -11,
                  np.inf, -np.inf], np.float32)])
    out, _ = atsi.atsi_debug_cpu_f16(list(f))
    with np.errstate(over="ignore"):
        ref = f.astype(np.float16).view(np.uint16)
    assert np.array_equal(np.array(out, np.uint16), ref)


def test_rejects_bad_arguments(pools):
    lib = atsi.lib()
    buf = (ctypes.c_uint8 * 64)()
    p = ctypes.cast(buf, ctypes.c_void_p)
    assert lib.atsi_cpu_linear(pools(1), p, p, 1, 33, p, 1, p) == 2
    assert lib.atsi_cpu_linear(pools(1), p, p, 0, 32, p, 1, p) == 2
    assert lib.atsi_cpu_linear(pools(1), p, p, 1, 32, p, 0, p) == 2
    assert lib.atsi_cpu_linear(None, p, p, 1, 32, p, 1, p) == 1
    assert lib.atsi_cpu_linear(pools(1), None, p, 1, 32, p, 1, p) == 1
    out = ctypes.c_void_p()
    assert lib.atsi_cpu_pool_create(0, ctypes.byref(out)) == 1
