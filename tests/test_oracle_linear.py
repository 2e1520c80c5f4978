"""Pins of the oracle's format, dequantisation and linear layer (CPU only).

None of these re-type the oracle's formulas: they check it against hand-worked
values, exact rational arithmetic and invariants that the mathematics fixes.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _pack(q_even, q_odd):
    """Inverse of the packing reading: two signed codes -> one byte."""
    return (int(q_even) + 8) | ((int(q_odd) + 8) << 4)


def test_nibble_table_golden():
    rows = []
    with open(os.path.join(GOLD, "nibble_table.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                b, a, c = line.split()
                rows.append((int(b, 16), int(a), int(c)))
    codes = np.array([[r[0] for r in rows]], np.uint8)
    q = oracle.unpack_codes(codes)[0]
    for i, (_, a, c) in enumerate(rows):
        assert (q[2 * i], q[2 * i + 1]) == (a, c)


def test_unpack_exhaustive_pack_identity():
    codes = np.arange(256, dtype=np.uint8)[None, :]
    q = oracle.unpack_codes(codes)[0]
    assert q.min() == -8 and q.max() == 7
    for b in range(256):
        assert _pack(q[2 * b], q[2 * b + 1]) == b
    # and every pair of codes survives pack -> unpack
    pairs = [(a, c) for a in range(-8, 8) for c in range(-8, 8)]
    packed = np.array([[_pack(a, c) for a, c in pairs]], np.uint8)
    back = oracle.unpack_codes(packed)[0]
    assert [(int(back[2 * i]), int(back[2 * i + 1])) for i in range(len(pairs))] == pairs


def test_dequant_exact_and_round_trip():
    n, k = 8, 128
    codes = synth.int4_codes(7, 1, n, k)
    scales = synth.group_scales(7, 1, n, k)
    w = oracle.dequant(codes, scales)
    q = oracle.unpack_codes(codes)
    for r in range(n):
        for c in range(0, k, 5):
            exact = Fraction(float(scales[r, c // 32])) * int(q[r, c])
            assert Fraction(float(w[r, c])) == exact
    # requantising with the known scale returns the code exactly
    s = np.repeat(scales.astype(np.float64), 32, axis=1)
    q2 = np.clip(np.rint(w / s), -8, 7).astype(np.int8)
    assert np.array_equal(q2, q)
    # fp32 dequant is exact too (<= 15 significant bits)
    assert np.array_equal(w.astype(np.float32).astype(np.float64), w)


def test_linear_hand_worked_golden():
    g = json.load(open(os.path.join(GOLD, "linear_tiny.json")))
    K, N = g["K"], g["N"]
    codes = np.array([[b] * (K // 2) for b in g["row_bytes"]], np.uint8)
    scales = np.array([[s] for s in g["scales"]], np.float16)
    x = np.stack([np.ones(K), np.arange(K) / 8.0]).astype(np.float16)
    y, zeta = oracle.linear(x, codes, scales)
    assert np.array_equal(y, np.array(g["y"]))
    assert np.all(zeta >= np.abs(y))


@pytest.mark.parametrize("K,N,M", [(32, 5, 3), (64, 3, 2), (96, 4, 1)])
def test_linear_bruteforce_rational(K, N, M):
    codes = synth.int4_codes(11, K, N, K)
    scales = synth.group_scales(11, K, N, K)
    x = synth.activations(11, K, M, K)
    y, zeta = oracle.linear(x, codes, scales)
    for m in range(M):
        for n in range(N):
            acc = Fraction(0)
            mag = Fraction(0)
            for kk in range(K):
                byte = int(codes[n, kk // 2])
                u = (byte >> (4 * (kk % 2))) & 0xF
                wv = Fraction(float(scales[n, kk // 32])) * (u - 8)
                xv = Fraction(float(x[m, kk]))
                acc += wv * xv
                mag += abs(wv * xv)
            assert abs(Fraction(float(y[m, n])) - acc) <= Fraction(1, 10 ** 13) * mag
            assert abs(Fraction(float(zeta[m, n])) - mag) <= Fraction(1, 10 ** 13) * mag


def test_linear_invariants():
    K, N, M = 256, 24, 4
    codes = synth.int4_codes(3, 1, N, K)
    scales = synth.group_scales(3, 1, N, K)
    x1 = synth.activations(3, 2, M, K).astype(np.float64)
    x2 = synth.activations(3, 3, M, K).astype(np.float64)
    y1, z1 = oracle.linear(x1, codes, scales)
    y2, z2 = oracle.linear(x2, codes, scales)
    y12, _ = oracle.linear(x1 + x2, codes, scales)
    assert np.all(np.abs(y12 - (y1 + y2)) <= 1e-13 * (z1 + z2))
    y2x, _ = oracle.linear(2.0 * x1, codes, scales)
    assert np.array_equal(y2x, 2.0 * y1)
    # permuting whole groups of 32 inputs (codes, scales and x together)
    gperm = synth.permutation(3, 4, K // 32)
    kperm = (gperm[:, None] * 32 + np.arange(32)[None, :]).reshape(-1)
    q = oracle.unpack_codes(codes)[:, kperm]
    u = (q + 8).astype(np.uint8)
    codes_p = (u[:, 0::2] | (u[:, 1::2] << 4)).astype(np.uint8)
    yp, _ = oracle.linear(x1[:, kperm], codes_p, scales[:, gperm])
    assert np.all(np.abs(yp - y1) <= 1e-13 * z1)
    # permuting inputs inside one group (the scale is shared)
    inner = np.arange(K)
    inner[:32] = synth.permutation(3, 5, 32)
    q2 = oracle.unpack_codes(codes)[:, inner]
    u2 = (q2 + 8).astype(np.uint8)
    yi, _ = oracle.linear(x1[:, inner], (u2[:, 0::2] | (u2[:, 1::2] << 4)).astype(np.uint8), scales)
    assert np.all(np.abs(yi - y1) <= 1e-13 * z1)
    # permuting output rows / token rows permutes y
    nperm = synth.permutation(3, 6, N)
    yn, _ = oracle.linear(x1, codes[nperm], scales[nperm])
    assert np.all(np.abs(yn - y1[:, nperm]) <= 1e-13 * z1[:, nperm])
    mperm = synth.permutation(3, 7, M)
    ym, _ = oracle.linear(x1[mperm], codes, scales)
    assert np.all(np.abs(ym - y1[mperm]) <= 1e-13 * z1[mperm])


def test_linear_exact_arithmetic_case_is_exact():
    """On the exact-arithmetic inputs the oracle's fp64 result is the exact value."""
    K, N, M = 4096, 6, 2
    codes = synth.int4_codes(5, 1, N, K)
    scales = synth.exact_scales(N, K)
    x = synth.exact_activations(5, 2, M, K)
    y, _ = oracle.linear(x, codes, scales)
    q = oracle.unpack_codes(codes).astype(np.int64)
    xi = np.rint(x.astype(np.float64) * 4).astype(np.int64)  # x = xi / 4
    exact = (xi @ q.T).astype(np.float64) * 2.0 ** -8          # s = 2^-6
    assert np.array_equal(y, exact)
