"""Pins of the plain-C fp64 linear oracle (oracle/c/q4_linear.c), the CPU
baseline's kernel, on the CPU: the hand-worked fixture, exact rational
brute force, an exhaustive check of its fp16 scale decoding, and thread-count
invariance.  None of these re-type its loops."""
import json
import os
from fractions import Fraction

import numpy as np

import synth
from oracle import c_linear

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_linear_tiny_golden():
    with open(os.path.join(GOLD, "linear_tiny.json")) as f:
        g = json.load(f)
    codes = np.array([[b] * (g["K"] // 2) for b in g["row_bytes"]], np.uint8)
    scales = np.array([[s] * (g["K"] // 32) for s in g["scales"]], np.float16)
    x = np.stack([np.ones(g["K"]), np.arange(g["K"]) / 8.0])  # the fixture's "row0 all ones; row1 k/8"
    y = c_linear.linear(x, codes, scales)
    assert np.array_equal(y, np.array(g["y"], np.float64))


def test_exact_rational_brute_force():
    for K, N, M in ((32, 3, 2), (64, 5, 3), (96, 4, 1)):
        codes = synth.int4_codes(31, K, N, K)
        scales = synth.group_scales(31, K, N, K)
        x = synth.activations(31, K + 1, M, K)
        y = c_linear.linear(x, codes, scales)
        for m in range(M):
            for n in range(N):
                acc = Fraction(0)
                for k in range(K):
                    byte = int(codes[n, k // 2])
                    q = ((byte >> (4 * (k % 2))) & 15) - 8
                    acc += Fraction(float(x[m, k])) * Fraction(float(scales[n, k // 32])) * q
                # fp64 accumulation of K exact products: relative error below K 2^-53 of sum |terms|
                bound = sum(abs(Fraction(float(x[m, k]))) for k in range(K)) * Fraction(8 * 0.02) * K * Fraction(2) ** -52
                assert abs(Fraction(float(y[m, n])) - acc) <= bound


def test_every_finite_fp16_scale_decodes_exactly():
    """Row n has scale bits n (all 63488 finite fp16 patterns) and one code q = 1
    at input 0, so y[0][n] is the scale itself; numpy's float16 is the reference."""
    bits = np.arange(65536, dtype=np.uint16)
    finite = bits[np.isfinite(bits.view(np.float16))]
    N = finite.size
    codes = np.full((N, 16), 0x88, np.uint8)
    codes[:, 0] = 0x89  # input 0: u = 9, q = 1; input 1: q = 0
    scales = finite.view(np.float16).reshape(N, 1)
    x = np.zeros((1, 32))
    x[0, 0] = 1.0
    y = c_linear.linear(x, codes, scales, threads=4)[0]
    assert np.array_equal(y, finite.view(np.float16).astype(np.float64))


def test_thread_count_invariance():
    codes = synth.int4_codes(32, 1, 77, 512)
    scales = synth.group_scales(32, 1, 77, 512)
    x = synth.activations(32, 2, 3, 512)
    y1 = c_linear.linear(x, codes, scales, threads=1)
    for t in (2, 7, 200):
        assert np.array_equal(c_linear.linear(x, codes, scales, threads=t), y1)
