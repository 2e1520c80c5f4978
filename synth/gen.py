"""Counter-based generator for every synthetic input.

The generator is SplitMix64 (Steele, Lea and Flood, "Fast splittable
pseudorandom number generators", OOPSLA 2014): output i of a stream with key
``k`` is ``mix64(k + (i + 1) * GOLDEN)`` where ``mix64`` is the published
variant-13 finaliser.  Because output i depends only on (key, i), any slice of
any tensor can be regenerated independently, which lets tests sample rows of
full-size workloads without materialising them.

Streams are keyed by (seed, uid, kind): ``seed`` names the workload, ``uid``
the tensor inside it and ``kind`` the role of the numbers (codes, scales, ...).

Distributions (the recipe of every workload):
  * int4 codes: each packed byte is a raw generator byte, so both nibbles are
    uniform over 0..15, i.e. the signed code q = u - 8 is uniform in [-8, 7];
  * group scales: a 16-bit integer k picks s = fp16(0.005 + 0.015 * k / 65536),
    a value in [0.005, 0.02] rounded to nearest-even in fp16;
  * activations: N(0, 1) by Box-Muller in fp64, rounded to fp16;
  * router weights: N(0, 1/H) in fp64, rounded to fp16, so x . W_r ~ N(0, 1);
  * exact-arithmetic inputs: scales 2**-6 and activations in {-4..4} / 4, on
    which every fp32 partial sum of the linear layer is exact.
"""
from __future__ import annotations

import numpy as np

MASK64 = (1 << 64) - 1
GOLDEN = 0x9E3779B97F4A7C15
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

# stream kinds
KIND_CODES = 1
KIND_SCALES = 2
KIND_ACT = 3
KIND_ROUTER = 4
KIND_PERM = 5
KIND_SCORE = 6
KIND_MISC = 7


def _mix64_int(z: int) -> int:
    z &= MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def _mix64(z: np.ndarray) -> np.ndarray:
    z = z ^ (z >> np.uint64(30))
    z = z * _M1
    z = z ^ (z >> np.uint64(27))
    z = z * _M2
    return z ^ (z >> np.uint64(31))


def stream_key(seed: int, uid: int, kind: int) -> int:
    """64-bit key of the stream (seed, uid, kind)."""
    k = _mix64_int(seed * GOLDEN + 0x632BE59BD9B4E019)
    k = _mix64_int(k ^ ((uid * 0xD1B54A32D192ED03) & MASK64))
    return _mix64_int(k + kind * GOLDEN)


def words(key: int, start: int, count: int) -> np.ndarray:
    """Outputs start .. start+count-1 of the stream with the given key."""
    with np.errstate(over="ignore"):
        idx = np.arange(start + 1, start + count + 1, dtype=np.uint64)
        return _mix64(np.uint64(key) + idx * np.uint64(GOLDEN))


def uniform01(key: int, n: int, start: int = 0) -> np.ndarray:
    """n doubles uniform on [0, 1) with 53 random bits each."""
    return (words(key, start, n) >> np.uint64(11)).astype(np.float64) * 2.0 ** -53


def normal(key: int, n: int, start: int = 0) -> np.ndarray:
    """n standard normal doubles, element i from outputs 2(start+i) and 2(start+i)+1."""
    w = words(key, 2 * start, 2 * n)
    u1 = ((w[0::2] >> np.uint64(11)).astype(np.float64) + 1.0) * 2.0 ** -53  # (0, 1]
    u2 = (w[1::2] >> np.uint64(11)).astype(np.float64) * 2.0 ** -53          # [0, 1)
    return np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * np.pi * u2)


def to_f16(a: np.ndarray) -> np.ndarray:
    """Round to fp16, nearest-even (numpy's float64 -> float16 cast)."""
    return np.asarray(a, dtype=np.float64).astype(np.float16)


def int4_codes(seed: int, uid: int, N: int, K: int, row0: int = 0, rows: int | None = None) -> np.ndarray:
    """Packed codes uint8[rows][K/2] of rows row0 .. row0+rows-1 of an N x K tensor."""
    assert K % 32 == 0
    rows = N - row0 if rows is None else rows
    rb = K // 2
    assert rb % 8 == 0
    key = stream_key(seed, uid, KIND_CODES)
    w = words(key, row0 * rb // 8, rows * rb // 8)
    return w.view(np.uint8).reshape(rows, rb)


def _scale_lut() -> np.ndarray:
    k = np.arange(65536, dtype=np.float64)
    return to_f16(0.005 + 0.015 * k / 65536.0)


_LUT = None


def group_scales(seed: int, uid: int, N: int, K: int, row0: int = 0, rows: int | None = None) -> np.ndarray:
    """fp16 group scales [rows][K/32], one per 32 consecutive inputs of a row."""
    global _LUT
    if _LUT is None:
        _LUT = _scale_lut()
    rows = N - row0 if rows is None else rows
    g = K // 32
    key = stream_key(seed, uid, KIND_SCALES)
    w = words(key, row0 * g, rows * g)
    return _LUT[(w & np.uint64(0xFFFF)).astype(np.int64)].reshape(rows, g)


def activations(seed: int, uid: int, M: int, K: int) -> np.ndarray:
    """fp16 activations [M][K], N(0, 1) rounded to nearest-even."""
    key = stream_key(seed, uid, KIND_ACT)
    return to_f16(normal(key, M * K)).reshape(M, K)


def exact_activations(seed: int, uid: int, M: int, K: int) -> np.ndarray:
    """fp16 activations [M][K] with values in {-4, ..., 4} / 4."""
    key = stream_key(seed, uid, KIND_ACT)
    v = (words(key, 0, M * K) % np.uint64(9)).astype(np.int64) - 4
    return to_f16(v * 0.25).reshape(M, K)


def sign_activations(seed: int, uid: int, M: int, K: int) -> np.ndarray:
    """fp16 activations [M][K] of +1 or -1 (every row has mean square exactly 1)."""
    key = stream_key(seed, uid, KIND_ACT)
    v = (words(key, 0, M * K) & np.uint64(1)).astype(np.int64) * 2 - 1
    return to_f16(v.astype(np.float64)).reshape(M, K)


def exact_scales(N: int, K: int) -> np.ndarray:
    """fp16 scales [N][K/32], all 2**-6."""
    return np.full((N, K // 32), 2.0 ** -6, dtype=np.float16)


def router_weights(seed: int, uid: int, H: int, E: int) -> np.ndarray:
    """fp16 router matrix [H][E] with entries N(0, 1/H)."""
    key = stream_key(seed, uid, KIND_ROUTER)
    return to_f16(normal(key, H * E) / np.sqrt(H)).reshape(H, E)


def permutation(seed: int, uid: int, n: int) -> np.ndarray:
    """Seeded permutation of 0..n-1 (stable argsort of n generator outputs)."""
    key = stream_key(seed, uid, KIND_PERM)
    return np.argsort(words(key, 0, n), kind="stable").astype(np.int64)


def scores(seed: int, uid: int, n: int) -> np.ndarray:
    """n seeded scores uniform on [0, 1)."""
    return uniform01(stream_key(seed, uid, KIND_SCORE), n)
