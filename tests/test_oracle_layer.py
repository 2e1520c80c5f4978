"""Pin of the oracle's decoder-layer composition (CPU only): a layer worked by
hand from single-code weights (tests/golden/decoder_layer_worked.json), with
the expected values written from the hand derivation's closed forms, and a
check that the plausible mis-compositions (feeding the FFN the norm of the
layer input, a post-norm order, a dropped residual, another head mapping)
all disagree with it."""
import json
import math
import os

import numpy as np

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def _single_code(N, col_offset, scales):
    """N x 32 tensor: row n holds q = 1 at input n + col_offset, 0 elsewhere."""
    q = np.zeros((N, 32), np.int64)
    for n in range(N):
        q[n, n + col_offset] = 1
    u = (q + 8).astype(np.uint8)
    codes = (u[:, 0::2] | (u[:, 1::2] << 4)).astype(np.uint8)
    return codes, np.asarray(scales, np.float16).reshape(N, 1)


def _fixture():
    with open(os.path.join(HERE, "golden", "decoder_layer_worked.json")) as f:
        g = json.load(f)
    W = {"q": _single_code(32, 0, [0.5] * 32), "k": _single_code(16, 16, [2.0] * 16),
         "v": _single_code(16, 0, [(n + 1) / 8 for n in range(16)]), "o": _single_code(32, 0, [1.0] * 32),
         "gate": _single_code(32, 0, [1.0] * 32), "up": _single_code(32, 0, [1.0] * 32),
         "down": _single_code(32, 0, [1.0] * 32)}
    h = np.stack([np.full(32, 2.0), np.full(32, 4.0)]).astype(np.float16)
    return g, W, h


def _silu(z):
    return z / (1.0 + math.exp(-z))


def _by_hand(h_const, fold_norm_of=None, post_norm=False, first_residual=True, head_of=lambda i: i // 2):
    """The hand derivation for a constant input row, with optional mistakes."""
    v = [(n + 1) / 8 for n in range(16)]
    attn = [v[8 * head_of(i) + d] for i in range(4) for d in range(8)]
    h1 = [(h_const if first_residual else 0.0) + a for a in attn]
    if post_norm:
        r = math.sqrt(sum(x * x for x in h1) / 32)
        h1 = [x / r for x in h1]
    src = h1 if fold_norm_of is None else fold_norm_of
    r = math.sqrt(sum(x * x for x in src) / 32)
    return [x + _silu(s / r) * (s / r) for x, s in zip(h1, src)]


def test_decoder_layer_worked_by_hand():
    g, W, h = _fixture()
    h2, zeta, aux = oracle.decoder_layer(h, W, g["n_heads"], g["n_kv"], g["head_dim"], eps=g["eps"])
    assert np.array_equal(aux["q"], np.full((2, 32), 0.5))
    assert np.array_equal(aux["k"], np.full((2, 16), 2.0))
    assert np.array_equal(aux["v"], np.tile([(n + 1) / 8 for n in range(16)], (2, 1)))
    # the hand-computed anchors: h1 of token 0 and both tokens' mean squares
    h1_0 = np.array(g["h1_token0"])
    assert math.isclose(float(np.mean(h1_0 ** 2)), g["mean_sq_h1"][0], rel_tol=0, abs_tol=0)
    assert math.isclose(float(np.mean((h1_0 + 2) ** 2)), g["mean_sq_h1"][1], rel_tol=0, abs_tol=0)
    for t, c in enumerate((2.0, 4.0)):
        want = np.array(_by_hand(c))
        assert np.allclose(h2[t], want, rtol=1e-14, atol=0), t
        # the same through the anchors alone
        h1 = h1_0 + (c - 2.0)
        b = h1 / math.sqrt(g["mean_sq_h1"][t])
        assert np.allclose(h2[t], h1 + b / (1 + np.exp(-b)) * b, rtol=1e-14, atol=0)
    assert np.all(zeta >= np.abs(h2))


def test_worked_layer_rejects_miscompositions():
    """Each plausible mistake moves some output by far more than rounding."""
    g, W, h = _fixture()
    h2, _, _ = oracle.decoder_layer(h, W, g["n_heads"], g["n_kv"], g["head_dim"], eps=g["eps"])
    for t, c in enumerate((2.0, 4.0)):
        wrong = {
            "FFN on rms(h)": _by_hand(c, fold_norm_of=[c] * 32),
            "post-norm": _by_hand(c, post_norm=True),
            "no first residual": _by_hand(c, first_residual=False),
            "head i takes KV head i % n_kv": _by_hand(c, head_of=lambda i: i % 2),
        }
        for name, w in wrong.items():
            assert np.max(np.abs(h2[t] - np.array(w))) > 1e-2, (t, name)
    # a dropped second residual: h2 would be the FFN output alone
    f_only = np.array(_by_hand(2.0)) - np.array(g["h1_token0"])
    assert np.max(np.abs(h2[0] - f_only)) > 1.0
