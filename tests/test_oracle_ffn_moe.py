"""Pins of the oracle's SwiGLU FFN, routing, bucketing, MoE and layer glue (CPU only)."""
import math

import numpy as np
import pytest

import oracle
import synth


def _qt(seed, uid, N, K):
    return synth.int4_codes(seed, uid, N, K), synth.group_scales(seed, uid, N, K)


def _diag_tensor(n, scale):
    """n x n quantised tensor with q = 1 on the diagonal and 0 elsewhere."""
    q = np.zeros((n, n), np.int64)
    np.fill_diagonal(q, 1)
    u = (q + 8).astype(np.uint8)
    codes = (u[:, 0::2] | (u[:, 1::2] << 4)).astype(np.uint8)
    return codes, np.full((n, n // 32), scale, np.float16)


# ----------------------------------------------------------------------------- SiLU / SwiGLU

def test_silu_closed_forms():
    assert oracle.silu(np.array([0.0]))[0] == 0.0
    z = np.linspace(-30, 30, 1001)
    assert np.all(np.abs(oracle.silu(z) - oracle.silu(-z) - z) <= 1e-14 * (1 + np.abs(z)))
    assert abs(oracle.silu(np.array([1.0]))[0] - 1.0 / (1.0 + math.exp(-1.0))) <= 1e-16
    assert abs(oracle.silu(np.array([1.0]))[0] - 0.7310585786300049) <= 1e-16
    # the derivative bound used for error propagation
    zz = np.linspace(-20, 20, 200001)
    s = 1.0 / (1.0 + np.exp(-zz))
    assert np.max(np.abs(s * (1 + zz * (1 - s)))) <= oracle.SILU_DERIV_MAX


def test_swiglu_ffn_identity_weights():
    """gate = 2 I, up = I, down = I gives y = silu(2x) * x (and not silu(x) * 2x)."""
    n = 64
    x = synth.activations(9, 1, 3, n)
    y, zeta, _ = oracle.swiglu_ffn(x, _diag_tensor(n, 2.0), _diag_tensor(n, 1.0), _diag_tensor(n, 1.0))
    xd = x.astype(np.float64)
    expect = (2 * xd) / (1 + np.exp(-2 * xd)) * xd
    assert np.all(np.abs(y - expect) <= 1e-14 * (1 + np.abs(expect)))
    assert np.all(zeta >= np.abs(y))


def test_ffn_zero_gate_gives_zero():
    n = 64
    zero = (np.full((n, n // 2), 0x88, np.uint8), np.full((n, n // 32), 0.01, np.float16))
    x = synth.activations(9, 2, 2, n)
    y, _, _ = oracle.swiglu_ffn(x, zero, _qt(9, 3, n, n), _qt(9, 4, n, n))
    assert np.all(y == 0)


def test_zeta_bounds_planted_perturbations():
    """zeta is a first-order bound: perturb every intermediate by at most eps*zeta
    (and round h to fp16) and the output moves by at most eps*zeta_y."""
    K, I, N, M, eps = 256, 96, 128, 4, 1e-3
    gate, up, down = _qt(13, 1, I, K), _qt(13, 2, I, K), _qt(13, 3, N, I)
    x = synth.activations(13, 4, M, K)
    y, zy, _ = oracle.swiglu_ffn(x, gate, up, down)
    rng_key = synth.stream_key(13, 5, 7)
    for trial in range(4):
        g, zg = oracle.linear(x, *gate)
        u, zu = oracle.linear(x, *up)
        r = synth.uniform01(rng_key, 2 * g.size, start=trial * 4 * g.size) * 2 - 1
        g2 = g + eps * zg * r[: g.size].reshape(g.shape)
        u2 = u + eps * zu * r[g.size:].reshape(u.shape)
        h2 = (oracle.silu(g2) * u2).astype(np.float16).astype(np.float64)
        y2, zy2 = oracle.linear(h2, *down)
        y2 = y2 + eps * zy2 * np.sign(synth.uniform01(rng_key, y2.size, start=trial * 7 * g.size).reshape(y2.shape) - 0.5)
        assert np.all(np.abs(y2 - y) <= 1.05 * eps * zy + 1e-12)


# ----------------------------------------------------------------------------- routing

def test_topk_weights_sum_to_one_and_match_renormalised_softmax():
    x = synth.activations(21, 1, 64, 256)
    wr = synth.router_weights(21, 2, 256, 128)
    logits, _ = oracle.router_logits(x, wr)
    idx, p = oracle.topk_route(logits, 8)
    assert np.all(np.abs(p.sum(axis=1) - 1.0) <= 8 * 2.0 ** -52)
    full = np.exp(logits - logits.max(axis=1, keepdims=True))
    full /= full.sum(axis=1, keepdims=True)
    sel = np.take_along_axis(full, idx.astype(np.int64), axis=1)
    assert np.allclose(sel / sel.sum(axis=1, keepdims=True), p, rtol=1e-13, atol=0)
    # rank order: weights non-increasing across slots; the selection really is the top 8
    assert np.all(np.diff(p, axis=1) <= 0)
    for t in range(64):
        ranked = sorted(range(128), key=lambda e: (-logits[t, e], e))
        assert list(idx[t]) == ranked[:8]


def test_topk_ties_lower_id_first_and_k_equals_e():
    logits = np.array([[1.0, 3.0, 3.0, 0.5, 3.0, -1.0]])
    idx, p = oracle.topk_route(logits, 3)
    assert list(idx[0]) == [1, 2, 4]
    assert np.allclose(p, 1 / 3)
    idx, p = oracle.topk_route(logits, 6)
    assert list(idx[0]) == [1, 2, 4, 0, 3, 5]
    full = np.exp(logits[0] - 3.0)
    assert np.allclose(p[0], full[idx[0]] / full.sum(), rtol=1e-15)


def test_router_logits_bias_and_magnitude():
    x = synth.activations(22, 1, 3, 64)
    wr = synth.router_weights(22, 2, 64, 16)
    b = np.linspace(-1, 1, 16)
    l0, z0 = oracle.router_logits(x, wr)
    l1, z1 = oracle.router_logits(x, wr, b)
    assert np.allclose(l1 - l0, b[None, :], rtol=0, atol=1e-15)
    # brute force over k for one entry
    acc = sum(float(x[1, k]) * float(wr[k, 5]) for k in range(64))
    assert abs(l0[1, 5] - acc) <= 1e-13 * z0[1, 5]


# ----------------------------------------------------------------------------- bucketing

def _bucket_bruteforce(idx, E):
    T, k = idx.shape
    perm = []
    for e in range(E):
        for t in range(T):
            for j in range(k):
                if idx[t, j] == e:
                    perm.append(k * t + j)
    return np.array(perm, np.int32)


@pytest.mark.parametrize("T,E,k", [(1, 128, 8), (37, 16, 4), (200, 128, 8)])
def test_bucket_invariants_and_bruteforce(T, E, k):
    key = synth.stream_key(31, T, 7)
    idx = np.stack([synth.permutation(31, 1000 + t, E)[:k] for t in range(T)]).astype(np.int32)
    counts, offsets, perm, inv = oracle.bucket(idx, E)
    assert counts.sum() == T * k and offsets[0] == 0 and offsets[-1] == T * k
    assert np.all(np.diff(offsets) == counts)
    assert np.array_equal(np.sort(perm), np.arange(T * k))
    assert np.array_equal(inv[perm], np.arange(T * k))
    for e in range(E):
        seg = perm[offsets[e]:offsets[e + 1]]
        assert np.all(idx.reshape(-1)[seg] == e)
        assert np.all(np.diff(seg // k) > 0)
    assert np.array_equal(perm, _bucket_bruteforce(idx, E))
    del key


def test_bucket_all_to_one_expert_and_empty_experts():
    T, E, k = 50, 32, 4
    idx = np.tile(np.array([[5, 0, 9, 31]], np.int32), (T, 1))
    counts, offsets, perm, inv = oracle.bucket(idx, E)
    assert counts[5] == T and counts[0] == T and counts[1] == 0
    assert np.array_equal(perm[offsets[5]:offsets[6]], np.arange(T) * k)
    assert np.array_equal(perm, _bucket_bruteforce(idx, E))


# ----------------------------------------------------------------------------- MoE

def _moe_setup(E=16, H=64, I=32, T=12, seed=41):
    experts = [(_qt(seed, 10 * e + 1, I, H), _qt(seed, 10 * e + 2, I, H), _qt(seed, 10 * e + 3, H, I))
               for e in range(E)]
    x = synth.activations(seed, 1, T, H)
    wr = synth.router_weights(seed, 2, H, E)
    bias = np.linspace(0.5, -0.5, E)
    return experts, x, wr, bias


def test_moe_matches_dense_bruteforce():
    experts, x, wr, bias = _moe_setup()
    E, k = len(experts), 4
    y, zeta, aux = oracle.moe_ffn(x, wr, bias, experts, k)
    # dense: every expert on every token, then keep the top-k by its own ranking
    all_out = np.stack([oracle.swiglu_ffn(x, *experts[e])[0] for e in range(E)], axis=1)
    xd = x.astype(np.float64)
    for t in range(x.shape[0]):
        lg = [sum(xd[t, kk] * float(wr[kk, e]) for kk in range(x.shape[1])) + bias[e] for e in range(E)]
        top = sorted(range(E), key=lambda e: (-lg[e], e))[:k]
        w = np.array([math.exp(lg[e] - lg[top[0]]) for e in top])
        w /= w.sum()
        yt = sum(w[j] * all_out[t, top[j]] for j in range(k))
        assert np.all(np.abs(y[t] - yt) <= 1e-12 * zeta[t])
        assert list(aux["idx"][t]) == top


def test_moe_relabelling_invariance():
    experts, x, wr, bias = _moe_setup(seed=43)
    y, zeta, _ = oracle.moe_ffn(x, wr, bias, experts, 4)
    perm = synth.permutation(43, 99, len(experts))
    y2, _, _ = oracle.moe_ffn(x, wr[:, perm], bias[perm], [experts[e] for e in perm], 4)
    assert np.all(np.abs(y2 - y) <= 1e-12 * zeta)


# ----------------------------------------------------------------------------- glue

def test_rmsnorm_closed_forms():
    c = 3.0
    n, _ = oracle.rmsnorm(np.full((2, 64), c), eps=1e-6)
    assert np.allclose(n, c / math.sqrt(c * c + 1e-6), rtol=1e-15)
    v = synth.activations(51, 1, 4, 256).astype(np.float64)
    n, _ = oracle.rmsnorm(v, eps=0.0)
    assert np.allclose((n * n).mean(axis=1), 1.0, rtol=1e-14)
    n2, _ = oracle.rmsnorm(-2.5 * v, eps=0.0)
    assert np.allclose(n2, -n, rtol=1e-14)


def test_gqa_stub_is_single_key_attention():
    nh, nkv, hd, m = 8, 2, 16, 3
    q = synth.activations(52, 1, m, nh * hd).astype(np.float64)
    k = synth.activations(52, 2, m, nkv * hd).astype(np.float64)
    v = synth.activations(52, 3, m, nkv * hd).astype(np.float64)
    ref = oracle.attention_single_key(q, k, v, nh, nkv, hd)
    assert np.array_equal(oracle.gqa_stub(v, nh, nkv, hd), ref)


def test_decoder_layer_zero_weights_is_identity():
    H = 64
    zero = lambda n, kk: (np.full((n, kk // 2), 0x88, np.uint8), np.full((n, kk // 32), 0.01, np.float16))
    W = {"q": zero(64, H), "k": zero(32, H), "v": zero(32, H), "o": zero(H, 64),
         "gate": zero(96, H), "up": zero(96, H), "down": zero(H, 96)}
    h = synth.activations(53, 1, 2, H)
    h2, _, _ = oracle.decoder_layer(h, W, n_heads=4, n_kv=2, head_dim=16)
    assert np.array_equal(h2, h.astype(np.float64))
