"""GPU parity of the MoE decoder layer (attention plus a routed MoE FFN, the
layers of the 235B-A22B-shaped stack) against the fp64 oracle, and
placement invariance with 40 % of the experts streamed from host."""
import numpy as np
import pytest

import oracle
import synth
from synth import configs
from tests.parity import check

pytestmark = pytest.mark.gpu

SMALL = dict(hidden=256, n_heads=4, n_kv=2, head_dim=64, n_experts=16, top_k=4, inter=96)
STACK = dict(hidden=configs.MOE_STACK.dense.hidden, n_heads=configs.MOE_STACK.dense.n_heads,
             n_kv=configs.MOE_STACK.dense.n_kv, head_dim=configs.MOE_STACK.dense.head_dim,
             n_experts=configs.MOE_STACK.moe.n_experts, top_k=configs.MOE_STACK.moe.top_k,
             inter=configs.MOE_STACK.moe.inter)


@pytest.fixture(scope="module")
def sess():
    from paper_2607_10183_amd.session import Session
    s = Session(workspace_bytes=3 << 30, n_slots=24)
    yield s
    s.close()


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _qt(seed, uid, N, K):
    return synth.int4_codes(seed, uid, N, K), synth.group_scales(seed, uid, N, K)


class _Layer:
    """One MoE decoder layer: seeded attention, router (capped-Zipf bias for
    the stack shape) and experts, registered with HBM and host copies."""

    def __init__(self, sess, seed, layer, shape):
        import torch
        from paper_2607_10183_amd.session import MoEDecoderLayer
        self.s = shape
        H, E, I = shape["hidden"], shape["n_experts"], shape["inter"]
        Hq, Hkv = shape["n_heads"] * shape["head_dim"], shape["n_kv"] * shape["head_dim"]
        kn = {"q": (H, Hq), "k": (H, Hkv), "v": (H, Hkv), "o": (Hq, H)}
        self.W = {r: _qt(seed, configs.dense_uid(layer, r), kn[r][1], kn[r][0]) for r in ("q", "k", "v", "o")}
        self.attn = {r: sess.register(*self.W[r], hbm=True, host=True) for r in ("q", "k", "v", "o")}
        self.experts = []
        tids = [[], [], []]
        for e in range(E):
            trio = tuple(_qt(seed, configs.expert_uid(layer, e, p), n, kk)
                         for p, (n, kk) in zip(("gate", "up", "down"), ((I, H), (I, H), (H, I))))
            self.experts.append(trio)
            for j, t in enumerate(sess.register_group(trio, hbm=True, host=True)):
                tids[j].append(t)
        self.tids = tids
        self.wr = synth.router_weights(seed, configs.router_uid(layer), H, E)
        if E == 128 and shape["top_k"] == 8:
            from synth.calibrate_router_bias import load_bias
            self.bias = load_bias().astype(np.float32)
        else:
            self.bias = (np.linspace(1.5, -1.5, E)[synth.permutation(seed, 3, E)]).astype(np.float32)
        self.moe = sess.moe_layer(_dev(self.wr), *tids, top_k=shape["top_k"], router_bias=torch.from_numpy(self.bias).cuda())
        a = self.attn
        self.layer = MoEDecoderLayer(self.moe, a["q"], a["k"], a["v"], a["o"], shape["n_heads"], shape["n_kv"],
                                     shape["head_dim"], 1e-6)

    def reference(self, hn):
        s = self.s
        box = {}

        def ffn(b, zb):
            y, zy, aux = oracle.moe_ffn(b, self.wr, self.bias.astype(np.float64), self.experts, s["top_k"], x_zeta=zb)
            box.update(aux)
            return y, zy

        ref, zeta, aux = oracle.decoder_layer(hn, self.W, s["n_heads"], s["n_kv"], s["head_dim"], 1e-6, ffn=ffn)
        return ref, zeta, aux, box


def _decided(gpu_logits, logits, k):
    """Tokens whose top-k set is unique: the oracle's k-th and (k+1)-th logits
    are further apart than twice the GPU's largest logit error on that token.
    (The router sees h after the attention half, in fp16, so its logits carry
    that half's rounding; the logit error itself is checked against the
    propagated magnitude.)"""
    delta = np.abs(gpu_logits - logits).max(axis=1)
    srt = -np.sort(-logits, axis=1)
    return srt[:, k - 1] - srt[:, k] > 2 * delta, delta


def _run_and_check(sess, L, M, seed, name):
    import torch
    s = L.s
    hn = synth.activations(seed, 400 + M, M, s["hidden"])
    h = _dev(hn)
    q_out = torch.empty((M, s["n_heads"] * s["head_dim"]), dtype=torch.float16, device="cuda")
    k_out = torch.empty((M, s["n_kv"] * s["head_dim"]), dtype=torch.float16, device="cuda")
    dbg = L.layer(h, q_out, k_out, debug=True)
    sess.sync()
    ref, zeta, aux, box = L.reference(hn)
    k = s["top_k"]
    lg = dbg["logits"].cpu().numpy().astype(np.float64)
    check(lg, box["logits"], box["logit_zeta"], name=f"{name} logits")
    dec, delta = _decided(lg, box["logits"], k)
    assert dec.sum() >= int(0.6 * M), f"{name}: too many near-tied routing decisions"
    idx = dbg["idx"].cpu().numpy()
    # every selection is a valid top-k of the oracle logits within the logit error
    kth = -np.sort(-box["logits"], axis=1)[:, k - 1]
    chosen = np.take_along_axis(box["logits"], idx.astype(np.int64), axis=1)
    assert np.all(chosen >= (kth - 2 * delta)[:, None]), f"{name}: a selection is not a valid top-k"
    for t in np.nonzero(dec)[0]:
        assert set(idx[t]) == set(box["idx"][t]), f"{name}: token {t} routed to other experts"
    if dec.any():
        check(h.cpu().numpy()[dec], ref[dec], zeta[dec], name=f"{name} h")
    a, za = oracle.rmsnorm(hn.astype(np.float64), 1e-6)
    qr, zq = oracle.linear(a, *L.W["q"], za)
    kr, zk = oracle.linear(a, *L.W["k"], za)
    check(q_out.cpu().numpy(), qr, zq, name=f"{name} q")
    check(k_out.cpu().numpy(), kr, zk, name=f"{name} k")
    # bucketing of the GPU's own routing is the oracle's bucketing of it
    for key, refv in zip(("counts", "offsets", "perm", "inv_perm"), oracle.bucket(idx, s["n_experts"])):
        assert np.array_equal(dbg[key].cpu().numpy(), refv), f"{name}: {key}"


@pytest.mark.parametrize("M", [1, 5, 16, 64])
def test_moe_decoder_layer_small(sess, M):
    L = _Layer(sess, 91, 0, SMALL)
    _run_and_check(sess, L, M, 91, f"moe layer small M={M}")


@pytest.fixture(scope="module")
def stack_layer(sess):
    # the last of the 94 layers (seeded like every layer of the stack)
    return _Layer(sess, configs.MOE_STACK.seed, configs.MOE_STACK.n_layers - 1, STACK)


@pytest.mark.parametrize("M", [1, 64])
def test_moe_stack_layer_parity(sess, stack_layer, M):
    """A 235B-A22B-shaped layer (hidden 4096, 64 / 4 heads, 128 experts of
    SwiGLU 1536, top-8) with 40 % of its experts streamed from host."""
    L = stack_layer
    host_exp = configs.moe_host_experts(frac=0.40, seed=configs.MOE_STACK.seed, layer=configs.MOE_STACK.n_layers - 1)
    mask = list(sess.placement)
    for j in range(3):
        for e in range(L.s["n_experts"]):
            mask[L.tids[j][e]] = int(host_exp[e])
    sess.set_placement(mask)
    try:
        _run_and_check(sess, L, M, configs.MOE_STACK.seed, f"moe stack layer M={M}")
    finally:
        for j in range(3):
            for e in range(L.s["n_experts"]):
                mask[L.tids[j][e]] = 0
        sess.set_placement(mask)


@pytest.mark.parametrize("M", [1, 64])
def test_moe_layer_placement_invariance(sess, stack_layer, M):
    """All-HBM, the seeded 40 % mask and all experts on host give bit-identical layers."""
    import torch
    L = stack_layer
    h0 = _dev(synth.activations(configs.MOE_STACK.seed, 500 + M, M, L.s["hidden"]))
    host_exp = configs.moe_host_experts(frac=0.40, seed=configs.MOE_STACK.seed, layer=configs.MOE_STACK.n_layers - 1)
    outs = []
    for mode in ("hbm", "mask", "host"):
        mask = list(sess.placement)
        for j in range(3):
            for e in range(L.s["n_experts"]):
                mask[L.tids[j][e]] = {"hbm": 0, "host": 1, "mask": int(host_exp[e])}[mode]
        sess.set_placement(mask)
        h = h0.clone()
        L.layer(h)
        outs.append(h)
    sess.sync()
    mask = list(sess.placement)
    for j in range(3):
        for e in range(L.s["n_experts"]):
            mask[L.tids[j][e]] = 0
    sess.set_placement(mask)
    for o in outs[1:]:
        assert torch.equal(outs[0], o)


@pytest.mark.parametrize("M,host_attn", [(1, False), (4, False), (1, True)])
def test_moe_layer_zero_copy(sess, stack_layer, M, host_attn):
    """Decode of the 235B-shaped layer with the seeded 40 % of experts on host,
    read in place (zero-copy): the all-HBM bits, and nothing copied; with the
    attention tensors on host too, those alone are copied."""
    import torch
    L = stack_layer
    h0 = _dev(synth.activations(configs.MOE_STACK.seed, 800 + M, M, L.s["hidden"]))
    host_exp = configs.moe_host_experts(frac=0.40, seed=configs.MOE_STACK.seed, layer=configs.MOE_STACK.n_layers - 1)

    def run(host):
        mask = list(sess.placement)
        for j in range(3):
            for e in range(L.s["n_experts"]):
                mask[L.tids[j][e]] = int(host_exp[e]) if host else 0
        for t in L.attn.values():
            mask[t] = int(host and host_attn)
        sess.set_placement(mask)
        h = h0.clone()
        L.layer(h)
        sess.sync()
        return h

    ref = run(False)
    try:
        sess.set_zero_copy(True)
        sess.stats(reset=True)
        got = run(True)
        st = sess.stats(reset=True)
    finally:
        sess.set_zero_copy(False)
        run(False)
    assert torch.equal(ref, got)
    attn_bytes = sum(configs.qbytes(*sess.shapes[t]) for t in L.attn.values())
    assert st["h2d_bytes"] == (attn_bytes if host_attn else 0)


def _sampled_layers():
    """The first layer and two seeded layers of the 94 (the last one is the
    stack_layer fixture above)."""
    n = configs.MOE_STACK.n_layers
    perm = [int(i) for i in synth.permutation(configs.MOE_STACK.seed, 97, n) if 0 < i < n - 1]
    return [0, perm[0], perm[1]]


@pytest.mark.parametrize("layer", _sampled_layers())
def test_moe_stack_sampled_layers(sess, layer):
    """Layers of the 235B-A22B-shaped stack besides the last: one decode
    token and a 64-token prefill chunk, all experts HBM-resident."""
    L = _Layer(sess, configs.MOE_STACK.seed, layer, STACK)
    for M in (1, 64):
        _run_and_check(sess, L, M, configs.MOE_STACK.seed, f"moe stack layer {layer} M={M}")

