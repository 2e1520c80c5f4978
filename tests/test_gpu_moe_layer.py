"""GPU parity of the MoE decoder layer (attention plus a routed MoE FFN, the
layers of the 235B-A22B-shaped stack) against the fp64 oracle, and
placement invariance with 40 % of the experts streamed from host."""
import numpy as np
import pytest

import oracle
import synth
from synth import configs
from tests import stages
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


def _run_and_check(sess, L, M, seed, name, sample=False):
    """The layer through the C ABI with every intermediate exposed; each stage
    against the oracle on the GPU's own input to it: attention (q, k, the
    attention output, O + residual), router logits on rms(h_attn), routing,
    bucketing, the routed experts' SwiGLU activations and down projections,
    and the combine with the residual.  Small calls also compare the whole
    layer with the oracle layer on the GPU's routing.  sample: check sampled
    rows, pairs and columns of the large stages (the routing, bucketing and
    combine are checked in full)."""
    import torch
    s = L.s
    H, E, k = s["hidden"], s["n_experts"], s["top_k"]
    hn = synth.activations(seed, 400 + M, M, H)
    h = _dev(hn)
    q_out = torch.empty((M, s["n_heads"] * s["head_dim"]), dtype=torch.float16, device="cuda")
    k_out = torch.empty((M, s["n_kv"] * s["head_dim"]), dtype=torch.float16, device="cuda")
    dbg = L.layer(h, q_out, k_out, debug=True)
    sess.sync()
    g = {n: t.cpu().numpy() for n, t in dict(dbg, q=q_out, k=k_out, h=h).items()}
    perm = synth.permutation(seed, 7, 1 << 20)
    rows = np.sort(perm[perm < M][:256]) if sample else np.arange(M)
    cols = np.sort(perm[perm < max(H, s["n_heads"] * s["head_dim"])][:256]) if sample else None
    stages.attention_stages(L.W, s["n_heads"], s["n_kv"], s["head_dim"], hn[rows], g["q"][rows], g["k"][rows],
                            g["attn"][rows], g["h_attn"][rows], name, cols=cols)
    # the MoE half on the GPU's own residual stream after attention
    h1 = g["h_attn"].astype(np.float64)
    x, _ = oracle.rmsnorm(h1, 1e-6)
    lr, zl = oracle.router_logits(x, L.wr, L.bias.astype(np.float64))
    check(g["logits"], lr, zl, name=f"{name} logits", tight=H * 2.0 ** -24 + 2.0 ** -20)
    idx, p = g["idx"], g["p"].astype(np.float64)
    decided = stages.moe_routing(g["logits"].astype(np.float64), idx, p, lr, E, k, name)
    assert decided.sum() >= int(0.6 * M), f"{name}: too many near-tied routing decisions"
    for key, refv in zip(("counts", "offsets", "perm", "inv_perm"), oracle.bucket(idx, E)):
        assert np.array_equal(g[key], refv), f"{name}: {key}"
    if sample:
        pairs = np.sort(synth.permutation(seed, 8, M * k)[:256])
        ci = np.sort(synth.permutation(seed, 9, s["inter"])[:128])
        ch = np.sort(synth.permutation(seed, 10, H)[:128])
    else:
        pairs = ci = ch = None
    stages.moe_stages(L.experts, x, idx, p, g["expert_h"], g["expert_out"], g["h"], name, res=h1, mfma=M > 4,
                      norm=True, pairs=pairs, cols_i=ci, cols_h=ch)
    if not sample:
        # the whole MoE half on the GPU's routing, and the whole layer where the
        # routing is decided, against the oracle layer
        yr, zr, _ = oracle.moe_ffn(x, L.wr, L.bias.astype(np.float64), L.experts, k, route=(idx, p))
        check(g["h"], h1 + yr, zr + np.abs(h1), name=f"{name} MoE half on the GPU's routing",
              rel_l2=stages.COMPOSITE_ROW_L2)
        ref, zeta, _, _ = L.reference(hn)
        if decided.any():
            check(g["h"][decided], ref[decided], zeta[decided], name=f"{name} layer", rel_l2=stages.COMPOSITE_ROW_L2)


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


def test_moe_stack_layer_prefill_2048(sess, stack_layer):
    """The 235B-A22B-shaped layer at a 2048-token prefill chunk (expert buckets
    of up to 2048 rows) with 40 % of its experts streamed from host: routing,
    bucketing and the combine in full, the other stages on sampled rows,
    routed pairs and columns."""
    L = stack_layer
    host_exp = configs.moe_host_experts(frac=0.40, seed=configs.MOE_STACK.seed, layer=configs.MOE_STACK.n_layers - 1)
    mask = list(sess.placement)
    for j in range(3):
        for e in range(L.s["n_experts"]):
            mask[L.tids[j][e]] = int(host_exp[e])
    sess.set_placement(mask)
    try:
        _run_and_check(sess, L, 2048, configs.MOE_STACK.seed, "moe stack layer M=2048", sample=True)
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

