"""GPU parity of MoE routing, bucketing and the routed expert FFN against the
fp64 oracle, plus placement invariance with streamed experts."""
import numpy as np
import pytest

import oracle
import synth
from synth import configs
from tests import stages
from tests.parity import check

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sess():
    from paper_2607_10183_amd.session import Session
    s = Session(workspace_bytes=2 << 30, n_slots=16)
    yield s
    s.close()


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _random_idx(seed, M, k, E):
    return np.stack([synth.permutation(seed, 5000 + t, E)[:k] for t in range(M)]).astype(np.int32)


@pytest.mark.parametrize("M,k,E", [(1, 8, 128), (37, 4, 16), (512, 8, 128), (2048, 8, 128), (3000, 8, 128),
                                   (64, 16, 64)])
def test_bucket_bitexact(sess, M, k, E):
    idx = _random_idx(81, M, k, E)
    outs = sess.moe_bucket(_dev(idx), E)
    sess.sync()
    for got, ref in zip(outs, oracle.bucket(idx, E)):
        assert np.array_equal(got.cpu().numpy(), ref)


def test_bucket_special_cases(sess):
    # every token picks expert 5 first; experts 1..4 stay empty
    M, k, E = 200, 4, 32
    idx = np.tile(np.array([[5, 0, 9, 31]], np.int32), (M, 1))
    outs = sess.moe_bucket(_dev(idx), E)
    sess.sync()
    for got, ref in zip(outs, oracle.bucket(idx, E)):
        assert np.array_equal(got.cpu().numpy(), ref)


def _logit_bound(zeta_ref, H):
    """Worst-case error of an fp32 sum of H exact fp16 products (any order),
    plus the bias add: (H + 64) * 2^-24 * sum |terms|."""
    return (H + 64) * 2.0 ** -24 * zeta_ref.max(axis=1)


def _route_decided(logits_ref, bound, k):
    """Tokens whose top-k set (and full order) the fp32 GPU logits cannot flip:
    consecutive gaps of the sorted oracle logits exceed twice the error bound."""
    srt = -np.sort(-logits_ref, axis=1)
    gaps = srt[:, :-1] - srt[:, 1:]
    boundary = gaps[:, k - 1] > 2 * bound
    order = np.all(gaps[:, :k] > 2 * bound[:, None], axis=1)
    return boundary, order


def _experts(seed, E, H, I):
    return [((synth.int4_codes(seed, 10 * e + 1, I, H), synth.group_scales(seed, 10 * e + 1, I, H)),
             (synth.int4_codes(seed, 10 * e + 2, I, H), synth.group_scales(seed, 10 * e + 2, I, H)),
             (synth.int4_codes(seed, 10 * e + 3, H, I), synth.group_scales(seed, 10 * e + 3, H, I)))
            for e in range(E)]


class _Setup:
    def __init__(self, sess, seed, E, H, I, k, host=False):
        import torch
        self.E, self.H, self.I, self.k = E, H, I, k
        self.experts = _experts(seed, E, H, I)
        self.wr = synth.router_weights(seed, 2, H, E)
        # a seeded skew so some experts draw many tokens and some none
        self.bias = (np.linspace(1.5, -1.5, E)[synth.permutation(seed, 3, E)]).astype(np.float32)
        groups = [sess.register_group(self.experts[e], hbm=True, host=host) for e in range(E)]
        self.tids = [[groups[e][j] for e in range(E)] for j in range(3)]
        self.layer = sess.moe_layer(_dev(self.wr), *self.tids, top_k=k, router_bias=torch.from_numpy(self.bias).cuda())


def _check_moe(y, dbg, st, xn, name):
    """Routing against the oracle logits; every token's output against the
    oracle evaluated on the GPU's own selection and weights (so near-tied
    tokens are checked too); the experts' stages teacher-forced."""
    ref, zeta, aux = oracle.moe_ffn(xn, st.wr, st.bias.astype(np.float64), st.experts, st.k)
    lg = dbg["logits"].cpu().numpy().astype(np.float64)
    check(lg, aux["logits"], aux["logit_zeta"], name=f"{name} logits", tight=st.H * 2.0 ** -24 + 2.0 ** -22)
    idx = dbg["idx"].cpu().numpy()
    p = dbg["p"].cpu().numpy().astype(np.float64)
    decided = stages.moe_routing(lg, idx, p, aux["logits"], st.E, st.k, name)
    n = len(decided)
    assert decided.sum() >= min(n - 1, 0.75 * n), f"{name}: too many near-tied routing decisions"
    # weights of tokens whose full order is decided against the oracle's
    bound = _logit_bound(aux["logit_zeta"], st.H)
    _, order = _route_decided(aux["logits"], bound, st.k)
    pz = oracle.softmax_weight_zeta(aux["p"], np.take_along_axis(aux["logit_zeta"], aux["idx"].astype(np.int64), 1))
    check(p[order], aux["p"][order], pz[order], name=f"{name} weights")
    stages.moe_stages(st.experts, xn.astype(np.float64), idx, p, dbg["expert_h"].cpu().numpy(),
                      dbg["expert_out"].cpu().numpy(), y.cpu().numpy(), name, mfma=xn.shape[0] > 4)
    check(y.cpu().numpy()[decided], ref[decided], zeta[decided], name=f"{name} output",
          rel_l2=stages.COMPOSITE_ROW_L2)
    ref_g, zeta_g, _ = oracle.moe_ffn(xn, st.wr, st.bias.astype(np.float64), st.experts, st.k, route=(idx, p))
    check(y.cpu().numpy(), ref_g, zeta_g, name=f"{name} output on the GPU's routing", rel_l2=stages.COMPOSITE_ROW_L2)
    # bucketing of the GPU's own routing is exactly the oracle's bucketing of it
    for key, refv in zip(("counts", "offsets", "perm", "inv_perm"), oracle.bucket(idx, st.E)):
        assert np.array_equal(dbg[key].cpu().numpy(), refv), f"{name}: {key}"


@pytest.mark.parametrize("M", [1, 3, 50])
def test_moe_small_parity(sess, M):
    st = _Setup(sess, 82, E=16, H=256, I=96, k=4)
    xn = synth.activations(82, 100 + M, M, st.H)
    y, dbg = st.layer(_dev(xn), debug=True)
    sess.sync()
    _check_moe(y, dbg, st, xn, f"moe small M={M}")


@pytest.mark.parametrize("k,M", [(12, 1), (16, 1), (9, 16), (16, 33), (9, 20)])
def test_moe_wide_topk_parity(sess, k, M):
    """More than 8 experts per token: the selection network keeps 16 per
    chunk; one token routes in the router's last workgroup, 20 and 33 in a
    second launch."""
    st = _Setup(sess, 83, E=64, H=256, I=96, k=k)
    xn = synth.activations(83, 100 + M, M, st.H)
    y, dbg = st.layer(_dev(xn), debug=True)
    sess.sync()
    _check_moe(y, dbg, st, xn, f"moe k={k} M={M}")


@pytest.fixture(scope="module")
def light_setup(sess):
    # hidden 768 and inter 512: three and two K-slices per light workgroup,
    # and output blocks the expert's rows do not fill
    return _Setup(sess, 85, E=16, H=768, I=512, k=4)


@pytest.mark.parametrize("light", [0, 32, 1 << 20])
@pytest.mark.parametrize("M", [5, 50, 300])
def test_moe_light_experts_parity(sess, light_setup, light, M):
    """Prefill experts on the grouped GEMM only (0), split by routed count
    (32: the light-expert kernels take experts of at most 32 pairs, one or two
    16-row tiles), or all on the light kernels (an expert of 200 pairs then
    has 13 tiles, the last one ragged)."""
    st = light_setup
    xn = synth.activations(85, 100 + M, M, st.H)
    sess.set_moe_light_rows(light)
    try:
        y, dbg = st.layer(_dev(xn), debug=True)
        sess.sync()
    finally:
        sess.set_moe_light_rows(-1)
    _check_moe(y, dbg, st, xn, f"moe light={light} M={M}")


@pytest.mark.parametrize("H,I", [(256, 1024), (1024, 256), (3072, 512)])
def test_moe_light_shapes(sess, H, I):
    """Light tiles of every height on other slice layouts: one K-slice and
    eight column groups (hidden 256), four slices and two groups (1024), and
    16-group slices at hidden 3072 (six slices, tiles of at most 32 rows);
    100 tokens route 400 pairs over 16 experts, so every tile height occurs."""
    st = _Setup(sess, 86, E=16, H=H, I=I, k=4)
    xn = synth.activations(86, 7, 100, H)
    sess.set_moe_light_rows(1 << 20)
    try:
        y, dbg = st.layer(_dev(xn), debug=True)
        sess.sync()
    finally:
        sess.set_moe_light_rows(-1)
    _check_moe(y, dbg, st, xn, f"moe light H={H} I={I}")


def test_moe_light_rows_range(sess):
    from paper_2607_10183_amd import atsi
    for bad in (-2, (1 << 20) + 1):
        with pytest.raises(atsi.AtsiError, match="ATSI_E_INVALID"):
            sess.set_moe_light_rows(bad)
    sess.set_moe_light_rows(-1)


@pytest.fixture(scope="module")
def cfg4(sess):
    shp = configs.MOE_LAYER.moe
    return _Setup(sess, configs.MOE_LAYER.seed, E=shp.n_experts, H=shp.hidden, I=shp.inter, k=shp.top_k, host=True)


@pytest.mark.parametrize("M", [1, 4, 512])
def test_moe_layer_parity(sess, cfg4, M):
    xn = synth.activations(configs.MOE_LAYER.seed, 200 + M, M, cfg4.H)
    y, dbg = cfg4.layer(_dev(xn), debug=True)
    sess.sync()
    _check_moe(y, dbg, cfg4, xn, f"moe_layer M={M}")


@pytest.mark.parametrize("M", [1, 512])
def test_moe_engine_checking_modes(sess, cfg4, M):
    """The seeded 40 % host mask under poisoned slots and with serialised
    copies gives the all-HBM output bit for bit."""
    import torch
    xn = synth.activations(configs.MOE_LAYER.seed, 400 + M, M, cfg4.H)
    x = _dev(xn)
    host_exp = configs.moe_host_experts()

    def run(mode):
        mask = list(sess.placement)
        for j in range(3):
            for e in range(cfg4.E):
                mask[cfg4.tids[j][e]] = {"hbm": 0, "mask": int(host_exp[e])}[mode]
        sess.set_placement(mask)
        y = cfg4.layer(x)
        sess.sync()
        return y

    ref = run("hbm")
    try:
        for poison, serialize in ((True, False), (False, True)):
            sess.set_debug(poison=poison, serialize=serialize)
            assert torch.equal(ref, run("mask")), (poison, serialize)
    finally:
        sess.set_debug()
        run("hbm")


@pytest.mark.parametrize("M", [1, 4, 512])
def test_moe_placement_invariance(sess, cfg4, M):
    """HBM-resident experts, the seeded 40 % host mask and all experts on host
    give bit-identical outputs (at decode sizes the all-resident layer indexes
    routed pairs directly, the others go through the buckets)."""
    import torch
    xn = synth.activations(configs.MOE_LAYER.seed, 300 + M, M, cfg4.H)
    x = _dev(xn)
    all_ids = [t for ids in cfg4.tids for t in ids]
    host_exp = configs.moe_host_experts()
    outs = []
    for mode in ("hbm", "mask", "host", "hbm"):
        mask = list(sess.placement)
        for j in range(3):
            for e in range(cfg4.E):
                mask[cfg4.tids[j][e]] = {"hbm": 0, "host": 1, "mask": int(host_exp[e])}[mode]
        sess.set_placement(mask)
        outs.append(cfg4.layer(x))
    sess.sync()
    mask = list(sess.placement)
    for t in all_ids:
        mask[t] = 0
    sess.set_placement(mask)
    for o in outs[1:]:
        assert torch.equal(outs[0], o)


@pytest.mark.parametrize("M", [1, 4, 512])
def test_moe_zero_copy(sess, cfg4, M):
    """Zero-copy mode with the seeded 40 % host mask: calls of at most 4
    tokens read the routed host experts in place (nothing is copied), larger
    ones keep the copy path; both give the all-HBM bits."""
    import torch
    x = _dev(synth.activations(configs.MOE_LAYER.seed, 600 + M, M, cfg4.H))
    host_exp = configs.moe_host_experts()

    def run(mode):
        mask = list(sess.placement)
        for j in range(3):
            for e in range(cfg4.E):
                mask[cfg4.tids[j][e]] = {"hbm": 0, "mask": int(host_exp[e])}[mode]
        sess.set_placement(mask)
        y = cfg4.layer(x)
        sess.sync()
        return y

    ref = run("hbm")
    copied = run("mask")
    try:
        sess.set_zero_copy(True)
        sess.stats(reset=True)
        outs = [run("mask") for _ in range(2)]
        st = sess.stats(reset=True)
    finally:
        sess.set_zero_copy(False)
        run("hbm")
    for y in outs:
        assert torch.equal(ref, y)
    assert torch.equal(ref, copied)
    if M <= 4:
        assert st["h2d_bytes"] == 0 and st["host_reads"] == 0
    else:
        assert st["h2d_bytes"] > 0


def test_zero_copy_needs_mapped_host_copies():
    """Zero-copy mode is refused while a host copy is ordinary (unmapped) host
    memory, and for a tensor with such a copy registered while it is on."""
    import torch
    from paper_2607_10183_amd import atsi
    from paper_2607_10183_amd.session import Session
    codes, scales = synth.int4_codes(84, 1, 64, 256), synth.group_scales(84, 1, 64, 256)
    dev_c = torch.from_numpy(codes).cuda()
    dev_s = torch.from_numpy(np.ascontiguousarray(scales).view(np.int16)).cuda()
    plain_c = torch.from_numpy(codes.copy())
    plain_s = torch.from_numpy(np.ascontiguousarray(scales).view(np.int16).copy())
    with Session(workspace_bytes=64 << 20, n_slots=2) as s2:
        s2.register(codes, scales, host=True)  # pinned host copy: fine
        s2.set_zero_copy(True)
        with pytest.raises(atsi.AtsiError, match="ATSI_E_INVALID"):
            s2.register_device(dev_c, dev_s, plain_c, plain_s)
        s2.set_zero_copy(False)
        s2.register_device(dev_c, dev_s, plain_c, plain_s)
        with pytest.raises(atsi.AtsiError, match="ATSI_E_INVALID"):
            s2.set_zero_copy(True)
        assert atsi.lib().atsi_set_zero_copy(s2.ctx, 2) == 1


def test_moe_decode_back_to_back(sess, cfg4):
    """Distinct single tokens queued back to back (decode with every expert
    resident) give bit for bit what each gives with a wait after it: the
    scratch that consecutive calls reuse is not raced."""
    import torch
    mask = list(sess.placement)
    for j in range(3):
        for e in range(cfg4.E):
            mask[cfg4.tids[j][e]] = 0
    sess.set_placement(mask)
    n = 24
    x = _dev(synth.activations(configs.MOE_LAYER.seed, 500, n, cfg4.H))
    ref = torch.empty((n, cfg4.H), dtype=torch.float16, device="cuda")
    for t in range(n):
        cfg4.layer(x[t:t + 1], ref[t:t + 1])
        sess.sync()
    for rep in range(2):
        y = torch.zeros_like(ref)
        for t in range(n):
            cfg4.layer(x[t:t + 1], y[t:t + 1])
        sess.sync()
        bad = (y != ref).any(dim=1).nonzero().flatten().tolist()
        assert not bad, f"pass {rep}: tokens {bad} differ from their one-at-a-time results"
