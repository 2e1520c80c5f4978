"""GPU parity of the hybrid CPU-GPU execution (Sec. 4.3-4.4): host-placed
tensors assigned to the CPU backend run there (activations staged through
pinned memory), the rest on the GPU, in every mix the layer allows, each
stage against the oracle at the same bounds as the all-GPU path; plus the
error paths and the per-tensor timing records (Alg. 3's snapshots)."""
import math

import numpy as np
import pytest

import oracle
import synth
from synth import configs
from tests import stages
from tests.parity import bits16, check, tight_eps

pytestmark = pytest.mark.gpu

THREADS = 8


@pytest.fixture(scope="module")
def sess():
    from paper_2607_10183_amd.session import Session
    s = Session(workspace_bytes=1 << 30, n_slots=4)
    s.attach_cpu(THREADS, staging_bytes=192 << 20)
    yield s
    s.close()


def _qt(seed, uid, N, K):
    return synth.int4_codes(seed, uid, N, K), synth.group_scales(seed, uid, N, K)


def _dev(xn):
    import torch
    return torch.from_numpy(np.ascontiguousarray(xn)).cuda()


def _host_cpu(sess, tids):
    """Place `tids` on the host and run them on the CPU backend."""
    mask = list(sess.placement)
    for t in tids:
        mask[t] = 1
    sess.set_placement(mask)
    on_cpu = list(sess.backends)
    for t in tids:
        on_cpu[t] = 1
    sess.set_backends(on_cpu)


def _reset(sess):
    sess.set_backends([0] * len(sess.shapes))
    sess.set_placement([0] * len(sess.shapes))


@pytest.mark.parametrize("K,N,M", [(4096, 4096, 1), (4096, 1024, 3), (640, 77, 16), (4096, 14336, 4),
                                   (2048, 768, 300)])
def test_cpu_linear_parity(sess, K, N, M):
    w = _qt(91, K + N, N, K)
    tid = sess.register(*w, hbm=True, host=True)
    _host_cpu(sess, [tid])
    sess.stats(reset=True)
    xn = synth.activations(91, M, M, K)
    y = sess.linear(tid, _dev(xn)).cpu().numpy()
    sess.sync()
    st = sess.stats(reset=True)
    _reset(sess)
    assert st["h2d_bytes"] == 0 and st["host_reads"] == 0, "a CPU-run tensor was copied to the GPU"
    ref, zeta = oracle.linear(xn, *w)
    check(y, ref, zeta, name=f"cpu linear {K}x{N} M={M}", tight=tight_eps(K))


@pytest.mark.parametrize("H,I,M", [(256, 96, 1), (4096, 14336, 1), (512, 160, 77)])
def test_cpu_ffn_parity(sess, H, I, M):
    gate, up, down = _qt(92, H + 1, I, H), _qt(92, H + 2, I, H), _qt(92, H + 3, H, I)
    t = [sess.register(*w, hbm=True, host=True) for w in (gate, up, down)]
    _host_cpu(sess, t)
    xn = synth.activations(92, M, M, H)
    y = sess.ffn(*t, _dev(xn)).cpu().numpy()
    sess.sync()
    _reset(sess)
    ref, zeta, _ = oracle.swiglu_ffn(xn, gate, up, down)
    check(y, ref, zeta, name=f"cpu ffn H={H} I={I} M={M}", rel_l2=stages.COMPOSITE_ROW_L2)


SMALL = configs.DenseShape(hidden=256, n_heads=4, n_kv=2, head_dim=64, inter=96)

# which roles run on the CPU (all are host-placed); q alone and k+v make the
# fused q/k/v launch mixed, its GPU part overlapping the CPU part
MIXES = [("q", "k", "v", "o", "gate", "up", "down"), ("q",), ("k", "v"), ("o", "down"), ("gate", "up"),
         ("q", "o", "gate", "up"), ()]


@pytest.mark.parametrize("shape,M", [(SMALL, 1), (SMALL, 5), (configs.DenseShape(), 1), (configs.DenseShape(), 8)])
@pytest.mark.parametrize("mix", range(len(MIXES)))
def test_hybrid_layer_parity(sess, shape, M, mix):
    """Every stage of the layer teacher-forced against the oracle, whichever
    backend ran it, and the whole layer against the oracle layer."""
    import torch
    roles = MIXES[mix]
    W = {r: _qt(93, configs.dense_uid(0, r), shape.kn(r)[1], shape.kn(r)[0]) for r in configs.ROLES}
    tids = {r: sess.register(*W[r], hbm=True, host=True) for r in configs.ROLES}
    mask = list(sess.placement)
    for r in configs.ROLES:
        mask[tids[r]] = 1
    sess.set_placement(mask)
    on_cpu = [0] * len(sess.shapes)
    for r in roles:
        on_cpu[tids[r]] = 1
    sess.set_backends(on_cpu)
    hn = synth.activations(93, 3000 + M, M, shape.hidden)
    h = _dev(hn)
    q_out = torch.empty((M, shape.n_heads * shape.head_dim), dtype=torch.float16, device="cuda")
    k_out = torch.empty((M, shape.n_kv * shape.head_dim), dtype=torch.float16, device="cuda")
    _, dbg = sess.decoder_layer(tids, h, shape.n_heads, shape.n_kv, shape.head_dim, 1e-6, q_out, k_out, debug=True)
    sess.sync()
    _reset(sess)
    name = f"hybrid layer H={shape.hidden} M={M} cpu={roles}"
    stages.attention_stages(W, shape.n_heads, shape.n_kv, shape.head_dim, hn, q_out, k_out, dbg["attn"],
                            dbg["h_attn"], name)
    stages.ffn_stages(W, dbg["h_attn"], dbg["act"], h, name)
    ref, zeta, _ = oracle.decoder_layer(hn, W, shape.n_heads, shape.n_kv, shape.head_dim, 1e-6)
    check(h.cpu().numpy(), ref, zeta, name=name, rel_l2=stages.COMPOSITE_ROW_L2)


def test_hybrid_layer_exact_inputs_bitexact(sess):
    """+-1 inputs, eps = 0 and scales 2^-6 (exact sums on both backends): the
    CPU-run q, k, grouped-query expansion and O + residual are bit-exact."""
    import torch
    shape = configs.DenseShape()
    hd = shape.head_dim
    M = 4
    W = {r: (synth.int4_codes(94, configs.dense_uid(0, r), shape.kn(r)[1], shape.kn(r)[0]),
             synth.exact_scales(shape.kn(r)[1], shape.kn(r)[0])) for r in configs.ROLES}
    tids = {r: sess.register(*W[r], hbm=True, host=True) for r in configs.ROLES}
    _host_cpu(sess, [tids[r] for r in ("q", "v", "o")])
    hn = synth.sign_activations(94, M, M, shape.hidden)
    h = _dev(hn)
    q_out = torch.empty((M, shape.n_heads * hd), dtype=torch.float16, device="cuda")
    k_out = torch.empty((M, shape.n_kv * hd), dtype=torch.float16, device="cuda")
    _, dbg = sess.decoder_layer(tids, h, shape.n_heads, shape.n_kv, hd, 0.0, q_out, k_out, debug=True)
    sess.sync()
    _reset(sess)
    x = hn.astype(np.float64)
    q, _ = oracle.linear(x, *W["q"])
    k, _ = oracle.linear(x, *W["k"])
    v, _ = oracle.linear(x, *W["v"])
    assert np.array_equal(bits16(q_out), bits16(q)), "q (CPU)"
    assert np.array_equal(bits16(k_out), bits16(k)), "k (GPU)"
    attn = oracle.gqa_stub(v.astype(np.float16), shape.n_heads, shape.n_kv, hd)
    assert np.array_equal(bits16(dbg["attn"]), bits16(attn)), "grouped-query expansion (CPU)"
    o, _ = oracle.linear(attn.astype(np.float64), *W["o"])
    assert np.array_equal(bits16(dbg["h_attn"]), bits16(x + o)), "O + residual (CPU)"


def test_hybrid_error_paths(sess):
    from paper_2607_10183_amd import atsi
    shape = SMALL
    W = {r: _qt(95, configs.dense_uid(0, r), shape.kn(r)[1], shape.kn(r)[0]) for r in configs.ROLES}
    tids = {r: sess.register(*W[r], hbm=True, host=True) for r in configs.ROLES}
    n = len(sess.shapes)
    # an HBM-placed tensor cannot run on the CPU
    on_cpu = [0] * n
    on_cpu[tids["q"]] = 1
    with pytest.raises(atsi.AtsiError, match="HBM"):
        sess.set_backends(on_cpu)
    # gate and up of one launch must share a backend
    _host_cpu(sess, [tids["gate"]])
    h = _dev(synth.activations(95, 1, 1, shape.hidden))
    with pytest.raises(atsi.AtsiError, match="share a backend"):
        sess.decoder_layer(tids, h, shape.n_heads, shape.n_kv, shape.head_dim)
    # the allocation-free entry point runs nothing on the CPU
    _host_cpu(sess, [tids["gate"], tids["up"]])
    y = _dev(np.zeros((1, shape.hidden), np.float16))
    with pytest.raises(atsi.AtsiError, match="CPU backend"):
        atsi.atsi_ffn_swiglu_noalloc(sess.ctx, tids["gate"], tids["up"], tids["down"], h.data_ptr(), 1, y.data_ptr())
    # staging too small for the launch
    from paper_2607_10183_amd.session import Session
    with Session(workspace_bytes=64 << 20, n_slots=2) as s2:
        s2.attach_cpu(2, staging_bytes=4096)
        t = s2.register(*_qt(95, 9, 512, 4096), hbm=True, host=True)
        s2.set_placement([1])
        s2.set_backends([1])
        with pytest.raises(atsi.AtsiError, match="staging"):
            s2.linear(t, _dev(synth.activations(95, 2, 8, 4096)))
        # detaching the backend while a tensor is assigned to it
        with pytest.raises(atsi.AtsiError):
            atsi.atsi_set_cpu_backend(s2.ctx, 0, 0, 0)
    sess.sync()
    _reset(sess)


def test_placement_to_hbm_resets_backend(sess):
    t = sess.register(*_qt(96, 1, 64, 256), hbm=True, host=True)
    _host_cpu(sess, [t])
    assert sess.backends[t] == 1
    sess.set_placement([0] * len(sess.shapes))
    assert sess.backends[t] == 0
    sess.stats(reset=True)
    y = sess.linear(t, _dev(synth.activations(96, 1, 1, 256)))
    sess.sync()
    assert sess.stats(reset=True)["h2d_bytes"] == 0


def test_timings_record_each_backend(sess):
    """Timing on: a layer with a CPU-run o and down, streamed (promoted) q, k,
    v, gate and up: each tensor gets the figures of what it did, all finite and
    positive, the others NaN."""
    import torch
    shape = configs.DenseShape()
    W = {r: _qt(97, configs.dense_uid(0, r), shape.kn(r)[1], shape.kn(r)[0]) for r in configs.ROLES}
    tids = {r: sess.register(*W[r], hbm=True, host=True) for r in configs.ROLES}
    _host_cpu(sess, [tids["o"], tids["down"]])
    mask = list(sess.placement)
    for r in configs.ROLES:
        mask[tids[r]] = 1
    sess.set_placement(mask)
    sess.set_timing(True)
    h = _dev(synth.activations(97, 1, 1, shape.hidden))
    for _ in range(3):
        sess.decoder_layer(tids, h, shape.n_heads, shape.n_kv, shape.head_dim, renorm_out=True)
    tm = sess.timings()
    sess.set_timing(False)
    _reset(sess)
    for r in configs.ROLES:
        t = tm[tids[r]]
        if r in ("o", "down"):
            assert t["t_cpu"] > 0 and t["d2h"] > 0 and t["h2d"] > 0, (r, t)
            assert math.isnan(t["t_gpu"]) and math.isnan(t["w"]), (r, t)
        else:
            assert t["t_gpu"] > 0 and t["w"] > 0, (r, t)
            assert math.isnan(t["t_cpu"]), (r, t)
    # a 29 MB copy at under 64 GB/s takes at least 0.45 ms
    assert tm[tids["gate"]]["w"] > 0.45e-3


def test_controller_rebuilds_runtime(sess):
    """Alg. 3's loop on the GPU: the controller's decisions follow the
    measured load (synthetic timing reads), BuildRuntime applies each new
    assignment to the library, and the layer computed under it still matches
    the oracle."""
    import torch
    from paper_2607_10183_amd import hybrid
    shape = configs.DenseShape()
    W = {r: _qt(98, configs.dense_uid(0, r), shape.kn(r)[1], shape.kn(r)[0]) for r in configs.ROLES}
    tids = {r: sess.register(*W[r], hbm=True, host=True) for r in configs.ROLES}
    units = hybrid.dense_units([tids])
    on_gpu = [1, 1, 1, 0, 0, 0]  # o, gate+up and down on the host
    sess.set_placement(hybrid.host_mask(sess, units, [1 - g for g in on_gpu]))
    model = {"t_gpu": [8e-6, 2e-6, 2e-6, 7e-6, 15e-6, 13e-6], "t_cpu": [2e-4, 1e-4, 1e-4, 2.5e-4, 6e-4, 4e-4],
             "w": [1.7e-4, 4e-5, 4e-5, 1.7e-4, 1.2e-3, 6e-4]}
    ctrl = hybrid.Controller(sess, units, on_gpu, hybrid.Snapshotter(units, model, model))
    nan = float("nan")
    n = len(sess.shapes)

    def reads(cpu_scale):
        tm = [{"t_gpu": nan, "t_cpu": nan, "d2h": nan, "h2d": nan, "w": nan} for _ in range(n)]
        for (_, roles, ts), tg, tc in zip(units, model["t_gpu"], model["t_cpu"]):
            for t in ts:
                tm[t].update(t_gpu=tg / len(ts), t_cpu=tc * cpu_scale / len(ts), d2h=0.0, h2d=0.0)
        return tm

    def run_and_check(tag):
        hn = synth.activations(98, 5, 1, shape.hidden)
        h = _dev(hn)
        q_out = torch.empty((1, shape.n_heads * shape.head_dim), dtype=torch.float16, device="cuda")
        k_out = torch.empty((1, shape.n_kv * shape.head_dim), dtype=torch.float16, device="cuda")
        _, dbg = sess.decoder_layer(tids, h, shape.n_heads, shape.n_kv, shape.head_dim, 1e-6, q_out, k_out,
                                    debug=True)
        sess.sync()
        stages.attention_stages(W, shape.n_heads, shape.n_kv, shape.head_dim, hn, q_out, k_out, dbg["attn"],
                                dbg["h_attn"], tag)
        stages.ffn_stages(W, dbg["h_attn"], dbg["act"], h, tag)

    try:
        did, _ = ctrl.step(0.0, 0.01, reads(1.0))
        assert did and ctrl.rb is not None
        first = list(ctrl.rb)
        assert sess.backends == hybrid.cpu_mask(sess, units, [1 - v for v in first])
        run_and_check(f"controller first assignment {first}")
        did, _ = ctrl.step(0.02, 0.01, reads(1.0))          # nothing changed
        assert not did
        did, _ = ctrl.step(0.03, 0.01, reads(50.0))         # CPU 50x slower, but within tau = 5 x 10 ms
        assert not did
        did, d = ctrl.step(0.2, 0.01, reads(50.0))          # after tau: re-schedule
        assert did and d > 0.15
        second = list(ctrl.rb)
        assert sum(second) >= sum(first), "a slower CPU must not move work to the CPU"
        assert sess.backends == hybrid.cpu_mask(sess, units, [1 - v for v in second])
        run_and_check(f"controller loaded assignment {second}")
    finally:
        ctrl.close()
        _reset(sess)
