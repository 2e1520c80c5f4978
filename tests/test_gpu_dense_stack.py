"""GPU parity of a stack of 8B-shaped decoder layers run as a decode loop of
8 sequences with the 30 %-of-bytes host placement and the schedule-driven
prefetch, against the oracle's layer-by-layer chain."""
import numpy as np
import pytest

import oracle
import synth
from synth import configs
from tests.parity import check

pytestmark = pytest.mark.gpu

WL = configs.DENSE_STACK
N_LAYERS = 4  # the first layers of the 32-layer stack, full shape


@pytest.fixture(scope="module")
def stack():
    from paper_2607_10183_amd.session import Session
    s = Session(workspace_bytes=2 << 30, n_slots=12)
    shape = WL.dense
    W, tids = [], []
    for layer in range(N_LAYERS):
        w = {r: (synth.int4_codes(WL.seed, configs.dense_uid(layer, r), shape.kn(r)[1], shape.kn(r)[0]),
                 synth.group_scales(WL.seed, configs.dense_uid(layer, r), shape.kn(r)[1], shape.kn(r)[0]))
             for r in configs.ROLES}
        W.append(w)
        tids.append({r: s.register(*w[r], hbm=True, host=True) for r in configs.ROLES})
    yield s, W, tids
    s.close()


def _place(sess, tids, host_rows):
    mask = list(sess.placement)
    for layer, row in enumerate(host_rows):
        for j, r in enumerate(configs.ROLES):
            mask[tids[layer][r]] = int(row[j])
    sess.set_placement(mask)
    order = [tids[layer][r] for layer in range(len(tids)) for r in ("q", "k", "v", "o", "gate", "up", "down")]
    sess.set_schedule(order)


def _decode(sess, tids, hn, steps):
    """steps passes of the whole stack over the same 8 sequences (the hidden
    state carries over), one decoder_layer call per layer and the hidden state
    renormalised by its RMS after every layer."""
    shape = WL.dense
    h = _dev(hn)
    for _ in range(steps):
        for layer in range(len(tids)):
            sess.decoder_layer(tids[layer], h, shape.n_heads, shape.n_kv, shape.head_dim, 1e-6, renorm_out=True)
    sess.sync()
    return h


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def test_dense_stack_decode_parity(stack):
    sess, W, tids = stack
    shape = WL.dense
    host_rows = configs.dense_stack_host_mask()[:N_LAYERS]
    assert host_rows.sum() > 0
    _place(sess, tids, host_rows)
    hn = synth.activations(WL.seed, 1, WL.decode_m, shape.hidden)
    try:
        h = _decode(sess, tids, hn, steps=2)
    finally:
        sess.set_schedule([])
        _place(sess, tids, np.zeros_like(host_rows))
        sess.set_schedule([])
    ref, zeta = hn.astype(np.float64), None
    for _ in range(2):
        for layer in range(N_LAYERS):
            ref, zeta, _ = oracle.decoder_layer(ref, W[layer], shape.n_heads, shape.n_kv, shape.head_dim, 1e-6,
                                                h_zeta=zeta)
            ref, zeta = oracle.rmsnorm(ref, 1e-6, zeta)
    # free-running drift over 8 layer applications (each layer's stages are
    # checked teacher-forced elsewhere): a looser per-token norm
    check(h.cpu().numpy(), ref, zeta, name=f"{N_LAYERS}-layer stack, 2 steps, M={WL.decode_m}", rel_l2=3e-3)


def test_dense_stack_placement_invariance(stack):
    """The stack placement with prefetch and all-HBM give bit-identical states."""
    import torch
    sess, W, tids = stack
    hn = synth.activations(WL.seed, 2, WL.decode_m, WL.dense.hidden)
    host_rows = configs.dense_stack_host_mask()[:N_LAYERS]
    outs = []
    for rows in (np.zeros_like(host_rows), host_rows, np.ones_like(host_rows)):
        _place(sess, tids, rows)
        outs.append(_decode(sess, tids, hn, steps=1))
    sess.set_schedule([])
    _place(sess, tids, np.zeros_like(host_rows))
    sess.set_schedule([])
    for o in outs[1:]:
        assert torch.equal(outs[0], o)


def test_solver_placement_runs_bit_identical(stack):
    """Alg. 1 end to end: per-tensor resident kernel times measured on the GPU
    (one per role), gains r = copy time over a nominal 50 GB/s link minus that
    time, the solver's mask for 30 % of the bytes on host; the stack runs with
    that mask and gives the all-HBM bits."""
    import torch
    from paper_2607_10183_amd import placement
    sess, W, tids = stack
    shape = WL.dense
    order = [tids[layer][r] for layer in range(N_LAYERS) for r in configs.ROLES]
    sizes = [configs.qbytes(*sess.shapes[t]) for t in order]
    t_role = {r: placement.kernel_seconds(sess, tids[0][r], WL.decode_m, reps=4) for r in configs.ROLES}
    assert all(0 < v < 1e-3 for v in t_role.values())
    t_gpu = [t_role[r] for _ in range(N_LAYERS) for r in configs.ROLES]
    host, obj = placement.solve(sizes, t_gpu, 50e9, 0.7 * sum(sizes))
    assert sum(s for s, h in zip(sizes, host) if not h) <= 0.7 * sum(sizes) + (1 << 20)
    assert 0 < sum(host) < len(host)
    hn = synth.activations(WL.seed, 3, WL.decode_m, shape.hidden)
    ref = _decode(sess, tids, hn, steps=1)
    mask = list(sess.placement)
    for t, h in zip(order, host):
        mask[t] = int(h)
    sess.set_placement(mask)
    sess.set_schedule(order)
    try:
        got = _decode(sess, tids, hn, steps=1)
    finally:
        sess.set_schedule([])
        sess.set_placement([0] * len(mask))
    assert torch.equal(ref, got)
