"""The boundary's error statuses and the streaming engine's slot reuse, on the
GPU through the C ABI: every status a call can return is produced by a call
that should return it, nothing is launched for a rejected call, and an
asynchronous failure is latched and returned by atsi_sync and later calls."""
import ctypes

import numpy as np
import pytest

import synth
from paper_2607_10183_amd import atsi

pytestmark = pytest.mark.gpu


def _qt(seed, uid, N, K):
    return synth.int4_codes(seed, uid, N, K), synth.group_scales(seed, uid, N, K)


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.fixture(scope="module")
def sess():
    from paper_2607_10183_amd.session import Session
    s = Session(workspace_bytes=64 << 20, n_slots=3)
    yield s
    s.close()


def _status(fn, *a):
    with pytest.raises(atsi.AtsiError) as ei:
        fn(*a)
    return atsi.STATUS[ei.value.status]


def test_status_unknown_tensor(sess):
    import torch
    x = torch.zeros((1, 256), dtype=torch.float16, device="cuda")
    y = torch.zeros((1, 64), dtype=torch.float16, device="cuda")
    assert _status(atsi.atsi_linear, sess.ctx, 12345, x.data_ptr(), 1, y.data_ptr()) == "ATSI_E_UNKNOWN_TENSOR"
    assert _status(atsi.atsi_prefetch, sess.ctx, -1) == "ATSI_E_UNKNOWN_TENSOR"
    assert _status(atsi.atsi_set_schedule, sess.ctx, [0, 999]) == "ATSI_E_UNKNOWN_TENSOR"


def test_status_shape(sess):
    import torch
    codes, scales = _qt(90, 1, 64, 256)
    tid = sess.register(codes, scales)
    # K not a multiple of 32, group other than 32
    assert _status(atsi.atsi_tensor_register, sess.ctx, 48, 64, 1 << 20, 1 << 20) == "ATSI_E_SHAPE"
    assert _status(atsi.atsi_tensor_register, sess.ctx, 256, 64, 1 << 20, 1 << 20, 0, 0, 64) == "ATSI_E_SHAPE"
    x = torch.zeros((1, 256), dtype=torch.float16, device="cuda")
    y = torch.zeros((1, 64), dtype=torch.float16, device="cuda")
    for M in (0, 65537):
        assert _status(atsi.atsi_linear, sess.ctx, tid, x.data_ptr(), M, y.data_ptr()) == "ATSI_E_SHAPE"
    # an FFN whose down projection does not match gate/up
    t2 = sess.register(*_qt(90, 2, 64, 256))
    assert _status(atsi.atsi_ffn_swiglu, sess.ctx, tid, tid, t2, x.data_ptr(), 1, y.data_ptr()) == "ATSI_E_SHAPE"
    assert _status(atsi.atsi_rmsnorm, sess.ctx, x.data_ptr(), 1, 12, 1e-6, x.data_ptr()) == "ATSI_E_SHAPE"


def test_status_invalid(sess):
    import torch
    tid = sess.register(*_qt(90, 3, 64, 256))
    x = torch.zeros((2, 256), dtype=torch.float16, device="cuda")
    y = torch.zeros((2, 64), dtype=torch.float16, device="cuda")
    # misaligned and NULL activations
    assert _status(atsi.atsi_linear, sess.ctx, tid, x.data_ptr() + 2, 1, y.data_ptr()) == "ATSI_E_INVALID"
    assert _status(atsi.atsi_linear, sess.ctx, tid, 0, 1, y.data_ptr()) == "ATSI_E_INVALID"
    assert _status(atsi.atsi_set_debug, sess.ctx, 4) == "ATSI_E_INVALID"
    assert _status(atsi.atsi_set_placement, sess.ctx, [0]) == "ATSI_E_INVALID"  # wrong length


def test_status_no_copy(sess):
    codes, scales = _qt(90, 4, 64, 256)
    tid = sess.register(codes, scales, hbm=True, host=False)
    mask = list(sess.placement)
    mask[tid] = 1
    assert _status(atsi.atsi_set_placement, sess.ctx, mask) == "ATSI_E_NO_COPY"
    assert _status(atsi.atsi_tensor_register, sess.ctx, 256, 64) == "ATSI_E_NO_COPY"
    # the placement was left as it was
    mask[tid] = 0
    sess.set_placement(mask)


def test_status_workspace():
    """A workspace too small for the call's scratch, or for the slots of a host tensor."""
    import torch
    from paper_2607_10183_amd.session import Session
    with Session(workspace_bytes=1 << 20, n_slots=2) as s:
        H, I, M = 1024, 4096, 128
        g, u, d = s.register(*_qt(90, 5, I, H)), s.register(*_qt(90, 6, I, H)), s.register(*_qt(90, 7, H, I))
        x = _dev(synth.activations(90, 8, M, H))
        y = torch.empty((M, H), dtype=torch.float16, device="cuda")
        assert _status(atsi.atsi_ffn_swiglu, s.ctx, g, u, d, x.data_ptr(), M, y.data_ptr()) == "ATSI_E_WORKSPACE"
        # two slots of a 2.3 MB host tensor do not fit in 1 MiB; the placement stays
        big = s.register(*_qt(90, 9, 1024, 4096), hbm=True, host=True)
        mask = list(s.placement)
        mask[big] = 1
        assert _status(atsi.atsi_set_placement, s.ctx, mask) == "ATSI_E_WORKSPACE"
        y1 = torch.empty((1, 1024), dtype=torch.float16, device="cuda")
        s.linear(big, _dev(synth.activations(90, 10, 1, 4096)), y1)
        s.sync()
        assert s.stats()["h2d_bytes"] == 0


def test_status_state_without_pinned_counts():
    """An MoE call with experts streamed on the copy path needs the pinned
    counts buffer; a context created without one refuses the call up front."""
    import torch
    E, H, I, k = 16, 256, 96, 4
    cs, ts = torch.cuda.Stream(), torch.cuda.Stream()
    ws = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")
    ctx = atsi.atsi_create(0, cs.cuda_stream, ts.cuda_stream, 0, ws.data_ptr(), ws.numel(), 0, 4)
    keep = []
    try:
        tids = [[], [], []]
        for e in range(E):
            for j, (n, kk) in enumerate(((I, H), (I, H), (H, I))):
                c, sc = _qt(91, 10 * e + j, n, kk)
                dc = torch.from_numpy(c).cuda()
                ds = torch.from_numpy(np.ascontiguousarray(sc).view(np.int16)).cuda()
                hb = torch.empty(c.nbytes + sc.nbytes, dtype=torch.uint8).pin_memory()
                hb.numpy()[:c.nbytes] = c.reshape(-1)
                hb.numpy()[c.nbytes:] = np.ascontiguousarray(sc).view(np.uint8).reshape(-1)
                keep += [dc, ds, hb]
                tids[j].append(atsi.atsi_tensor_register(ctx, kk, n, dc.data_ptr(), ds.data_ptr(), hb.data_ptr(),
                                                         hb.data_ptr() + c.nbytes))
        wr = _dev(synth.router_weights(91, 2, H, E))
        ids = [(ctypes.c_int32 * E)(*t) for t in tids]
        moe = atsi.atsi_moe(E, k, H, I, wr.data_ptr(), None, *[ctypes.cast(a, ctypes.POINTER(ctypes.c_int32))
                                                                for a in ids])
        x = _dev(synth.activations(91, 3, 8, H))
        y = torch.empty((8, H), dtype=torch.float16, device="cuda")
        torch.cuda.synchronize()
        atsi.atsi_moe_ffn(ctx, moe, x.data_ptr(), 8, y.data_ptr())  # all resident: fine
        mask = [0] * (3 * E)
        mask[tids[0][3]] = 1
        atsi.atsi_set_placement(ctx, mask)
        assert _status(atsi.atsi_moe_ffn, ctx, moe, x.data_ptr(), 8, y.data_ptr()) == "ATSI_E_STATE"
        atsi.atsi_sync(ctx)
    finally:
        atsi.atsi_destroy(ctx)


def test_latched_async_error_reported_by_sync():
    """A failure found on the GPU after the call returned (here: the error flag
    of the single-launch decode layer's bounded barrier, set from the host
    after a normal launch, as a barrier that ran out of polls would set it) is
    returned by atsi_sync and by every later call of the context."""
    import os
    import torch
    from paper_2607_10183_amd.session import Session
    from synth import configs
    old = os.environ.get("ATSI_FUSED_DECODE_LAYER")
    os.environ["ATSI_FUSED_DECODE_LAYER"] = "1"
    ws_bytes = 1 << 28
    try:
        s = Session(workspace_bytes=ws_bytes, n_slots=2)
    finally:
        if old is None:
            del os.environ["ATSI_FUSED_DECODE_LAYER"]
        else:
            os.environ["ATSI_FUSED_DECODE_LAYER"] = old
    try:
        shape = configs.DenseShape()
        tids = {r: s.register(*_qt(92, configs.dense_uid(0, r), shape.kn(r)[1], shape.kn(r)[0]))
                for r in configs.ROLES}
        h = _dev(synth.activations(92, 1, 1, shape.hidden))
        s.decoder_layer(tids, h, shape.n_heads, shape.n_kv, shape.head_dim)
        s.sync()  # a normal launch: no error
        s.decoder_layer(tids, h, shape.n_heads, shape.n_kv, shape.head_dim)
        # the barrier words sit at the top of the workspace (353 words rounded
        # up to 1536 bytes); the error flag is word 320 of them
        with torch.cuda.stream(s.cs):
            s.ws[ws_bytes - 1536 + 4 * 320:ws_bytes - 1536 + 4 * 321] = torch.tensor([1, 0, 0, 0], dtype=torch.uint8,
                                                                                      device="cuda")
        with pytest.raises(atsi.AtsiError, match="ATSI_E_HIP.*barrier"):
            s.sync()
        x = torch.zeros((1, shape.hidden), dtype=torch.float16, device="cuda")
        with pytest.raises(atsi.AtsiError, match="ATSI_E_HIP"):
            s.linear(tids["q"], x)
        with pytest.raises(atsi.AtsiError, match="ATSI_E_HIP"):
            s.sync()
    finally:
        s.close()


def test_eviction_of_an_in_flight_prefetch():
    """Three slots; a schedule of a later call's tensors fills all but one of
    them with prefetched copies; then a launch needs two other host tensors on
    demand, so the engine drops a prefetched copy that may still be in flight
    and reuses its slot.  Under poisoned slots the output must equal the
    all-HBM bits (a late prefetched copy landing on the reused slot would not)."""
    import torch
    from paper_2607_10183_amd.session import Session
    H, I, M = 4096, 1024, 1
    with Session(workspace_bytes=256 << 20, n_slots=3) as s:
        gate, up = s.register(*_qt(93, 1, I, H), hbm=True, host=True), s.register(*_qt(93, 2, I, H), hbm=True, host=True)
        later = [s.register(*_qt(93, 3 + i, I, H), hbm=True, host=True) for i in range(2)]
        x = _dev(synth.activations(93, 9, M, H))
        ref = s.gate_up(gate, up, x)
        s.sync()
        s.set_placement([1] * len(s.placement))
        s.set_debug(poison=True)
        try:
            for rep in range(4):
                s.set_schedule(later)
                atsi.atsi_prefetch(s.ctx, later[0])
                got = s.gate_up(gate, up, x)
                s.sync()
                assert torch.equal(got, ref), rep
                s.set_schedule([])
        finally:
            s.set_debug()
            s.set_schedule([])
            s.set_placement([0] * len(s.placement))
