"""The allocation-free SwiGLU entry point (atsi_ffn_swiglu_noalloc) against the
workspace one (atsi_ffn_swiglu), through the C ABI: two calls in a row, the
second smaller, give the same bits where both take the same kernels; a
512-token chunk (whose down projection runs unsplit here) stays within the
oracle's bounds; and a size beyond the static scratch is refused."""
import numpy as np
import pytest

import oracle
import synth
from tests.parity import check

pytestmark = pytest.mark.gpu


def _qt(seed, uid, N, K):
    return synth.int4_codes(seed, uid, N, K), synth.group_scales(seed, uid, N, K)


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _run(s, fn, tids, x, H):
    import torch
    M = x.shape[0]
    with torch.cuda.stream(s.cs):
        y = torch.full((M, H), float("nan"), dtype=torch.float16, device="cuda")
    s._wait_torch()
    fn(s.ctx, *tids, x.data_ptr(), M, y.data_ptr())
    s._torch_waits()
    return y


def test_noalloc_matches_workspace_entry_point():
    import torch
    from paper_2607_10183_amd import atsi
    from paper_2607_10183_amd.session import Session
    H, I = 2048, 768
    W = [_qt(95, 1, I, H), _qt(95, 2, I, H), _qt(95, 3, H, I)]
    with Session(workspace_bytes=64 << 20, n_slots=2) as s:
        tids = [s.register(*w) for w in W]
        for M in (64, 5, 1):  # 128-row GEMM, batched decode, GEMV; each smaller than the last
            x = _dev(synth.activations(95, 10 + M, M, H))
            want = _run(s, atsi.atsi_ffn_swiglu, tids, x, H)
            got = _run(s, atsi.atsi_ffn_swiglu_noalloc, tids, x, H)
            s.sync()
            assert torch.equal(want, got), M
        with pytest.raises(atsi.AtsiError, match="ATSI_E_WORKSPACE"):
            x = _dev(synth.activations(95, 99, 11000, H))
            _run(s, atsi.atsi_ffn_swiglu_noalloc, tids, x, H)


def test_noalloc_prefill_chunk_and_host_tensors():
    """The 8B-shaped FFN at 512 tokens, then at 3 with gate and down streamed
    from host: against the oracle, and the second call against the workspace
    entry point bit for bit."""
    import torch
    from paper_2607_10183_amd import atsi
    from paper_2607_10183_amd.session import Session
    H, I = 4096, 14336
    W = [_qt(96, 1, I, H), _qt(96, 2, I, H), _qt(96, 3, H, I)]
    with Session(workspace_bytes=256 << 20, n_slots=3) as s:
        tids = [s.register(*w, hbm=True, host=True) for w in W]
        xn = synth.activations(96, 1, 512, H)
        y = _run(s, atsi.atsi_ffn_swiglu_noalloc, tids, _dev(xn), H).cpu().numpy()
        s.sync()
        rows = np.arange(0, 512, 16)
        ref, zeta, _ = oracle.swiglu_ffn(xn[rows], *W)
        check(y[rows], ref, zeta, name="noalloc FFN, 512 tokens", rel_l2=1e-2)
        s.set_placement([1, 0, 1])
        x3 = _dev(synth.activations(96, 2, 3, H))
        got = _run(s, atsi.atsi_ffn_swiglu_noalloc, tids, x3, H)
        want = _run(s, atsi.atsi_ffn_swiglu, tids, x3, H)
        s.sync()
        s.set_placement([0, 0, 0])
        assert torch.equal(want, got)
