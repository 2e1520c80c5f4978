"""GPU parity of the quantised linear layer (decode GEMV and prefill GEMM)
against the fp64 oracle, through the C ABI."""
import numpy as np
import pytest

import oracle
import synth
from tests.parity import bits16, check, tight_eps

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sess():
    from paper_2607_10183_amd.session import Session
    s = Session(workspace_bytes=512 << 20, n_slots=4)
    yield s
    s.close()


def _x(seed, uid, M, K, exact=False):
    import torch
    xn = synth.exact_activations(seed, uid, M, K) if exact else synth.activations(seed, uid, M, K)
    return xn, torch.from_numpy(xn).cuda()


@pytest.mark.parametrize("host", [False, True])
def test_unpack_bitexact(sess, host):
    K, N = 4096, 300
    codes = synth.int4_codes(61, 1, N, K)
    scales = synth.group_scales(61, 1, N, K)
    tid = sess.register(codes, scales, hbm=not host, host=host)
    q = sess.unpack(tid)
    sess.sync()
    assert np.array_equal(q.cpu().numpy(), oracle.unpack_codes(codes))


def assert_doubles(y2, y1):
    """y(2x) is 2 y(x) bit for bit wherever the fp16 output is normal: every
    product and fp32 partial sum scales exactly, and so does the final
    rounding in the normal range.  In the subnormal output range the rounding
    grid is absolute (2^-24), so there the two may differ by one step."""
    a = np.ascontiguousarray(y2.detach().cpu().numpy())
    b = (2 * y1.float()).half().cpu().numpy()
    normal = np.abs(y1.float().cpu().numpy()) >= 2.0 ** -13
    assert np.array_equal(a.view(np.uint16)[normal], b.view(np.uint16)[normal])
    assert np.all(np.abs(a[~normal].astype(np.float64) - b[~normal].astype(np.float64)) <= 2.0 ** -24)


EXACT_SHAPES = [  # (K, N, M): GEMV for M = 1, the batched-decode kernel for 2 <= M <= 16 when
    # K % 128 == 0 (else GEMV launches up to M = 4, GEMM above), GEMM for larger M; ragged N and M
    (32, 7, 1), (96, 33, 3), (768, 2048, 1), (4096, 1000, 4), (14336, 257, 2), (4096, 4096, 1),
    (4096, 1000, 5), (768, 300, 64), (4096, 520, 100), (14336, 130, 512), (2048, 4096, 16), (96, 65, 129),
    (4096, 700, 8), (8192, 300, 7), (14336, 257, 8), (14336, 130, 6), (256, 96, 8),
    (160, 70, 2), (224, 50, 4), (96, 40, 6), (128, 20, 16), (384, 17, 3),
    # 512-row-tile prefill GEMM (taken from 256 rows and 192 tiles of 128 outputs):
    # ragged M, a K step left half full, two row tiles
    (96, 24576, 300), (64, 24576, 520),
    # the same with K split into ranges (fewer than 192 tiles): 6 ranges of the
    # 4096 x 4096 tile grid, 8 ranges with a half-full last step and ragged N,
    # two row tiles, and 8 ranges over 14336 inputs (the ragged N = 130 above)
    (4096, 4096, 512), (4128, 600, 512), (8192, 1000, 700),
]


@pytest.mark.parametrize("K,N,M", EXACT_SHAPES)
def test_exact_arithmetic_bitexact(sess, K, N, M):
    """Scales 2^-6 and activations in {-4..4}/4 make every fp32 partial sum
    exact, so the fp16 output must equal the nearest-even rounding of the exact
    result, bit for bit."""
    codes = synth.int4_codes(62, K * 7 + N, N, K)
    scales = synth.exact_scales(N, K)
    xn, x = _x(62, M, M, K, exact=True)
    tid = sess.register(codes, scales)
    y = sess.linear(tid, x)
    sess.sync()
    ref, _ = oracle.linear(xn, codes, scales)
    assert np.array_equal(bits16(y), bits16(ref))


RANDOM_SHAPES = [  # linear4096 (decode 1, batch 16) and the dense-layer tensors
    (4096, 4096, 1), (4096, 4096, 16), (4096, 1024, 1), (4096, 14336, 1), (14336, 4096, 1),
    (4096, 4096, 2), (4096, 1024, 4), (4096, 1024, 512), (4096, 14336, 512), (14336, 4096, 512),
    (4096, 4096, 3), (2048, 768, 37), (4096, 14336, 8), (14336, 4096, 8), (4096, 6144, 5),
    (512, 24576, 600), (4096, 24576, 257),  # 512-row-tile GEMM
]


@pytest.mark.parametrize("K,N,M", RANDOM_SHAPES)
def test_random_parity(sess, K, N, M):
    codes = synth.int4_codes(63, K + N, N, K)
    scales = synth.group_scales(63, K + N, N, K)
    xn, x = _x(63, M, M, K)
    tid = sess.register(codes, scales)
    y = sess.linear(tid, x).cpu().numpy()
    sess.sync()
    rows = np.arange(N) if N * M <= 4096 * 512 else synth.permutation(63, 9, N)[:2048]
    ref, zeta = oracle.linear(xn, codes[rows], scales[rows])
    # exact products on the GEMV and the batched-decode kernel; fp16-rounded
    # dequantised weights on the MFMA GEMM (every K here is a multiple of 128)
    check(y[:, rows], ref, zeta, name=f"linear K={K} N={N} M={M}", tight=tight_eps(K, mfma=M > 16))


@pytest.mark.parametrize("M", [1, 3, 16, 200])
def test_scaling_by_two_and_determinism(sess, M):
    import torch
    K, N = 4096, 777
    codes = synth.int4_codes(64, 1, N, K)
    scales = synth.group_scales(64, 1, N, K)
    xn, x = _x(64, M, M, K)
    tid = sess.register(codes, scales)
    y1 = sess.linear(tid, x)
    y2 = sess.linear(tid, (2 * x).contiguous())
    y3 = sess.linear(tid, x)
    sess.sync()
    assert torch.equal(y1, y3)
    assert_doubles(y2, y1)


@pytest.mark.parametrize("K,N,M", [(128, 24576, 300), (4096, 4096, 512)])
def test_wide_gemm_scaling_by_two_and_determinism(sess, K, N, M):
    """The 512-row-tile GEMM, with one K range and with six: y(2x) equals
    2 y(x) (exact products, sums scaled exactly) and repeated calls are
    bit-identical (the ranges are added in a fixed order)."""
    import torch
    codes = synth.int4_codes(66, 1, N, K)
    scales = synth.group_scales(66, 1, N, K)
    xn, x = _x(66, M, M, K)
    tid = sess.register(codes, scales)
    y1 = sess.linear(tid, x)
    y2 = sess.linear(tid, (2 * x).contiguous())
    y3 = sess.linear(tid, x)
    sess.sync()
    assert torch.equal(y1, y3)
    assert_doubles(y2, y1)


@pytest.mark.parametrize("M", [1, 4, 64, 512])
def test_placement_invariance(sess, M):
    """HBM-resident and host-streamed reads of the same tensor give bit-identical outputs."""
    import torch
    K, N = 4096, 1024
    codes = synth.int4_codes(65, M, N, K)
    scales = synth.group_scales(65, M, N, K)
    xn, x = _x(65, M, M, K)
    tid = sess.register(codes, scales, hbm=True, host=True)
    y_hbm = sess.linear(tid, x)
    sess.place(tid, True)
    sess.stats(reset=True)
    y_host = [sess.linear(tid, x) for _ in range(3)]
    sess.sync()
    st = sess.stats(reset=True)
    sess.place(tid, False)
    # each of the three launches consumed the tensor's bytes once
    assert st["host_reads"] == 3 and st["host_read_bytes"] == 3 * (codes.nbytes + scales.nbytes)
    for yh in y_host:
        assert torch.equal(y_hbm, yh)


def test_read_probe_leaves_memory_and_checks_arguments(sess):
    """The measurement probe reads device memory without changing it, and
    refuses misaligned or ragged buffers."""
    import torch
    from paper_2607_10183_amd import atsi
    buf = torch.randint(0, 256, (1 << 20,), dtype=torch.uint8, device="cuda")
    before = buf.clone()
    atsi.atsi_debug_read_probe(sess.ctx, buf.data_ptr(), buf.numel())
    atsi.atsi_debug_read_probe(sess.ctx, buf.data_ptr(), 4096 + 16)  # a ragged tail of chunks
    sess.sync()
    assert torch.equal(buf, before)
    for ptr, n in ((buf.data_ptr() + 8, 4096), (buf.data_ptr(), 100), (buf.data_ptr(), 0), (0, 4096)):
        with pytest.raises(atsi.AtsiError, match="ATSI_E_INVALID"):
            atsi.atsi_debug_read_probe(sess.ctx, ptr, n)
