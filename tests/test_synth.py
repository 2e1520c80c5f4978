"""The seeded input generator: determinism, slicing and distributions (CPU only)."""
import numpy as np

import synth
from synth import configs


def test_splitmix64_reference_outputs():
    # SplitMix64 seeded with 0 (state advanced by GOLDEN before mixing): published first output
    assert int(synth.words(0, 0, 1)[0]) == 0xE220A8397B1DCDAF


def test_determinism_and_row_slicing():
    a = synth.int4_codes(1, 2, 64, 256)
    b = synth.int4_codes(1, 2, 64, 256)
    assert np.array_equal(a, b)
    assert np.array_equal(synth.int4_codes(1, 2, 64, 256, row0=10, rows=7), a[10:17])
    s = synth.group_scales(1, 2, 64, 256)
    assert np.array_equal(synth.group_scales(1, 2, 64, 256, row0=5, rows=3), s[5:8])
    assert not np.array_equal(a, synth.int4_codes(1, 3, 64, 256))


def test_distributions():
    codes = synth.int4_codes(2, 1, 512, 4096)
    nib = np.concatenate([(codes & 15).ravel(), (codes >> 4).ravel()])
    hist = np.bincount(nib, minlength=16) / nib.size
    assert np.all(np.abs(hist - 1 / 16) < 2e-3)
    s = synth.group_scales(2, 1, 512, 4096).astype(np.float64)
    assert s.min() >= 0.005 - 1e-6 and s.max() <= 0.02 + 1e-5
    x = synth.activations(2, 3, 64, 4096).astype(np.float64)
    assert abs(x.mean()) < 0.01 and abs(x.std() - 1) < 0.01
    wr = synth.router_weights(2, 4, 2048, 128).astype(np.float64)
    assert abs(wr.std() * np.sqrt(2048) - 1) < 0.01
    xe = synth.exact_activations(2, 5, 8, 256).astype(np.float64)
    assert set(np.unique(xe * 4).astype(int)) <= set(range(-4, 5))


def test_placement_recipes():
    m2 = configs.dense_layer_host_mask()
    assert m2.sum() == 3
    shape = configs.DenseShape()
    m3 = configs.dense_stack_host_mask()
    sizes = np.array([configs.qbytes(*shape.kn(r)) for r in configs.ROLES])
    host = (m3 * sizes[None, :]).sum()
    total = 32 * sizes.sum()
    assert host <= 0.30 * total and host >= 0.30 * total - sizes.max()
    m4 = configs.moe_host_experts()
    assert m4.sum() == 51
    assert shape.layer_bytes() == 122_683_392


def test_router_bias_reproduces_capped_zipf_out_of_sample():
    """The fitted bias gives the capped Zipf(1.1) expert loads on fresh logits
    (within 15 % per expert at 65,536 tokens)."""
    from synth.calibrate_router_bias import capped_zipf, load_bias
    import json, os
    b = load_bias().astype(np.float64)
    d = json.load(open(os.path.join(os.path.dirname(synth.__file__), "router_bias_e128_k8.json")))
    rank = np.array(d["rank"])
    target = capped_zipf(128, 8)[rank]
    assert abs(target.sum() - 8) < 1e-9 and target.max() == 1.0
    T = 65536
    z = synth.normal(synth.stream_key(777, 1, 7), T * 128).reshape(T, 128)
    sel = np.argpartition(-(z + b), 7, axis=1)[:, :8]
    frac = np.bincount(sel.ravel(), minlength=128) / T
    assert np.all(np.abs(frac - target) <= 0.15 * target)
