"""The C-ABI library loads, exports what include/atsi.h declares, and rejects
bad arguments before touching HIP (CPU only: no compute calls)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "atsi.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(atsi_[a-z_0-9]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    from paper_2607_10183_amd import atsi
    return atsi.lib()


def test_header_declares_the_boundary():
    names = _declared()
    for required in ("atsi_create", "atsi_destroy", "atsi_last_error", "atsi_tensor_register",
                     "atsi_set_placement", "atsi_linear", "atsi_sync"):
        assert required in names


def test_every_declared_symbol_is_exported(lib):
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_covers_every_declared_symbol():
    from paper_2607_10183_amd import atsi
    missing = [n for n in _declared() if not hasattr(atsi, n)]
    assert not missing, missing


def test_create_validates_before_hip(lib):
    from paper_2607_10183_amd import atsi
    P = ctypes.c_void_p
    out = P()
    # null out
    assert lib.atsi_create(0, 1, 2, None, 256, 1 << 20, None, 4, None) == 1
    # same stream twice / null stream / second transfer stream equal to another
    assert lib.atsi_create(0, 1, 1, None, 256, 1 << 20, None, 4, ctypes.byref(out)) == 1
    assert lib.atsi_create(0, 0, 2, None, 256, 1 << 20, None, 4, ctypes.byref(out)) == 1
    assert lib.atsi_create(0, 1, 2, 2, 256, 1 << 20, None, 4, ctypes.byref(out)) == 1
    assert lib.atsi_create(0, 1, 2, 1, 256, 1 << 20, None, 4, ctypes.byref(out)) == 1
    assert "second transfer stream" in atsi.atsi_last_error(None)
    # misaligned workspace, bad slot count
    assert lib.atsi_create(0, 1, 2, 3, 255, 1 << 20, None, 4, ctypes.byref(out)) == 1
    assert lib.atsi_create(0, 1, 2, 3, 256, 1 << 20, None, 1, ctypes.byref(out)) == 1
    assert "n_slots" in atsi.atsi_last_error(None)
    assert out.value is None


def test_create_without_gpu_fails_cleanly(lib):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    from paper_2607_10183_amd import atsi
    out = ctypes.c_void_p()
    st = lib.atsi_create(0, 1, 2, 3, 256, 1 << 20, None, 4, ctypes.byref(out))
    assert st == 6 and out.value is None
    assert "GPU" in atsi.atsi_last_error(None)


def test_null_context_is_invalid(lib):
    assert lib.atsi_sync(None) == 1
    assert lib.atsi_destroy(None) == 1
    assert lib.atsi_linear(None, 0, None, 1, None) == 1
    assert lib.atsi_get_stats(None, None, 0) == 1
