"""The C-ABI library loads and exports every symbol include/dsi.h declares;
host-side validation rejects bad calls before any device work (CPU only)."""
import ctypes
import os
import re

import pytest

from paper_2405_14105_amd import dsi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dsi.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dsi_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(dsi.LIB_PATH):
        from paper_2405_14105_amd import build
        build.build()
    return dsi.load()


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("dsi_model_create", "dsi_prefill", "dsi_verify", "dsi_kv_rollback", "dsi_accept"):
        assert required in names
    assert set(names) == set(dsi.EXPORTED)


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name
        assert isinstance(getattr(lib, name), ctypes._CFuncPtr)


def test_header_is_plain_c():
    text = open(HEADER).read()
    for banned in ("at::", "c10::", "torch::", "#include <hip", "#include <torch"):
        assert banned not in text


def test_host_validation_without_device(lib):
    # null config: rejected before any HIP call
    out = ctypes.c_void_p()
    assert lib.dsi_model_create(None, None, ctypes.byref(out)) == dsi.DSI_EINVAL
    # bad shapes
    bad = dsi.make_config(1, 100, 2, 2, 32, 64, 10)        # d_model not a multiple of 32
    assert lib.dsi_model_create(ctypes.byref(bad), None, ctypes.byref(out)) == dsi.DSI_EINVAL
    bad = dsi.make_config(1, 128, 3, 2, 32, 64, 10)        # heads not a multiple of kv heads
    assert lib.dsi_model_create(ctypes.byref(bad), None, ctypes.byref(out)) == dsi.DSI_EINVAL
    bad = dsi.make_config(1, 128, 2, 2, 48, 64, 10)        # unsupported head_dim
    assert lib.dsi_model_create(ctypes.byref(bad), None, ctypes.byref(out)) == dsi.DSI_EINVAL
    assert "head_dim" in dsi.dsi_last_error()
    # dsi_accept argument checks
    P = ctypes.c_void_p(16)
    assert lib.dsi_accept(None, 0, 3, 100, P, P, P, P, 1.0, 0, P, P) == dsi.DSI_EINVAL
    assert lib.dsi_accept(None, 9, 7, 100, P, P, P, P, 1.0, 0, P, P) == dsi.DSI_EINVAL   # 64 rows max
    assert lib.dsi_accept(None, 1, 3, 100, P, P, None, P, 1.0, 0, P, P) == dsi.DSI_EINVAL  # q missing
    assert lib.dsi_accept(None, 1, 3, 100, P, P, P, P, 0.0, 0, P, P) == dsi.DSI_EINVAL   # T <= 0
    assert lib.dsi_accept(None, 1, 3, 100, P, P, P, P, 1.0, 7, P, P) == dsi.DSI_EINVAL   # mode
    assert lib.dsi_verify(None, None, None, None, None) == dsi.DSI_EINVAL
    assert lib.dsi_kv_rollback(None, 0, 0) == dsi.DSI_EINVAL
