"""Host-side checks of the C-ABI library that need no GPU: it loads, exports
every symbol the header declares, validates configurations before any HIP
call, and its host-side data order equals the oracle's bit for bit."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import synthetic
from tests.conftest import ROOT

g = pytest.importorskip("paper_2310_10211_amd")

OK, E_ARG, E_SHAPE, E_WORKSPACE, E_ORDER, E_HIP, E_UNSUPPORTED = 0, -1, -2, -3, -4, -5, -6


def _lib():
    try:
        return g.lib()
    except ImportError as e:
        pytest.skip(str(e))


def test_library_exports_every_declared_symbol():
    L = _lib()
    with open(os.path.join(ROOT, "include", "gevo.h")) as f:
        hdr = f.read()
    declared = set(re.findall(r"^\s*(?:gevo_status|void|const char\*)\s+(gevo_\w+)\s*\(", hdr, re.M))
    assert len(declared) >= 14
    assert declared == set(g.EXPORTED)
    for name in declared:
        assert hasattr(L, name), name


@pytest.mark.parametrize("i", [1, 2, 3, 4, 5])
def test_workspace_bytes_for_every_config(i):
    _lib()
    c = synthetic.config(i)
    n = g.workspace_bytes(c, c["n_train"], c["n_test"])
    assert n > 0 and n % 256 == 0
    weights = sum(c["dims"][l - 1] * c["dims"][l] for l in range(1, len(c["dims"])))
    assert n >= c["P"] * weights * 4                       # at least the fp32 masters


def _rc(cfg, n_train=100, n_test=50):
    keep = []
    s = g.config_struct(cfg, n_train, n_test, keep)
    out = ctypes.c_size_t()
    return _lib().gevo_pop_workspace_bytes(ctypes.byref(s), ctypes.byref(out))


@pytest.mark.parametrize("over,code", [
    (dict(), OK),
    (dict(dims=[784, 10]), OK),
    (dict(dims=[784, 64, 32, 10]), OK),
    (dict(dims=[784, 64, 32, 16, 10]), E_UNSUPPORTED),     # deeper than the build supports
    (dict(dims=[784, 256, 33]), E_UNSUPPORTED),            # > 32 classes
    (dict(dims=[784, 0, 10]), E_SHAPE),
    (dict(batch=0), E_ARG),
    (dict(batch=257), E_UNSUPPORTED),
    (dict(P=0), E_ARG),
    (dict(lr=(0.1, 0.01)), E_ARG),
    (dict(lr=(0.0, 0.1)), E_ARG),                          # log-uniform needs lo > 0
    (dict(lr=(0.0, 0.0)), OK),
    (dict(dens=(0.5, 1.5)), E_ARG),
    (dict(dens=(0.7, 0.6)), E_ARG),
    (dict(dtype="f32", dims=[784, 2048, 1024, 10]), E_UNSUPPORTED),   # fp32 output layer over 1024 wide
    (dict(dims=[784, 2048, 512, 10]), OK),
])
def test_config_validation(over, code):
    cfg = synthetic.config(3, **over)
    assert _rc(cfg) == code


def test_split_sizes_validated():
    cfg = synthetic.config(3)
    assert _rc(cfg, n_train=0, n_test=10) == OK            # prediction only
    assert _rc(cfg, n_train=10, n_test=0) == E_SHAPE
    assert _rc(cfg, n_train=-1, n_test=10) == E_SHAPE


def test_abi_version_checked():
    keep = []
    s = g.config_struct(synthetic.config(3), 10, 10, keep)
    s.abi_version = 99
    out = ctypes.c_size_t()
    assert _lib().gevo_pop_workspace_bytes(ctypes.byref(s), ctypes.byref(out)) == E_ARG
    assert _lib().gevo_pop_workspace_bytes(None, ctypes.byref(out)) == E_ARG


def test_init_rejects_bad_workspace_before_any_hip_call():
    L = _lib()
    keep = []
    s = g.config_struct(synthetic.config(3), 100, 50, keep)
    h = ctypes.c_void_p()
    dummy = ctypes.c_void_p(0x100000)                        # never dereferenced: rejected first
    assert L.gevo_pop_init(ctypes.byref(s), None, 1 << 40, dummy, dummy, dummy, dummy, None, ctypes.byref(h)) == E_WORKSPACE
    assert L.gevo_pop_init(ctypes.byref(s), ctypes.c_void_p(0x100010), 1 << 40, dummy, dummy, dummy, dummy, None,
                           ctypes.byref(h)) == E_WORKSPACE   # misaligned
    assert L.gevo_pop_init(ctypes.byref(s), ctypes.c_void_p(0x100000), 256, dummy, dummy, dummy, dummy, None,
                           ctypes.byref(h)) == E_WORKSPACE   # too small
    assert L.gevo_pop_init(ctypes.byref(s), ctypes.c_void_p(0x100000), 1 << 40, dummy, dummy, None, dummy, None,
                           ctypes.byref(h)) == E_ARG         # missing test split
    assert L.gevo_pop_init(ctypes.byref(s), ctypes.c_void_p(0x100000), 1 << 40, None, dummy, dummy, dummy, None,
                           ctypes.byref(h)) == E_ARG         # missing train split with n_train > 0
    assert L.gevo_pop_init(ctypes.byref(s), ctypes.c_void_p(0x100000), 1 << 40, dummy, dummy, dummy, dummy, None,
                           None) == E_ARG
    assert h.value is None


def test_null_handles_rejected():
    L = _lib()
    assert L.gevo_pop_train_epoch(None, 0) == E_ARG
    assert L.gevo_pop_predict(None) == E_ARG
    assert L.gevo_pop_scores(None, None, None, None, None, None) == E_ARG
    L.gevo_pop_destroy(None)


@pytest.mark.parametrize("seed,epoch,n", [(10214, 0, 60000), (10214, 1, 60000), (7, 3, 1), (7, 3, 0),
                                          (2**40 + 5, 9, 1003)])
def test_host_data_order_equals_oracle(seed, epoch, n):
    _lib()
    np.testing.assert_array_equal(g.epoch_permutation(seed, epoch, n), oracle.permutation(seed, epoch, n))


def test_status_strings():
    L = _lib()
    for code in (OK, E_ARG, E_SHAPE, E_WORKSPACE, E_ORDER, E_HIP, E_UNSUPPORTED):
        assert L.gevo_status_str(code)
    assert L.gevo_status_str(12345) == b"unknown status"


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(g, "_lib", None)
    monkeypatch.setattr(g, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        g.lib()
