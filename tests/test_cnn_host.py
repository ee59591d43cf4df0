"""Host side of the convolutional prediction workload's C-ABI: the parameter
count against the oracle's definition, shape validation and argument checks
that return before any HIP call (no GPU needed)."""
import ctypes

import pytest

import synthetic
from oracle import cnn

g = pytest.importorskip("paper_2310_10211_amd")

OK, E_ARG, E_WORKSPACE, E_UNSUPPORTED = 0, -1, -3, -6


def _lib():
    try:
        return g.lib()
    except OSError as e:  # pragma: no cover - the library is built by build()
        pytest.skip(f"libgevo not built: {e}")


def _rc_count(cfg):
    n = ctypes.c_size_t()
    c = g.cnn_config_struct(cfg)
    return _lib().gevo_cnn_param_count(ctypes.byref(c), ctypes.byref(n)), n.value


@pytest.mark.parametrize("key", ["small", "full"])
def test_param_count_matches_the_oracle(key):
    cfg = synthetic.cnn_config(key)
    rc, n = _rc_count(cfg)
    assert rc == OK and n == cnn.param_count(cfg)
    base, x, y = synthetic.cnn_inputs(cfg, n_test=3)
    assert base.size == n and x.shape == (3, cfg["H"], cfg["W"], cfg["C"])


@pytest.mark.parametrize("over,code", [
    (dict(stem=48), E_UNSUPPORTED),                        # stem channels not a multiple of 32
    (dict(stem=544), E_UNSUPPORTED),                       # over 512
    (dict(blocks=[(1, 96)]), E_UNSUPPORTED),               # block channels not a multiple of 128
    (dict(blocks=[(1, 1152)]), E_UNSUPPORTED),             # over 1024
    (dict(blocks=[(3, 128)]), E_UNSUPPORTED),              # stride 3
    (dict(blocks=[]), E_UNSUPPORTED),
    (dict(blocks=[(2, 128)] * 5), E_UNSUPPORTED),          # more than four blocks
    (dict(H=2, W=2, blocks=[(2, 128)]), E_UNSUPPORTED),    # 64 images x 1 pixel: not a multiple of 256 rows
    (dict(H=4, W=4, blocks=[(2, 128)]), OK),               # 64 x 4 rows
    (dict(classes=1), E_UNSUPPORTED),
    (dict(classes=33), E_UNSUPPORTED),
    (dict(C=5), E_UNSUPPORTED),
    (dict(C=4), OK),
    (dict(H=96, W=96), E_UNSUPPORTED),                     # padded image over the stem's 56 KiB of LDS
    (dict(H=64, W=64), OK),
    (dict(P=0), E_ARG),
    (dict(dens=(0.8, 0.7)), E_ARG),
    (dict(dens=(0.5, 1.5)), E_ARG),
    (dict(noise_std=-1.0), E_ARG),
])
def test_shape_and_argument_validation(over, code):
    cfg = synthetic.cnn_config("small", **over)
    if len(cfg["blocks"]) > g.CNN_MAX_BLOCKS:
        c = g.cnn_config_struct(dict(cfg, blocks=cfg["blocks"][:g.CNN_MAX_BLOCKS]))
        c.n_blocks = len(cfg["blocks"])
        n = ctypes.c_size_t()
        assert _lib().gevo_cnn_param_count(ctypes.byref(c), ctypes.byref(n)) == code
        return
    if not cfg["blocks"]:
        c = g.cnn_config_struct(dict(cfg, blocks=[(1, 128)]))
        c.n_blocks = 0
        n = ctypes.c_size_t()
        assert _lib().gevo_cnn_param_count(ctypes.byref(c), ctypes.byref(n)) == code
        return
    assert _rc_count(cfg)[0] == code


def test_workspace_grows_with_the_test_split_and_rejects_an_empty_one():
    L = _lib()
    c = g.cnn_config_struct(synthetic.cnn_config("full"))
    b = []
    for n in (1, 64, 65, 10000):
        out = ctypes.c_size_t()
        assert L.gevo_cnn_workspace_bytes(ctypes.byref(c), n, ctypes.byref(out)) == OK
        b.append(out.value)
    assert b[0] == b[1] < b[2] < b[3]
    out = ctypes.c_size_t()
    assert L.gevo_cnn_workspace_bytes(ctypes.byref(c), 0, ctypes.byref(out)) == E_ARG


def test_abi_version_checked():
    c = g.cnn_config_struct(synthetic.cnn_config("small"))
    c.abi_version = 99
    n = ctypes.c_size_t()
    assert _lib().gevo_cnn_param_count(ctypes.byref(c), ctypes.byref(n)) == E_ARG
    assert _lib().gevo_cnn_param_count(None, ctypes.byref(n)) == E_ARG


def test_init_rejects_bad_arguments_before_any_hip_call():
    L = _lib()
    c = g.cnn_config_struct(synthetic.cnn_config("small"))
    h = ctypes.c_void_p()
    dummy = ctypes.c_void_p(0x100000)                        # never dereferenced: rejected first
    hp = ctypes.cast(dummy, ctypes.POINTER(ctypes.c_float))
    big = 1 << 40
    assert L.gevo_cnn_init(ctypes.byref(c), ctypes.c_void_p(0x100010), big, hp, dummy, dummy, 150, None,
                           ctypes.byref(h)) == E_WORKSPACE   # misaligned
    assert L.gevo_cnn_init(ctypes.byref(c), dummy, 256, hp, dummy, dummy, 150, None,
                           ctypes.byref(h)) == E_WORKSPACE   # too small
    assert L.gevo_cnn_init(ctypes.byref(c), dummy, big, None, dummy, dummy, 150, None, ctypes.byref(h)) == E_ARG
    assert L.gevo_cnn_init(ctypes.byref(c), dummy, big, hp, None, dummy, 150, None, ctypes.byref(h)) == E_ARG
    assert L.gevo_cnn_init(ctypes.byref(c), dummy, big, hp, dummy, dummy, 0, None, ctypes.byref(h)) == E_ARG
    assert L.gevo_cnn_init(ctypes.byref(c), dummy, big, hp, dummy, dummy, 150, None, None) == E_ARG
    assert h.value is None


def test_null_handles_rejected():
    L = _lib()
    assert L.gevo_cnn_predict(None) == E_ARG
    assert L.gevo_cnn_scores(None, None, None, None) == E_ARG
    assert L.gevo_cnn_export(None, 0, None, None, None) == E_ARG
    assert L.gevo_cnn_remove_layer(None, 0, 1) == E_ARG
    assert L.gevo_cnn_set_profiling(None, 1) == E_ARG
    assert L.gevo_cnn_kernel_stats(None, 0, None, None) == E_ARG
    L.gevo_cnn_destroy(None)
