"""Pins of the convolutional prediction workload's CPU oracle (oracle/cnn.py)
against library routines, definitions and brute force."""
import math

import numpy as np
import pytest
from scipy.signal import correlate2d
from scipy.special import logsumexp

import oracle
from oracle import cnn


@pytest.mark.parametrize("stride", [1, 2])
def test_depthwise_conv_matches_scipy_correlate(stride):
    rng = np.random.default_rng(1)
    a = rng.normal(size=(2, 9, 7, 3))
    w = rng.normal(size=(9, 3))
    got = cnn.conv3x3_depthwise(a, w, stride)
    for n in range(2):
        for c in range(3):
            full = correlate2d(a[n, :, :, c], w[:, c].reshape(3, 3), mode="same", boundary="fill")
            assert np.allclose(got[n, :, :, c], full[::stride, ::stride], rtol=1e-12, atol=1e-12)


def test_depthwise_identity_filter_returns_its_input():
    rng = np.random.default_rng(2)
    a = rng.random((1, 6, 6, 4))
    w = np.zeros((9, 4))
    w[4] = 1.0                                                 # centre tap
    assert np.array_equal(cnn.conv3x3_depthwise(a, w, 1), a)
    assert np.array_equal(cnn.conv3x3_depthwise(a, w, 2), a[:, ::2, ::2, :])


def test_full_conv_matches_brute_force_loops():
    rng = np.random.default_rng(3)
    n, H, W, C, M = 1, 5, 4, 3, 2
    a = rng.normal(size=(n, H, W, C))
    w = rng.normal(size=(9 * C, M))
    got = cnn.conv3x3_full(a, w)
    for y in range(H):
        for x in range(W):
            for m in range(M):
                s = 0.0
                for dy in range(3):
                    for dx in range(3):
                        yy, xx = y + dy - 1, x + dx - 1
                        if 0 <= yy < H and 0 <= xx < W:
                            for c in range(C):
                                s += a[0, yy, xx, c] * w[(3 * dy + dx) * C + c, m]
                assert abs(got[0, y, x, m] - s) < 1e-12


def test_softmax_stats_match_logsumexp_and_first_argmax():
    z = np.array([[1.0, 3.0, 3.0, -2.0], [0.5, 0.5, 0.5, 0.5], [10.0, -1.0, 2.0, 9.0]])
    y = np.array([2, 0, 0])
    ce, corr = cnn.softmax_stats(z, y)
    assert abs(ce - sum(logsumexp(z[i]) - z[i, y[i]] for i in range(3))) < 1e-12
    assert corr == 2                                           # row 0: first maximum is class 1


def test_tensor_init_is_the_chain_initialisation_of_each_layer():
    dims = [12, 7, 5]
    base = np.random.default_rng(4).normal(size=oracle.param_count(dims))
    for v in (0, 3):
        params, mask = oracle.variant_init(9, v, dims, 1 << 23, 1, base, 0.05)
        off, moff = 0, 0
        for l in range(1, len(dims)):
            K, N = dims[l - 1], dims[l]
            W, b, M = cnn.tensor_init(9, v, l - 1, K, N, 1 << 23, base[off:off + K * N].reshape(K, N),
                                      base[off + K * N:off + K * N + N], 0.05)
            assert np.array_equal(W.ravel(), params[off:off + K * N])
            assert np.array_equal(b, params[off + K * N:off + K * N + N])
            assert np.array_equal(M.ravel(), mask[moff:moff + K * N])
            off += K * N + N
            moff += K * N


def test_tensor_init_layer_index_decorrelates_equal_shapes():
    W0, _, M0 = cnn.tensor_init(9, 1, 0, 9, 16, 1 << 23)
    W1, _, M1 = cnn.tensor_init(9, 1, 1, 9, 16, 1 << 23)
    assert not np.array_equal(W0, W1) and not np.array_equal(M0, M1)


TINY = dict(C=3, stem=2, blocks=[(2, 3)], classes=3, seed=11, dens=(1.0, 1.0), noise_std=0.0)


def _brute_forward(cfg, params, img):
    """Pure-Python per-pixel forward of one image (fp64, no rounding)."""
    p = cnn.unpack(params, cfg)
    H, W, C = img.shape
    Ws, bs = p["stem"]
    a = [[[max(0.0, bs[m] + sum(img[y + dy - 1][x + dx - 1][c] * Ws[(3 * dy + dx) * C + c][m]
                                 for dy in range(3) for dx in range(3) for c in range(C)
                                 if 0 <= y + dy - 1 < H and 0 <= x + dx - 1 < W))
           for m in range(cfg["stem"])] for x in range(W)] for y in range(H)]
    ch = cfg["stem"]
    for i, (s, co) in enumerate(cfg["blocks"]):
        Wd, bd = p[f"dw{i}"]
        Ho, Wo = (H - 1) // s + 1, (W - 1) // s + 1
        d = [[[max(0.0, bd[c] + sum(a[s * yo + dy - 1][s * xo + dx - 1][c] * Wd[3 * dy + dx][c]
                                     for dy in range(3) for dx in range(3)
                                     if 0 <= s * yo + dy - 1 < H and 0 <= s * xo + dx - 1 < W))
               for c in range(ch)] for xo in range(Wo)] for yo in range(Ho)]
        Wp, bp = p[f"pw{i}"]
        a = [[[max(0.0, bp[m] + sum(d[y][x][c] * Wp[c][m] for c in range(ch))) for m in range(co)]
              for x in range(Wo)] for y in range(Ho)]
        H, W, ch = Ho, Wo, co
    h = [sum(a[y][x][c] for y in range(H) for x in range(W)) / (H * W) for c in range(ch)]
    Wf, bf = p["fc"]
    return [bf[k] + sum(h[c] * Wf[c][k] for c in range(ch)) for k in range(cfg["classes"])]


def test_forward_matches_brute_force_on_a_tiny_net():
    rng = np.random.default_rng(5)
    params = rng.normal(0, 0.5, cnn.param_count(TINY))
    x = rng.random((2, 5, 4, 3)).astype(np.float32)
    got = cnn.forward_logits(TINY, params, x, mode="f64")
    for i in range(2):
        want = _brute_forward(TINY, params, x[i].astype(np.float64))
        assert np.allclose(got[i], want, rtol=1e-12, atol=1e-12)


def test_bf16_mode_rounds_activations_to_bfloat16():
    rng = np.random.default_rng(6)
    params = rng.normal(0, 0.5, cnn.param_count(TINY))
    x = rng.random((1, 4, 4, 3)).astype(np.float32)
    z16 = cnn.forward_logits(TINY, params, x, mode="bf16")
    z64 = cnn.forward_logits(TINY, params, x, mode="f64")
    assert not np.array_equal(z16, z64)
    assert np.allclose(z16, z64, rtol=0.05, atol=0.05)


def test_pooling_of_a_constant_map_is_the_constant():
    cfg = dict(C=1, stem=1, blocks=[(1, 1)], classes=2, seed=1)
    params = np.zeros(cnn.param_count(cfg))
    p = cnn.unpack(params, cfg)
    p["stem"][1][:] = 0.75                                    # stem bias: constant 0.75 map
    p["dw0"][0][4, 0] = 1.0                                   # identity depthwise filter
    p["pw0"][0][0, 0] = 1.0                                   # identity pointwise layer
    p["fc"][0][0, :] = [1.0, -1.0]
    z = cnn.forward_logits(cfg, params, np.zeros((1, 4, 4, 1), np.float32), mode="f64")
    assert np.allclose(z[0], [0.75, -0.75])
    assert math.isclose(cnn.softmax_stats(z, np.array([0]))[0], math.log1p(math.exp(-1.5)))


def test_variant_params_apply_noise_and_mask_to_the_base():
    cfg = dict(TINY, dens=(0.5, 0.5), noise_std=0.01)
    base = np.random.default_rng(7).normal(size=cnn.param_count(cfg))
    th = cnn.thresholds(cfg, [2])[0]
    params, mask = cnn.variant_params(cfg, base, 2, th)
    pb, pp = cnn.unpack(base, cfg), cnn.unpack(params, cfg)
    moff = 0
    for name, K, N in cnn.tensors(cfg):
        Wb, bb = pb[name]
        W, b = pp[name]
        M = mask[moff:moff + K * N].reshape(K, N).astype(bool)
        moff += K * N
        assert np.all(W[~M] == 0.0)
        assert np.all(np.abs(W[M] / Wb[M] - 1.0) < 0.1)       # 1 + 0.01 eps
        assert np.array_equal(b, bb)                           # biases are not perturbed
    assert 0.35 < mask.mean() < 0.65


# A removed block layer (section 6.1 takes a convolution layer out of MobileNet)
# is the identity map plus the shape repair of section 4.1.  On non-negative
# inputs (every block layer reads a ReLU output) that equals the same layer with
# identity weights: the depthwise centre tap 1 (at stride 2 it reads exactly the
# pixels (2 yo, 2 xo)), or the pointwise matrix with ones on its diagonal (the
# first channels kept when it narrows; when it widens, the appended channels
# have no weights and bias 1, so relu(1) = 1 pads them with value 1), and zero
# biases otherwise.  These pins compare the skip code against those layers
# computed by the convolution code pinned above.
REMOVAL = dict(C=3, stem=4, blocks=[(1, 3), (2, 5), (2, 2)], classes=3, seed=12, dens=(1.0, 1.0),
               noise_std=0.0)


def _with_identity(cfg, params, name):
    out = np.array(params, np.float64)
    off = 0
    for tname, K, N in cnn.tensors(cfg):
        if tname == name:
            W = np.zeros((K, N))
            if name.startswith("dw"):
                W[4, :] = 1.0                                     # centre tap (dy, dx) = (1, 1)
            else:
                for k in range(min(K, N)):
                    W[k, k] = 1.0
            out[off:off + K * N] = W.ravel()
            out[off + K * N:off + K * N + N] = 0.0
            if name.startswith("pw"):
                out[off + K * N + K:off + K * N + N] = 1.0     # appended channels (none when N <= K)
            return out
        off += K * N + N
    raise KeyError(name)


@pytest.mark.parametrize("mode", ["f64", "bf16"])
@pytest.mark.parametrize("gone", [("dw0",), ("dw1",), ("pw1",), ("pw2",), ("pw0",), ("dw1", "pw1", "dw2")])
def test_removed_layers_equal_identity_layers(mode, gone):
    rng = np.random.default_rng(21)
    params = np.abs(rng.normal(0, 0.5, cnn.param_count(REMOVAL)))      # every unit stays active
    x = rng.random((2, 5, 7, 3)).astype(np.float32)
    ident = params
    for name in gone:
        ident = _with_identity(REMOVAL, ident, name)
    got = cnn.forward_logits(REMOVAL, params, x, mode=mode, removed=gone)
    want = cnn.forward_logits(REMOVAL, ident, x, mode=mode)
    assert np.array_equal(got, want)
    assert not np.array_equal(got, cnn.forward_logits(REMOVAL, params, x, mode=mode))


def test_removed_layer_ignores_its_parameters_and_repairs_shapes():
    rng = np.random.default_rng(22)
    a = rng.random((1, 5, 7, 3))
    d = cnn.removed_depthwise(a, 2)
    assert d.shape == (1, 3, 4, 3) and np.array_equal(d[0, 1, 2], a[0, 2, 4])
    assert d.shape[1:3] == cnn.conv3x3_depthwise(a, np.ones((9, 3)), 2).shape[1:3]
    assert np.array_equal(cnn.removed_depthwise(a, 1), a)
    wide = cnn.removed_pointwise(a, 5)
    assert np.array_equal(wide[..., :3], a) and np.all(wide[..., 3:] == 1.0)
    assert np.array_equal(cnn.removed_pointwise(a, 2), a[..., :2])
    params = np.abs(rng.normal(0, 0.5, cnn.param_count(REMOVAL)))
    x = rng.random((1, 5, 7, 3)).astype(np.float32)
    other = params + (_with_identity(REMOVAL, params, "pw1") != params) * 7.0   # pw1 changed, nothing else
    assert not np.array_equal(other, params)
    assert np.array_equal(cnn.forward_logits(REMOVAL, params, x, mode="f64", removed=("pw1",)),
                          cnn.forward_logits(REMOVAL, other, x, mode="f64", removed=("pw1",)))
