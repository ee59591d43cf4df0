"""Oracle pins of a removed hidden layer (section 6.1 removes a layer of the
net; section 4.1 repairs the shapes by dropping values or padding with 1): the
layer takes its identity form (oracle.removed_layer_form) and trains with
learning rate 0 (the `frozen` bits of oracle.train_steps).  On non-negative
inputs the net then computes, and trains, exactly like the net without that
layer, with the next layer reading the kept inputs (narrowing) or the kept
inputs followed by inputs of value 1 (widening)."""
import numpy as np
import pytest

import oracle
from oracle import nsga2 as ns


def _layers(dims, params):
    out, off = [], 0
    for l in range(1, len(dims)):
        k = dims[l - 1] * dims[l]
        out.append((params[off:off + k].reshape(dims[l - 1], dims[l]), params[off + k:off + k + dims[l]]))
        off += k + dims[l]
    return out


def _flat(layers):
    return np.concatenate([np.concatenate([W.ravel(), b]) for W, b in layers])


def _case(seed, dims):
    rng = np.random.default_rng(seed)
    params = rng.normal(0, 0.3, oracle.param_count(dims))
    X = (rng.random((48, dims[0])) * (rng.random((48, dims[0])) < 0.6)).astype(np.float32)   # >= 0, with zeros
    y = rng.integers(0, dims[-1], 48).astype(np.int32)
    return params, X, y


def _removed(dims, params, l, widths=None):
    widths = widths or list(dims)
    layers = _layers(dims, params)
    W, b, m = oracle.removed_layer_form(dims, widths, l)
    layers[l - 1] = (W, b)
    mask = np.ones(oracle.weight_count(dims), np.uint8)
    off = sum(dims[j - 1] * dims[j] for j in range(1, l))
    mask[off:off + W.size] = m.ravel()
    return _flat(layers), mask


@pytest.mark.parametrize("mode", ["f64", "bf16"])
def test_removed_narrowing_layer_predicts_like_the_net_without_it(mode):
    dims = [20, 16, 12, 4]                       # remove layer 2 (16 -> 12): the first 12 units pass on
    params, X, y = _case(1, dims)
    full, _ = _removed(dims, params, 2)
    (W1, b1), _, (W3, b3) = _layers(dims, full)
    small = _flat([(W1, b1), (np.vstack([W3, np.zeros((4, 4))]), b3)])   # [20, 16, 4], units 12..15 unread
    assert oracle.predict(mode, dims, full, X, y) == oracle.predict(mode, [20, 16, 4], small, X, y)


def test_removed_widening_layer_pads_with_ones():
    dims = [20, 8, 12, 4]                        # remove layer 2 (8 -> 12): units 8..11 hold the value 1
    params, X, y = _case(2, dims)
    full, _ = _removed(dims, params, 2)
    (W1, b1), (W2, b2), (W3, b3) = _layers(dims, full)
    assert np.all(b2[:8] == 0) and np.all(b2[8:] == 1) and np.array_equal(W2[:, :8], np.eye(8))
    small = _flat([(W1, b1), (W3[:8], b3 + W3[8:].sum(axis=0))])          # [20, 8, 4]
    ce_full, hit_full = oracle.predict("f64", dims, full, X, y)
    ce_small, hit_small = oracle.predict("f64", [20, 8, 4], small, X, y)
    assert hit_full == hit_small and abs(ce_full - ce_small) <= 1e-12 * abs(ce_small)


def test_removed_layer_follows_narrowed_widths():
    W, b, m = oracle.removed_layer_form([20, 16, 12, 4], [20, 10, 7, 4], 2)
    assert W.shape == (16, 12) and np.array_equal(np.argwhere(W == 1), np.array([[k, k] for k in range(7)]))
    assert not np.any(b) and np.array_equal(m, (W != 0).astype(np.uint8))
    W, b, m = oracle.removed_layer_form([20, 16, 12, 4], [20, 5, 9, 4], 2)
    assert np.array_equal(np.argwhere(W == 1), np.array([[k, k] for k in range(5)]))
    assert np.array_equal(b, np.r_[np.zeros(5), np.ones(4), np.zeros(3)])


@pytest.mark.parametrize("mode", ["f64", "bf16"])
def test_frozen_removed_layer_trains_like_the_net_without_it(mode):
    dims = [20, 16, 12, 4]
    params, X, y = _case(3, dims)
    full, mask = _removed(dims, params, 2)
    (W1, b1), _, (W3, b3) = _layers(dims, full)
    small = _flat([(W1, b1), (np.vstack([W3, np.zeros((4, 4))]), b3)])
    smask = np.ones(oracle.weight_count([20, 16, 4]), np.uint8)
    smask[20 * 16 + 12 * 4:] = 0                 # the rows of units 12..15 stay +0
    perm = oracle.permutation(5, 0, 48)
    ce_f, co_f = oracle.train_steps(mode, dims, full, mask, 0.05, X, y, perm, 16, 0, 3, frozen=0b010)
    ce_s, co_s = oracle.train_steps(mode, [20, 16, 4], small, smask, 0.05, X, y, perm, 16, 0, 3)
    assert co_f == co_s and abs(ce_f - ce_s) <= 1e-12 * abs(ce_s)
    (V1, c1), (V2, c2), (V3, c3) = _layers(dims, full)
    (S1, d1), (S3, d3) = _layers([20, 16, 4], small)
    np.testing.assert_allclose(V1, S1, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(V3, S3[:12], rtol=1e-12, atol=1e-15)
    assert np.array_equal(V2, np.eye(16, 12)) and not np.any(c2)     # the removed layer did not move


def test_without_the_frozen_bit_the_identity_layer_trains():
    dims = [20, 16, 12, 4]
    params, X, y = _case(4, dims)
    full, mask = _removed(dims, params, 2)
    perm = oracle.permutation(5, 0, 48)
    oracle.train_steps("f64", dims, full, mask, 0.05, X, y, perm, 16, 0, 3)
    (_, _), (V2, _), (_, _) = _layers(dims, full)
    assert not np.array_equal(V2, np.eye(16, 12))


def test_layer_edit_structure_and_density():
    dims = [784, 256, 128, 10]
    e = [(ns.LAYER_EDIT, 2, 0), (ns.BIAS_EDIT, 2, 0), (ns.PRUNE_EDIT, 7, 2 ** 23)]
    assert ns.removed_layers(e, dims) == [0, 1, 0]
    widths, keep = ns.structure(e, dims)
    assert keep == [1, 1, 1]                     # a removed layer keeps its identity biases
    total = 784 * 256 + 256 * 128 + 128 * 10
    assert ns.density(e, dims) == 0.5 * ((784 * 256 + 128 * 10) / total)
