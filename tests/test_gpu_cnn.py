"""GPU parity of the convolutional prediction workload: the HIP path (through
the C-ABI) against the CPU oracle (oracle/cnn.py) on the same seeded inputs.

Bars: masks, densities and biases bit-exact; weights within 2e-6 relative
(the GPU draws the noise's normal deviate with binary32 log and cos, so the
factor 1 + std eps may differ from the oracle's fp64 draw in its last bits;
with no noise they are bit-exact); per variant the mean
test cross-entropy within 2e-3 relative and the number of correct images
within max(1, n/200).  The oracle rounds the same values to bfloat16 as the
kernels (input, weights, every activation, the pooled features) and sums in
fp64; the kernels sum in fp32 in another order, so an activation lands on the
other side of a bf16 rounding boundary with probability about K 2^-16 (K the
length of its sum) and then moves by one bf16 ulp (2^-8 relative).  These
independent one-ulp moves change the mean loss by far less than 2e-3, and
move an argmax only for images whose two largest logits are that close.
"""
import math

import numpy as np
import pytest

import oracle
import synthetic
from oracle import cnn

pytestmark = pytest.mark.gpu

CNN_LOSS_RTOL = 2e-3


def _torch():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _pop(cfg, base, x, y):
    _torch()
    import paper_2310_10211_amd as g
    print(f"[gpu] CnnPopulation {cfg['name']} P={cfg['P']} HxWxC={cfg['H']}x{cfg['W']}x{cfg['C']} "
          f"stem={cfg['stem']} blocks={cfg['blocks']} n_test={len(y)}", flush=True)
    return g.CnnPopulation(cfg, base, x, y)


def _check(scores, ref, variants, n):
    for v in variants:
        ce, corr = ref[v]
        got_loss = float(scores["test_loss"][v])
        want_loss = ce / n
        assert abs(got_loss - want_loss) <= CNN_LOSS_RTOL * abs(want_loss), (v, got_loss, want_loss)
        got_corr = round(float(scores["test_acc"][v]) * n)
        assert abs(got_corr - corr) <= max(1, n // 200), (v, got_corr, corr)


SMALL_SHAPES = [
    dict(),                                                    # 8x8x3, stem 32, blocks (1,128) (2,128)
    dict(name="p4-dwsep-cnn4x4x4-64-128-7", P=4, H=4, W=4, C=4, stem=64, blocks=[(2, 128)], classes=7,
         n_test=70, seed=33, noise_std=0.0),
    dict(name="p3-dwsep-cnn8x8x1-32-128-256-32", P=3, C=1, blocks=[(1, 128), (2, 256)], classes=32,
         n_test=64, seed=34, dens=(0.2, 0.9), noise_std=0.05),
    # stride-1 depthwise layers after pointwise ones (the fused kernel with S = 1)
    dict(name="p2-dwsep-cnn8x8x3-32-128-128-256-10", P=2, blocks=[(2, 128), (1, 128), (1, 256)], n_test=100,
         seed=35),
    # a 256-channel pointwise input: that pair runs unfused, the first pair fused in two strips
    dict(name="p2-dwsep-cnn8x8x3-32-256-128-128-10", P=2, blocks=[(1, 256), (1, 128), (2, 128)], n_test=100,
         seed=36),
    # a stem map too large to stay in LDS: the stem and the first depthwise layer run unfused
    dict(name="p2-dwsep-cnn32x32x3-64-128-10", P=2, H=32, W=32, stem=64, blocks=[(2, 128)], n_test=70, seed=37),
]


@pytest.mark.parametrize("over", SMALL_SHAPES)
def test_variants_equal_the_oracle(over):
    cfg = synthetic.cnn_config("small", **over)
    base, x, y = synthetic.cnn_inputs(cfg)
    pop = _pop(cfg, base, x, y)
    ths = cnn.thresholds(cfg, range(cfg["P"]))
    for v in range(cfg["P"]):
        e = pop.export(v)
        params, mask = cnn.variant_params(cfg, base.astype(np.float64), v, ths[v])
        _, dens, _ = oracle.variant_hparams(cfg["seed"], v, (1e-3, 1e-3), cfg["dens"])
        assert e["density"] == float(dens)
        assert np.array_equal(e["mask"], mask), v
        np.testing.assert_allclose(e["params"], params, rtol=2e-6, atol=0)
        off = moff = 0
        for _, K, N in cnn.tensors(cfg):                          # pruned weights are +0
            W = e["params"][off:off + K * N][mask[moff:moff + K * N] == 0]
            assert np.all(W == 0) and not np.any(np.signbit(W))
            off += K * N + N
            moff += K * N
        if cfg["noise_std"] == 0.0:
            assert e["params"].tobytes() == params.astype(np.float32).tobytes(), v
    pop.close()


@pytest.mark.parametrize("over", SMALL_SHAPES)
def test_prediction_matches_the_oracle(over):
    cfg = synthetic.cnn_config("small", **over)
    base, x, y = synthetic.cnn_inputs(cfg)
    pop = _pop(cfg, base, x, y)
    pop.predict()
    s = pop.scores()
    ref = cnn.evaluate(cfg, base.astype(np.float64), x, y, range(cfg["P"]), mode="bf16")
    _check(s, ref, range(cfg["P"]), len(y))
    assert np.all(s["time_s"] > 0)
    pop.close()


def test_full_shape_sampled_variants():
    """The full net (32x32x3, stem 32, four blocks up to 512 channels, P = 64)
    in the launch configuration of the benchmark, over the first 1,000 test
    images (15 chunks and a ragged one of 40); variants 0 and 63 against the
    oracle."""
    cfg = synthetic.cnn_config("full")
    base, x, y = synthetic.cnn_inputs(cfg, n_test=1000)
    pop = _pop(cfg, base, x, y)
    pop.predict()
    s = pop.scores()
    ref = cnn.evaluate(cfg, base.astype(np.float64), x, y, [0, 63], mode="bf16")
    _check(s, ref, [0, 63], len(y))
    pop.close()


def test_density_zero_leaves_only_the_head_bias():
    """With every weight pruned the logits are the head's biases for every
    image: the mean loss is the mean of lse(b) - b_y, the accuracy the share
    of labels equal to the first maximal bias (closed form, no oracle)."""
    cfg = synthetic.cnn_config("small", dens=(0.0, 0.0))
    base, x, y = synthetic.cnn_inputs(cfg)
    pop = _pop(cfg, base, x, y)
    pop.predict()
    s = pop.scores()
    b = base[-cfg["classes"]:].astype(np.float64)
    lse = math.log(np.exp(b - b.max()).sum()) + b.max()
    want_loss = float(np.mean(lse - b[y]))
    want_acc = float(np.mean(y == int(np.argmax(b))))
    for v in range(cfg["P"]):
        assert pop.export(v)["mask"].sum() == 0
        assert abs(float(s["test_loss"][v]) - want_loss) <= 1e-5 * abs(want_loss)
        assert abs(float(s["test_acc"][v]) - want_acc) < 1e-6
    pop.close()


def test_identical_variants_score_identically_and_predict_is_repeatable():
    cfg = synthetic.cnn_config("small", dens=(1.0, 1.0), noise_std=0.0)
    base, x, y = synthetic.cnn_inputs(cfg)
    pop = _pop(cfg, base, x, y)
    pop.predict()
    s1 = pop.scores()
    pop.predict()
    s2 = pop.scores()
    assert np.all(s1["test_loss"] == s1["test_loss"][0]) and np.all(s1["test_acc"] == s1["test_acc"][0])
    assert s1["test_loss"].tobytes() == s2["test_loss"].tobytes()
    assert s1["test_acc"].tobytes() == s2["test_acc"].tobytes()
    pop.close()


def test_scores_before_predict_is_an_order_error():
    cfg = synthetic.cnn_config("small", P=2, n_test=64)
    base, x, y = synthetic.cnn_inputs(cfg)
    pop = _pop(cfg, base, x, y)
    import paper_2310_10211_amd as g
    with pytest.raises(g.GevoError, match="order"):
        pop.scores()
    pop.close()


def test_labels_outside_the_classes_are_rejected():
    cfg = synthetic.cnn_config("small", P=2, n_test=64)
    base, x, y = synthetic.cnn_inputs(cfg)
    y = y.copy()
    y[5] = cfg["classes"]
    import paper_2310_10211_amd as g
    with pytest.raises(g.GevoError, match="shape"):
        _pop(cfg, base, x, y)


@pytest.mark.parametrize("over", [dict(), SMALL_SHAPES[3], SMALL_SHAPES[4], SMALL_SHAPES[5]])
def test_launch_plan_matches_the_benchmark_cost_model(over):
    """The benchmark's roofline prices each kernel kind from its own copy of
    the library's fusion rules; the kinds and launch counts the library
    reports must be the ones it prices."""
    import bench
    cfg = synthetic.cnn_config("full", **over) if not over else synthetic.cnn_config("small", **over)
    base, x, y = synthetic.cnn_inputs(cfg, n_test=min(cfg["n_test"], 200))
    pop = _pop(cfg, base, x, y)
    pop.set_profiling(True)
    pop.predict()
    st = pop.kernel_stats()
    costs = bench.cnn_costs(cfg, len(y))
    chunks = (len(y) + 63) // 64
    nb = len(cfg["blocks"])
    fused = sum(1 for i in range(nb - 1) if bench.cnn_fuse_rows(
        ([cfg["stem"]] + [c for _, c in cfg["blocks"]])[i], cfg["blocks"][i][1],
        _sizes(cfg)[i + 1][1], cfg["blocks"][i + 1][0], _sizes(cfg)[i + 2][0]))
    assert {k for k, (_, n) in st.items() if n and k != "reduce"} == set(costs)
    assert st["pw_dw"][1] == chunks * fused
    assert st["pointwise"][1] == chunks * (nb - fused)
    assert st["depthwise"][1] == chunks * (nb - fused)
    assert st["stem"][1] == st["pool"][1] == st["head"][1] == chunks
    pop.close()


def _sizes(cfg):
    out = [(cfg["H"], cfg["W"])]
    for s, _ in cfg["blocks"]:
        h, w = out[-1]
        out.append(((h - 1) // s + 1, (w - 1) // s + 1))
    return out


# Removed block layers (a structural edit: section 6.1 removes a convolution
# layer, section 4.1 repairs the shapes).  Per variant the names it loses;
# the kinds covered: a stride-1 depthwise layer on the stem output, a
# stride-2 depthwise layer inside the fused pointwise + depthwise kernel, a
# widening pointwise layer (32 -> 128 channels, channels of value 1 appended), a
# narrowing one (256 -> 128, the first kept), a square one, and variant 0
# left whole.
REMOVAL_CASES = [
    (dict(P=4, n_test=100, seed=41), {1: ("dw0",), 2: ("pw0", "dw1"), 3: ("pw1",)}),
    (dict(name="p4-dwsep-cnn8x8x3-32-256-128-128-10", P=4, blocks=[(1, 256), (1, 128), (2, 128)], n_test=100,
          seed=42), {1: ("pw1",), 2: ("dw2", "pw2"), 3: ("dw0", "pw0", "dw1")}),
]


def _tensor_slices(cfg):
    off = moff = 0
    out = {}
    for name, K, N in cnn.tensors(cfg):
        out[name] = (off, moff, K, N)
        off += K * N + N
        moff += K * N
    return out


@pytest.mark.parametrize("over,gone", REMOVAL_CASES)
def test_removed_layers_match_the_oracle(over, gone):
    cfg = synthetic.cnn_config("small", **over)
    base, x, y = synthetic.cnn_inputs(cfg)
    pop = _pop(cfg, base, x, y)
    for v, names in gone.items():
        for name in names:
            print(f"[gpu] remove {name} from variant {v}", flush=True)
            pop.remove_layer(v, name)
    pop.predict()
    s = pop.scores()
    ref = cnn.evaluate(cfg, base.astype(np.float64), x, y, range(cfg["P"]), mode="bf16", removed=gone)
    _check(s, ref, range(cfg["P"]), len(y))
    whole = cnn.evaluate(cfg, base.astype(np.float64), x, y, list(gone), mode="bf16")
    assert any(abs(whole[v][0] - ref[v][0]) > 1e-2 * abs(ref[v][0]) for v in gone)   # the edits matter
    # exported: the removed layers in identity form, every other tensor the variant's own
    ths = cnn.thresholds(cfg, range(cfg["P"]))
    sl = _tensor_slices(cfg)
    for v in range(cfg["P"]):
        e = pop.export(v)
        params, mask = cnn.variant_params(cfg, base.astype(np.float64), v, ths[v])
        for name, (off, moff, K, N) in sl.items():
            W = e["params"][off:off + K * N].reshape(K, N)
            b = e["params"][off + K * N:off + K * N + N]
            if name in gone.get(v, ()):
                ident = np.zeros((K, N), np.float32)
                bias = np.zeros(N, np.float32)
                if name.startswith("dw"):
                    ident[4, :] = 1.0
                else:
                    ident[np.arange(min(K, N)), np.arange(min(K, N))] = 1.0
                    bias[K:] = 1.0                                   # appended channels hold the value 1
                assert W.tobytes() == ident.tobytes() and b.tobytes() == bias.tobytes(), name
                assert np.array_equal(e["mask"][moff:moff + K * N], (ident != 0).ravel().astype(np.uint8))
            else:
                assert np.array_equal(e["mask"][moff:moff + K * N], mask[moff:moff + K * N]), (v, name)
                np.testing.assert_allclose(W.ravel(), params[off:off + K * N], rtol=2e-6, atol=0)
                assert b.tobytes() == params[off + K * N:off + K * N + N].astype(np.float32).tobytes()
    pop.close()


def test_remove_layer_rejects_the_stem_the_head_and_bad_indexes():
    cfg = synthetic.cnn_config("small", P=2, n_test=64, seed=43)
    base, x, y = synthetic.cnn_inputs(cfg)
    pop = _pop(cfg, base, x, y)
    n_t = len(cnn.tensors(cfg))
    for v, layer in [(0, 0), (0, n_t - 1), (0, n_t), (2, 1)]:
        with pytest.raises(Exception):
            pop.remove_layer(v, layer)
    pop.predict()                                   # the handle still works, no variant edited
    s = pop.scores()
    ref = cnn.evaluate(cfg, base.astype(np.float64), x, y, range(cfg["P"]), mode="bf16")
    _check(s, ref, range(cfg["P"]), len(y))
    pop.close()
