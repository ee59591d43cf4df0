"""GPU parity: the HIP path (through the C-ABI) against the CPU oracle on the same
seeded inputs.

Bars (per variant): masks, learning rates, densities, data order and the
initial Xavier weights bit-exact; fp32 losses within 1e-4 relative; bf16
losses within 2e-2 relative; accuracy within 0.5 percentage points; one SGD
step from an identical fp32 state within 1e-5 relative.
"""
import math
import sys

import numpy as np
import pytest

import oracle
import synthetic

pytestmark = pytest.mark.gpu

F32_LOSS_RTOL = 1e-4
BF16_LOSS_RTOL = 2e-2
ACC_ATOL = 0.005


def _torch():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _pop(cfg, data, **kw):
    _torch()
    import paper_2310_10211_amd as g
    print(f"[gpu] Population {cfg.get('name', '')} P={cfg['P']} dims={cfg['dims']} dtype={cfg['dtype']} "
          f"n_train={len(data['y_train'])} n_test={len(data['y_test'])}", flush=True)
    return g.Population(cfg, data["x_train"], data["y_train"], data["x_test"], data["y_test"], **kw)


def _small(i, P=None, n_train=None, n_test=None, **over):
    c = synthetic.config(i, **over)
    if P is not None:
        c["P"] = P
    d = synthetic.dataset(c, n_train, n_test)
    return c, d


def _rel(a, b):
    return abs(a - b) / max(abs(b), 1e-30)


def _check_losses(gpu, ref, variants, rtol, acc_tol=ACC_ATOL, train=True):
    for v in variants:
        r = ref[v]
        if train:
            assert _rel(float(gpu["train_loss"][v]), r["train_loss"][-1]) <= rtol, (v, gpu["train_loss"][v], r["train_loss"][-1])
            assert abs(float(gpu["train_acc"][v]) - r["train_acc"][-1]) <= acc_tol, (v, gpu["train_acc"][v], r["train_acc"][-1])
        assert _rel(float(gpu["test_loss"][v]), r["test_loss"]) <= rtol, (v, gpu["test_loss"][v], r["test_loss"])
        assert abs(float(gpu["test_acc"][v]) - r["test_acc"]) <= acc_tol, (v, gpu["test_acc"][v], r["test_acc"])


# ------------------------------------------------------------------- exactness
def test_bf16_rounding_is_exact_over_all_encodings():
    """The bf16 kernels round with gfx950's packed conversion instruction.  Over
    all 2^32 binary32 encodings, in both operand pairings, it equals the
    bit-level round-to-nearest-even (NaN -> quiet NaN), denormals included."""
    _torch()
    import paper_2310_10211_amd as g
    print("[gpu] exhaustive bf16 rounding check", flush=True)
    assert g.check_bf16_rounding() == [0, 0]


@pytest.mark.parametrize("i", [1, 3, 5])
def test_population_init_bit_exact(i):
    cfg, data = _small(i, P=6, n_train=600, n_test=300)
    pop = _pop(cfg, data)
    ref = oracle.population(cfg)
    for v in range(cfg["P"]):
        e = pop.export(v)
        assert e["lr"] == ref[v]["lr"] and e["density"] == ref[v]["density"]
        np.testing.assert_array_equal(e["mask"], ref[v]["mask"])
        np.testing.assert_array_equal(e["params"], ref[v]["params"].astype(np.float32))
    pop.close()


def test_base_noise_init_matches_oracle():
    cfg, data = _small(4, P=5, n_test=300, dims=[784, 64, 32, 10])
    pop = _pop(cfg, data)
    ref = oracle.population(cfg)
    for v in range(cfg["P"]):
        e = pop.export(v)
        np.testing.assert_array_equal(e["mask"], ref[v]["mask"])
        np.testing.assert_allclose(e["params"], ref[v]["params"], rtol=2e-6, atol=1e-7)
        W = e["params"][:784 * 64][e["mask"][:784 * 64] == 0]
        assert np.all(W == 0) and not np.any(np.signbit(W))
    pop.close()


def test_epoch_data_order_exact():
    cfg, data = _small(3, P=2, n_train=1000, n_test=256)
    pop = _pop(cfg, data)
    for e in range(2):
        pop.train_epoch(e)
        perm = oracle.permutation(cfg["seed"], e, 1000)
        np.testing.assert_array_equal(pop.epoch_labels(), data["y_train"][perm])
    pop.close()


# ------------------------------------------------------------- hand example
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_hand_example_one_step(dtype, golden):
    g = golden("mlp_2_3_2_sgd.txt")
    cfg = dict(name="2-3-2", dims=[2, 3, 2], P=1, batch=2, dtype=dtype, seed=1, lr=(1.0, 1.0),
               dens=(1.0, 1.0), init="xavier")
    X = np.array(g["x"], np.float32).reshape(2, 2)
    y = np.array(g["y"], np.int32)
    data = dict(x_train=X, y_train=y, x_test=X, y_test=y)
    pop = _pop(cfg, data)
    params = np.concatenate([g["W1"], g["b1"], g["W2"], g["b2"]]).astype(np.float32)
    pop.import_params(0, params)
    pop.predict()
    s = pop.scores()
    assert float(s["test_loss"][0]) == pytest.approx(g["loss0"][0], rel=1e-6)
    pop.train_epoch(0)      # one step over both samples (permutation irrelevant: full batch)
    s = pop.scores()
    assert float(s["train_loss"][0]) == pytest.approx(g["loss0"][0], rel=1e-6)
    after = pop.export(0)["params"]
    exp = np.concatenate([g["W1_after"], g["b1_after"], g["W2_after"], g["b2_after"]]).astype(np.float32)
    np.testing.assert_array_equal(after, exp)
    pop.predict()
    assert float(pop.scores()["test_loss"][0]) == pytest.approx(g["loss1"][0], rel=1e-6)
    pop.close()


# ----------------------------------------------------------- step-level parity
@pytest.mark.parametrize("dims", [[784, 128, 10], [200, 96, 64, 10]])
def test_one_step_from_identical_state_fp32(dims):
    cfg, data = _small(2, P=3, n_train=256, n_test=256, dims=dims, batch=128)
    if dims[0] != 784:
        data["x_train"] = data["x_train"][:, :dims[0]].copy()
        data["x_test"] = data["x_test"][:, :dims[0]].copy()
    pop = _pop(cfg, data)
    ref = oracle.population(cfg)
    perm = oracle.permutation(cfg["seed"], 0, 256)
    pop.train_steps(0, 0, 1)
    for v in range(cfg["P"]):
        st = ref[v]
        p = st["params"].copy()
        oracle.train_steps("f32", dims, p, st["mask"], st["lr"], data["x_train"], data["y_train"], perm,
                           cfg["batch"], 0, 1)
        got = pop.export(v)["params"]
        for (Wg, bg), (Wr, br) in zip(oracle.unpack(got.astype(np.float64), dims), oracle.unpack(p, dims)):
            scale = max(np.max(np.abs(Wr)), 1e-30)
            assert np.max(np.abs(Wg - Wr)) <= 1e-5 * scale
            bscale = max(np.max(np.abs(br)), 1e-3)
            assert np.max(np.abs(bg - br)) <= 1e-5 * bscale
    pop.close()


# --------------------------------------------------------- end-to-end parity
def test_config1_full_fp32():
    """P=4 784-128-10 fp32, 2,048 train / 512 test, batch 32, 1 epoch: full size."""
    cfg, data = _small(1)
    pop = _pop(cfg, data)
    pop.train_epoch(0)
    pop.predict()
    s = pop.scores()
    ref = oracle.evaluate(cfg, data)
    _check_losses(s, ref, range(4), F32_LOSS_RTOL)
    for v in range(4):
        np.testing.assert_array_equal(pop.export(v)["mask"], ref[v]["mask"])
    pop.close()


def test_bf16_two_layer_ragged_batch():
    """784-256-10 bf16 (config 3 shape), 4,100 train rows -> last batch of 4, 2 epochs."""
    cfg, data = _small(3, P=8, n_train=4100, n_test=1000, epochs=2)
    pop = _pop(cfg, data)
    pop.train_epoch(0)
    pop.train_epoch(1)
    pop.predict()
    s = pop.scores()
    ref = oracle.evaluate(cfg, data, epochs=2)
    _check_losses(s, ref, range(8), BF16_LOSS_RTOL)
    pop.close()


@pytest.mark.parametrize("dims,batch,n_train", [
    ([784, 128, 10], 32, 700),      # hidden 128, batch tile 32, ragged tail
    ([784, 100, 10], 64, 650),      # hidden 100 (padded to 128), batch tile 64
    ([784, 128, 10], 128, 600),     # hidden 128, batch tile 128
    ([784, 256, 10], 50, 620),      # hidden 256, batch 50 (tile 64)
    ([300, 250, 7], 20, 500),       # input 300 (10 column blocks), hidden 250, 7 classes, tile 32
    ([784, 256, 16], 128, 600),     # 16 classes: the largest count of the 16-row logits tiles
    ([784, 128, 24], 64, 600),      # 24 classes: 32-row logits tiles
])
def test_bf16_two_layer_shapes(dims, batch, n_train):
    """Two-layer bf16 nets at the other hidden widths and batch tiles of the per-variant training kernel."""
    cfg, data = _small(3, P=3, n_train=n_train, n_test=300, dims=dims, batch=batch)
    if dims[0] != 784:
        data["x_train"] = data["x_train"][:, :dims[0]].copy()
        data["x_test"] = data["x_test"][:, :dims[0]].copy()
    if dims[-1] != 10:                 # spread the ten synthetic classes over all dims[-1] labels
        for split in ("y_train", "y_test"):
            y = data[split]
            data[split] = ((y + 10 * (np.arange(len(y)) % 3)) % dims[-1]).astype(y.dtype)
    pop = _pop(cfg, data)
    pop.train_epoch(0)
    pop.predict()
    s = pop.scores()
    ref = oracle.evaluate(cfg, data, epochs=1)
    _check_losses(s, ref, range(3), BF16_LOSS_RTOL)
    pop.close()


@pytest.mark.parametrize("i,dims,batch", [
    (3, None, None),
    (5, [1024, 256, 128, 10], 256),      # hidden layers on the streaming kernel's register-image masters
])
def test_export_import_round_trip_between_epochs_is_exact(i, dims, batch):
    """Exporting and re-importing every variant between epochs (the register-image
    copies of the fused two-layer kernel and of the streamed hidden layers are
    rebuilt from the imported master) leaves the run bitwise unchanged."""
    over = {"epochs": 2}
    if dims:
        over.update(dims=dims, batch=batch)
    cfg, data = _small(i, P=3, n_train=700, n_test=256, **over)
    if dims and dims[0] != 3072:
        data["x_train"] = data["x_train"][:, :dims[0]].copy()
        data["x_test"] = data["x_test"][:, :dims[0]].copy()
    runs = []
    for round_trip in (False, True):
        pop = _pop(cfg, data)
        pop.train_epoch(0)
        if round_trip:
            for v in range(cfg["P"]):
                pop.import_params(v, pop.export(v)["params"])
        pop.train_epoch(1)
        runs.append([pop.export(v)["params"].tobytes() for v in range(cfg["P"])])
        pop.close()
    differing = [v for v in range(cfg["P"]) if runs[0][v] != runs[1][v]]
    assert not differing, f"variants whose parameters differ: {differing}"


def test_bf16_one_step_after_import_matches_oracle():
    """An imported state trains from that state: one bf16 SGD step of the
    784-256-10 net against the oracle from the same state."""
    cfg, data = _small(3, P=2, n_train=256, n_test=256)
    dims = cfg["dims"]
    pop = _pop(cfg, data)
    ref = oracle.population(cfg)
    rng = np.random.default_rng(5)
    perm = oracle.permutation(cfg["seed"], 0, 256)
    for v in range(cfg["P"]):
        st = ref[v]
        p = st["params"] + 0.01 * rng.standard_normal(st["params"].shape)
        pop.import_params(v, p.astype(np.float32))             # masked weights are imported as +0
        st["params"] = pop.export(v)["params"].astype(np.float64)
    pop.train_steps(0, 0, 1)
    for v in range(cfg["P"]):
        st = ref[v]
        q = st["params"].copy()
        oracle.train_steps("bf16", dims, q, st["mask"], st["lr"], data["x_train"], data["y_train"], perm,
                           cfg["batch"], 0, 1)
        got = pop.export(v)["params"].astype(np.float64)
        for (Wg, bg), (Wr, br) in zip(oracle.unpack(got, dims), oracle.unpack(q, dims)):
            assert np.max(np.abs(Wg - Wr)) <= 1e-4 * max(np.max(np.abs(Wr)), 1e-30)
            assert np.max(np.abs(bg - br)) <= 1e-4 * max(np.max(np.abs(br)), 1e-3)
    pop.close()


def test_bf16_three_layer():
    """Three weight layers (config 5 structure) at reduced width, batch 256 with a ragged tail."""
    cfg, data = _small(5, P=4, n_train=1300, n_test=600, dims=[3072, 160, 96, 10])
    pop = _pop(cfg, data)
    pop.train_epoch(0)
    pop.predict()
    s = pop.scores()
    ref = oracle.evaluate(cfg, data, epochs=1)
    _check_losses(s, ref, range(4), BF16_LOSS_RTOL)
    pop.close()


@pytest.mark.parametrize("dims,batch,n_train", [
    ([3072, 256, 128, 10], 256, 1300),    # both hidden layers on the streaming kernel, ragged tail of 20
    ([512, 128, 256, 10], 100, 730),      # batch tile 128
    ([3072, 192, 128, 10], 256, 800),     # first hidden layer on the blocked kernel (192 units), second streamed
    ([3072, 256, 160, 10], 256, 700),     # second layer's 256 inputs streamed, 160 units on the blocked kernel
    ([1024, 384, 256, 10], 128, 700),     # three 128-unit tiles per variant, batch tile 128
])
def test_bf16_deep_nets_on_the_streaming_layer_kernel(dims, batch, n_train):
    """Hidden layers whose widths are multiples of 128 and whose inputs are
    multiples of 64, at batch tiles 128 and 256, train through the streaming
    hidden-layer kernel; the other layers of the same nets through the
    blocked one."""
    cfg, data = _small(5, P=3, n_train=n_train, n_test=400, dims=dims, batch=batch)
    if dims[0] != 3072:
        data["x_train"] = data["x_train"][:, :dims[0]].copy()
        data["x_test"] = data["x_test"][:, :dims[0]].copy()
    pop = _pop(cfg, data)
    pop.train_epoch(0)
    pop.predict()
    s = pop.scores()
    ref = oracle.evaluate(cfg, data, epochs=1)
    _check_losses(s, ref, range(3), BF16_LOSS_RTOL)
    pop.close()


def test_fp32_three_layer():
    cfg, data = _small(2, P=3, n_train=700, n_test=300, dims=[784, 96, 64, 10], batch=64)
    pop = _pop(cfg, data)
    pop.train_epoch(0)
    pop.predict()
    s = pop.scores()
    ref = oracle.evaluate(cfg, data, epochs=1)
    _check_losses(s, ref, range(3), F32_LOSS_RTOL)
    pop.close()


def test_prediction_only_population():
    cfg, data = _small(4, P=16, n_test=1000, dims=[784, 128, 64, 10])
    pop = _pop(cfg, data)
    pop.predict()
    s = pop.scores()
    ref = oracle.evaluate(cfg, data, epochs=0)
    _check_losses(s, ref, range(16), BF16_LOSS_RTOL, train=False)
    assert np.all(np.isnan(s["train_loss"]))
    pop.close()


def test_single_layer_net():
    """Degenerate depth: no hidden layer (multinomial logistic regression)."""
    cfg, data = _small(3, P=3, n_train=500, n_test=256, dims=[784, 10], batch=50)
    pop = _pop(cfg, data)
    pop.train_epoch(0)
    pop.predict()
    ref = oracle.evaluate(cfg, data, epochs=1)
    _check_losses(pop.scores(), ref, range(3), BF16_LOSS_RTOL)
    pop.close()


# --------------------------------------------------------------- invariants
def test_lr_zero_leaves_weights_bitwise_unchanged():
    cfg, data = _small(3, P=3, n_train=512, n_test=256, lr=(0.0, 0.0))
    pop = _pop(cfg, data)
    before = [pop.export(v)["params"] for v in range(3)]
    pop.train_epoch(0)
    for v in range(3):
        assert pop.export(v)["params"].tobytes() == before[v].tobytes()
    pop.close()


def test_masked_weights_stay_plus_zero_and_divergence_is_contained():
    cfg, data = _small(3, P=12, n_train=1024, n_test=256, lr=(1e-2, 1e4), dens=(0.3, 0.6))
    pop = _pop(cfg, data)
    pop.train_epoch(0)
    pop.predict()
    s = pop.scores()
    ref = oracle.evaluate(cfg, data, epochs=1)
    healthy = [v for v in range(12) if ref[v]["lr"] < 0.3]
    assert healthy and len(healthy) < 12
    _check_losses(s, ref, healthy, BF16_LOSS_RTOL)
    for v in range(12):
        e = pop.export(v)
        W = e["params"][:784 * 256]
        z = W[e["mask"][:784 * 256] == 0]
        assert np.all(z == 0) and not np.any(np.signbit(z))
        if v not in healthy:
            assert not math.isfinite(float(s["train_loss"][v])) or s["train_loss"][v] > 2.0
    pop.close()


def test_variants_are_independent_of_population_size():
    cfg8, data = _small(3, P=8, n_train=640, n_test=256)
    cfg3 = dict(cfg8, P=3)
    a = _pop(cfg8, data)
    b = _pop(cfg3, data)
    for p in (a, b):
        p.train_epoch(0)
        p.predict()
    sa, sb = a.scores(), b.scores()
    for v in range(3):
        assert a.export(v)["params"].tobytes() == b.export(v)["params"].tobytes()
        assert sa["train_loss"][v] == sb["train_loss"][v] and sa["test_acc"][v] == sb["test_acc"][v]
    a.close(); b.close()


def test_runs_are_deterministic_and_steps_compose():
    cfg, data = _small(3, P=4, n_train=1000, n_test=256)
    a = _pop(cfg, data)
    a.train_epoch(0)
    b = _pop(cfg, data)
    T = b.steps_per_epoch
    b.train_steps(0, 0, 3)
    b.train_steps(0, 3, T)
    for v in range(4):
        assert a.export(v)["params"].tobytes() == b.export(v)["params"].tobytes()
    assert a.scores()["train_loss"].tobytes() == b.scores()["train_loss"].tobytes()
    a.close(); b.close()


def test_call_order_errors():
    import paper_2310_10211_amd as g
    cfg, data = _small(3, P=2, n_train=512, n_test=256)
    pop = _pop(cfg, data)
    with pytest.raises(g.GevoError):
        pop.train_epoch(1)                    # epochs start at 0
    pop.train_steps(0, 0, 1)
    with pytest.raises(g.GevoError):
        pop.train_steps(0, 2, 3)              # must continue where it stopped
    pop.close()


# --------------------------------------------- full-size sampled parity checks
def _sampled_training_parity(i, steps, sample, rtol, mode):
    cfg = synthetic.config(i)
    data = synthetic.dataset(cfg)
    pop = _pop(cfg, data)
    pop.train_steps(0, 0, steps)
    s = pop.scores()
    ref = oracle.evaluate(cfg, data, variants=sample, epochs=1, steps=steps, do_predict=False, mode=mode)
    for v in sample:
        assert _rel(float(s["train_loss"][v]), ref[v]["train_loss"][0]) <= rtol, (v, s["train_loss"][v],
                                                                                 ref[v]["train_loss"][0])
        assert abs(float(s["train_acc"][v]) - ref[v]["train_acc"][0]) <= 2 * ACC_ATOL + 1.0 / (steps * cfg["batch"])
    pop.close()


def test_config2_full_size_sampled_fp32():
    _sampled_training_parity(2, 12, [0, 31, 63], F32_LOSS_RTOL, "f32")


def test_config3_full_size_sampled_bf16():
    _sampled_training_parity(3, 12, [0, 100, 255], BF16_LOSS_RTOL, "bf16")


def test_config5_full_size_sampled_bf16():
    _sampled_training_parity(5, 3, [0, 127], BF16_LOSS_RTOL, "bf16")


def test_config4_full_size_sampled_predict():
    cfg = synthetic.config(4)
    data = synthetic.dataset(cfg)
    pop = _pop(cfg, data)
    pop.predict()
    s = pop.scores()
    sample = [0, 511, 1023]
    ref = oracle.evaluate(cfg, data, variants=sample, epochs=0)
    _check_losses(s, ref, sample, BF16_LOSS_RTOL, train=False)
    pop.close()
