"""Per-element output-gradient scale (the 2fcNet mutation of section 6.2
replaces the scalar 1/32 by a tensor of the gradient's shape).  CPU pins of
the oracle's scale tensor, and GPU parity of both training kernels."""
import numpy as np
import pytest

import oracle
import synthetic

DIMS = [12, 7, 5, 4]


def _batch(seed, b):
    rng = np.random.default_rng(seed)
    X = rng.random((b, DIMS[0]), dtype=np.float32)
    y = rng.integers(0, DIMS[-1], b).astype(np.int32)
    params = rng.normal(0, 0.5, oracle.param_count(DIMS))
    return X, y, params


@pytest.mark.parametrize("mode", ["f32", "bf16"])
def test_scale_tensor_of_one_over_b_is_the_scalar_path(mode):
    X, y, params = _batch(1, 8)
    ce0, g0, _, _ = oracle.batch_grad(mode, DIMS, params, X, y)
    S = np.full((8, DIMS[-1]), np.float32(1.0 / 8), np.float32)
    ce1, g1, _, _ = oracle.batch_grad(mode, DIMS, params, X, y, gscale=S)
    assert ce0 == ce1 and np.array_equal(g0, g1)


@pytest.mark.parametrize("mode", ["f64", "f32", "bf16"])
def test_doubling_the_scale_doubles_every_gradient_exactly(mode):
    X, y, params = _batch(2, 8)
    rng = np.random.default_rng(3)
    S = (rng.integers(1, 9, (8, DIMS[-1])) / 16.0).astype(np.float32)
    _, g1, _, _ = oracle.batch_grad(mode, DIMS, params, X, y, gscale=S)
    _, g2, _, _ = oracle.batch_grad(mode, DIMS, params, X, y, gscale=2 * S)
    assert np.array_equal(g2, 2 * g1)


def test_row_constant_scale_is_the_gradient_of_the_weighted_loss():
    """With S[i][c] = s_i the gradient is d/dtheta of sum_i s_i CE_i (central differences, fp64)."""
    X, y, params = _batch(4, 6)
    s = np.array([0.5, 1.0, 0.25, 2.0, 0.125, 1.5], np.float32)
    S = np.repeat(s[:, None], DIMS[-1], axis=1)
    _, g, _, _ = oracle.batch_grad("f64", DIMS, params, X, y, gscale=S)

    def loss(p):
        return sum(float(s[i]) * oracle.batch_grad("f64", DIMS, p, X[i:i + 1], y[i:i + 1], scale=1.0)[0]
                   for i in range(6))

    rng = np.random.default_rng(5)
    for j in rng.choice(params.size, 25, replace=False):
        h = 1e-6
        pp, pm = params.copy(), params.copy()
        pp[j] += h
        pm[j] -= h
        fd = (loss(pp) - loss(pm)) / (2 * h)
        assert abs(fd - g[j]) <= 1e-6 * max(1.0, abs(fd)), (j, fd, g[j])


def test_a_zero_row_drops_its_sample():
    X, y, params = _batch(6, 8)
    S = np.full((8, DIMS[-1]), np.float32(0.125), np.float32)
    S[3] = 0.0
    _, g, _, _ = oracle.batch_grad("f64", DIMS, params, X, y, gscale=S)
    keep = [i for i in range(8) if i != 3]
    _, g7, _, _ = oracle.batch_grad("f64", DIMS, params, X[keep], y[keep], gscale=S[keep])
    assert np.array_equal(g, g7)


def test_train_steps_with_scale_of_one_over_b_match_the_scalar_steps():
    cfg = synthetic.config(1)
    data = synthetic.dataset(cfg, 256, 64)
    dims = cfg["dims"]
    _, _, th = oracle.variant_hparams(cfg["seed"], 0, cfg["lr"], cfg.get("dens", (1.0, 1.0)), cfg.get("dens_list"))
    p0, mask = oracle.variant_init(cfg["seed"], 0, dims, th)
    perm = oracle.permutation(cfg["seed"], 0, 256)
    B = cfg["batch"]
    pa, pb = p0.copy(), p0.copy()
    ra = oracle.train_steps("f32", dims, pa, mask, 0.05, data["x_train"], data["y_train"], perm, B, 0, 256 // B)
    S = np.full((B, dims[-1]), np.float32(1.0 / B), np.float32)
    rb = oracle.train_steps("f32", dims, pb, mask, 0.05, data["x_train"], data["y_train"], perm, B, 0, 256 // B,
                            gscale=S)
    assert ra == rb and np.array_equal(pa, pb)


# --------------------------------------------------------------------- GPU parity
def _pop(cfg, data):
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2310_10211_amd as g
    print(f"[gpu] Population P={cfg['P']} dims={cfg['dims']} dtype={cfg['dtype']} "
          f"n_train={len(data['y_train'])}", flush=True)
    return g.Population(cfg, data["x_train"], data["y_train"], data["x_test"], data["y_test"])


def _paper_like(B, C, seed, P):
    """Mostly ones, one row holding a one-hot label vector (the shape of the
    2fcNet mutation's tensor), plus a variant with random positive scales."""
    rng = np.random.default_rng(seed)
    S = np.ones((P, B, C), np.float32)
    for v in range(P):
        S[v, B // 2] = 0.0
        S[v, B // 2, rng.integers(C)] = 1.0
        if v % 2:
            S[v] = (rng.uniform(0.25, 1.0, (B, C)) / B).astype(np.float32)
    return S


@pytest.mark.gpu
@pytest.mark.parametrize("i,dims,mode,rtol", [
    (1, None, "f32", 1e-4),                       # output kernel, fp32
    (3, None, "bf16", 2e-2),                      # fused kernel, up to 16 classes
    (3, [784, 128, 24], "bf16", 2e-2),            # fused kernel, 32-row logits tiles
    (3, [200, 96, 64, 10], "bf16", 2e-2),         # three layers: output kernel, bf16
])
def test_training_with_a_scale_tensor_matches_oracle(i, dims, mode, rtol):
    cfg = synthetic.config(i)
    cfg["P"] = 4
    if dims:
        cfg["dims"] = dims
    data = synthetic.dataset(cfg, 600, 128)
    if dims and dims[0] != 784:
        data["x_train"] = np.ascontiguousarray(data["x_train"][:, :dims[0]])
        data["x_test"] = np.ascontiguousarray(data["x_test"][:, :dims[0]])
    C = cfg["dims"][-1]
    if C != 10:
        for split in ("y_train", "y_test"):
            yy = data[split]
            data[split] = ((yy + 10 * (np.arange(len(yy)) % 3)) % C).astype(yy.dtype)
    pop = _pop(cfg, data)
    B = cfg["batch"]
    S = _paper_like(B, C, 17, 4)
    pop.set_grad_scale(S)
    pop.train_epoch(0)
    s = pop.scores()
    n = len(data["y_train"])
    perm = oracle.permutation(cfg["seed"], 0, n)
    for v in range(4):
        lr, _, th = oracle.variant_hparams(cfg["seed"], v, cfg["lr"], cfg.get("dens", (1.0, 1.0)), cfg.get("dens_list"))
        params, mask = oracle.variant_init(cfg["seed"], v, cfg["dims"], th)
        ce, _ = oracle.train_steps(mode, cfg["dims"], params, mask, lr, data["x_train"], data["y_train"], perm, B, 0,
                                   -(-n // B), gscale=S[v])
        ref = ce / n
        assert abs(float(s["train_loss"][v]) - ref) <= rtol * abs(ref), (v, s["train_loss"][v], ref)
    pop.close()


@pytest.mark.gpu
@pytest.mark.parametrize("i", [1, 3])
def test_scale_tensor_of_one_over_b_is_bitwise_the_scalar_path_on_gpu(i):
    cfg = synthetic.config(i)
    cfg["P"] = 4
    B = cfg["batch"]
    data = synthetic.dataset(cfg, 4 * B, 128)                  # whole batches only
    runs = []
    for use in (False, True):
        pop = _pop(cfg, data)
        if use:
            pop.set_grad_scale(np.full((4, B, cfg["dims"][-1]), np.float32(1.0 / B), np.float32))
        pop.train_epoch(0)
        runs.append([pop.export(v)["params"].tobytes() for v in range(4)])
        pop.close()
    assert [a == b for a, b in zip(*runs)] == [True] * 4
