"""gevo_pop_predict_noalloc (prediction whose scratch is the library's static
device array) against gevo_pop_predict (scratch in the caller's workspace):
the same scores bit for bit, on two calls in a row where the second has a
smaller input (the static array then still holds the first call's data)."""
import numpy as np
import pytest

import synthetic

pytestmark = pytest.mark.gpu


def _torch():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _data(i, n_train, n_test, dims):
    d = synthetic.dataset(synthetic.config(i), n_train, n_test)
    if dims[0] != d["x_train"].shape[1]:
        for k in ("x_train", "x_test"):
            d[k] = np.ascontiguousarray(d[k][:, :dims[0]])
    return d


def _both(pop):
    pop.predict()
    a = pop.scores()
    pop.predict_noalloc()
    b = pop.scores()
    return a, b


def _same(a, b, what):
    for k in ("test_loss", "test_acc"):
        assert np.array_equal(a[k].view(np.uint32), b[k].view(np.uint32)), (what, k, a[k][:4], b[k][:4])


def test_noalloc_prediction_equals_prediction_twice_second_smaller():
    _torch()
    import paper_2310_10211_amd as g
    # first call: 40 variants of the prediction workload's 784-512-256-10 net
    # over 1,000 rows; their scratch needs three groups in the static array
    cfg = synthetic.config(4, P=40)
    data = _data(4, 0, 1000, cfg["dims"])
    print(f"[gpu] noalloc call 1: P={cfg['P']} dims={cfg['dims']} n_test=1000", flush=True)
    pop = g.Population(cfg, data["x_train"], data["y_train"], data["x_test"], data["y_test"])
    a, b = _both(pop)
    _same(a, b, "call 1")
    assert np.all(np.isfinite(a["test_loss"]))
    pop.close()
    # second call, smaller: 6 variants of 784-256-10 trained one epoch, 300 rows
    cfg = synthetic.config(3, P=6)
    data = _data(3, 600, 300, cfg["dims"])
    print(f"[gpu] noalloc call 2: P={cfg['P']} dims={cfg['dims']} n_test=300", flush=True)
    pop = g.Population(cfg, data["x_train"], data["y_train"], data["x_test"], data["y_test"])
    pop.train_epoch(0)
    a, b = _both(pop)
    _same(a, b, "call 2")
    pop.close()


@pytest.mark.parametrize("i,dims,batch", [
    (5, [1024, 256, 128, 10], 256),     # hidden layers on the prediction GEMM and the older forward kernel
    (2, [784, 96, 10], 64),             # fp32
])
def test_noalloc_prediction_other_paths(i, dims, batch):
    _torch()
    import paper_2310_10211_amd as g
    cfg = synthetic.config(i, P=5, dims=dims, batch=batch)
    data = _data(i, 500, 400, dims)
    print(f"[gpu] noalloc paths: P=5 dims={dims}", flush=True)
    pop = g.Population(cfg, data["x_train"], data["y_train"], data["x_test"], data["y_test"])
    pop.train_epoch(0)
    a, b = _both(pop)
    _same(a, b, str(dims))
    pop.close()


def test_noalloc_rejects_a_variant_larger_than_the_static_scratch():
    """One variant of 8192-8192-256-10 bf16 needs a 128 MiB weight copy of its
    first layer: the call returns GEVO_E_UNSUPPORTED before launching
    anything, and the handle still predicts through the workspace."""
    _torch()
    import paper_2310_10211_amd as g
    dims = [8192, 8192, 256, 10]
    cfg = synthetic.config(4, P=1, dims=dims)
    rng = np.random.default_rng(3)
    x = rng.random((256, 8192), dtype=np.float32)
    y = (np.arange(256) % 10).astype(np.int32)
    print("[gpu] noalloc oversize: P=1 dims=[8192, 8192, 256, 10]", flush=True)
    pop = g.Population(cfg, None, None, x, y)
    with pytest.raises(g.GevoError, match="unsupported"):
        pop.predict_noalloc()
    pop.predict()
    assert np.isfinite(pop.scores()["test_loss"][0])
    pop.close()
