"""Seeded synthetic inputs and workload definitions.

This module holds no arithmetic of the evaluated method: it only produces input
arrays (images, labels) and the workload parameters.  Both the CPU oracle side
and the GPU side receive identical arrays from here.

The paper measures fitness on MNIST (60,000 train / 10,000 test, 28x28 grey
images, section 5) and on CIFAR-10 (50,000 train / 10,000 test, 32x32 RGB,
section 5).  Neither dataset is available here, so seeded stand-ins with the
same shapes, sizes and value structure are generated instead; no item of either
dataset is reproduced.

Samples are generated in independently seeded chunks of 1,000, so the first n
samples of a split do not depend on the split's total size.

* MNIST-shaped: 784 pixels with levels k/255 and about 80 % exact zeros.  Each
  class has a few sparse "ink" styles built partly from a shared stroke pool
  (so classes overlap); a sample takes one style of its class, drops some ink,
  mixes in a faint second style from another class, adds stray pixels and
  intensity noise, then is clipped and quantised.
* CIFAR-shaped: 3,072 values (32x32x3, channel-last), dense, levels k/255, mean
  about 0.47 and s.d. about 0.25.  Classes are smooth low-frequency colour
  fields; samples add a per-sample smooth field, a brightness/contrast jitter
  and pixel noise.
Labels are class-balanced and shuffled by the seed.
"""
from __future__ import annotations

import numpy as np

DATA_SEED = 2310
_CHUNK = 1000          # samples per independently seeded chunk
POP_SEED_BASE = 10211

# The five evaluated workloads (population size P, layer widths, batch, dtype,
# epochs, split sizes, learning-rate and pruning-density distributions).
CONFIGS = {
    1: dict(name="p4-mlp784-128-10-f32", dims=[784, 128, 10], P=4, batch=32, dtype="f32", epochs=1,
            n_train=2048, n_test=512, lr=(1e-3, 1e-1), dens_list=[1.0, 0.9, 0.7, 0.5],
            init="xavier", data="mnist"),
    2: dict(name="p64-mlp784-256-10-f32", dims=[784, 256, 10], P=64, batch=128, dtype="f32", epochs=3,
            n_train=60000, n_test=10000, lr=(1e-3, 3e-1), dens=(0.4, 1.0), init="xavier", data="mnist"),
    3: dict(name="p256-mlp784-256-10-bf16", dims=[784, 256, 10], P=256, batch=128, dtype="bf16", epochs=2,
            n_train=60000, n_test=10000, lr=(1e-3, 3e-1), dens=(0.4, 1.0), init="xavier", data="mnist"),
    4: dict(name="p1024-predict-mlp784-512-256-10-bf16", dims=[784, 512, 256, 10], P=1024, batch=128,
            dtype="bf16", epochs=0, n_train=0, n_test=10000, lr=(0.0, 0.0), dens=(0.5, 1.0),
            init="base_noise", noise_std=0.01, data="mnist"),
    5: dict(name="p128-mlp3072-1024-512-10-bf16", dims=[3072, 1024, 512, 10], P=128, batch=256, dtype="bf16",
            epochs=2, n_train=50000, n_test=10000, lr=(1e-4, 1e-1), dens=(0.3, 1.0), init="xavier",
            data="cifar"),
}
for _i, _c in CONFIGS.items():
    _c["seed"] = POP_SEED_BASE + _i
    _c["index"] = _i


def config(i: int, **overrides) -> dict:
    c = dict(CONFIGS[i])
    c.update(overrides)
    return c


def _balanced_labels(rng, n, classes=10):
    y = np.arange(n, dtype=np.int32) % classes
    rng.shuffle(y)
    return y


def mnist_like(n_train: int, n_test: int, seed: int = DATA_SEED):
    """(x_train, y_train, x_test, y_test): float32 [n, 784] in k/255, int32 labels."""
    rng = np.random.default_rng(seed)
    d, classes, styles = 784, 10, 3
    pool = rng.choice(d, size=300, replace=False)            # shared stroke pixels
    protos = np.zeros((classes, styles, d), dtype=np.float32)
    for c in range(classes):
        own = rng.choice(d, size=120, replace=False)          # class-specific pixels
        for s in range(styles):
            px = np.concatenate([rng.choice(pool, 70, replace=False), rng.choice(own, 80, replace=False)])
            protos[c, s, px] = rng.uniform(0.5, 1.0, size=px.size)

    def make(n, split):
        xs, ys = [], []
        for i in range((n + _CHUNK - 1) // _CHUNK):
            x, y = make_chunk(np.random.default_rng([seed, split, i]), _CHUNK)
            xs.append(x)
            ys.append(y)
        if not xs:
            return np.zeros((0, d), np.float32), np.zeros((0,), np.int32)
        return np.concatenate(xs)[:n], np.concatenate(ys)[:n]

    def make_chunk(rng, n):
        y = _balanced_labels(rng, n, classes)
        st = rng.integers(0, styles, size=n)
        other = (y + rng.integers(1, classes, size=n)) % classes
        ost = rng.integers(0, styles, size=n)
        x = protos[y, st] * rng.uniform(0.7, 1.3, size=(n, 1)).astype(np.float32)
        x *= (rng.random((n, d)) > 0.25)                      # ink dropout
        mix = rng.uniform(0.0, 0.9, size=(n, 1)).astype(np.float32) * (rng.random((n, 1)) < 0.5)
        x += mix * protos[other, ost]                         # faint second style
        stray = rng.random((n, d)) < 0.01
        x[stray] += rng.uniform(0.2, 1.0, size=int(stray.sum())).astype(np.float32)
        ink = x > 0
        x[ink] += rng.normal(0.0, 0.12, size=int(ink.sum())).astype(np.float32)
        x = np.clip(x, 0.0, 1.0)
        x = (np.rint(x * 255.0) / 255.0).astype(np.float32)
        return x, y

    xtr, ytr = make(n_train, 0)
    xte, yte = make(n_test, 1)
    return xtr, ytr, xte, yte


def cifar_like(n_train: int, n_test: int, seed: int = DATA_SEED):
    """(x_train, y_train, x_test, y_test): float32 [n, 3072] (32x32x3) in k/255."""
    rng = np.random.default_rng(seed + 1)
    classes, H = 10, 32
    yy, xx = np.meshgrid(np.arange(H), np.arange(H), indexing="ij")
    protos = np.zeros((classes, H, H, 3), dtype=np.float32)
    for c in range(classes):
        for ch in range(3):
            f = np.zeros((H, H))
            for _ in range(3):
                fy, fx = rng.uniform(0.0, 2.5, size=2)
                ph = rng.uniform(0, 2 * np.pi)
                f += rng.uniform(0.3, 1.0) * np.cos(2 * np.pi * (fy * yy + fx * xx) / H + ph)
            protos[c, :, :, ch] = 0.47 + 0.14 * f / 3.0 + rng.uniform(-0.05, 0.05)

    def make(n, split):
        nc = (n + _CHUNK - 1) // _CHUNK
        x = np.empty((nc * _CHUNK, 3072), dtype=np.float32)
        y = np.empty((nc * _CHUNK,), dtype=np.int32)
        for i in range(nc):
            r = np.random.default_rng([seed + 1, split, i])
            x[i * _CHUNK:(i + 1) * _CHUNK], y[i * _CHUNK:(i + 1) * _CHUNK] = make_chunk(r, _CHUNK)
        return x[:n], y[:n]

    def make_chunk(rng, m):
        y = _balanced_labels(rng, m, classes)
        img = protos[y] * rng.uniform(0.7, 1.3, size=(m, 1, 1, 1)).astype(np.float32)
        img += rng.uniform(-0.1, 0.1, size=(m, 1, 1, 3)).astype(np.float32)
        low = rng.normal(0.0, 0.18, size=(m, 8, 8, 3)).astype(np.float32)
        img += np.repeat(np.repeat(low, 4, axis=1), 4, axis=2)       # per-sample smooth field
        img += rng.normal(0.0, 0.12, size=img.shape).astype(np.float32)
        img = np.clip(img, 0.0, 1.0)
        return (np.rint(img * 255.0) / 255.0).reshape(m, 3072).astype(np.float32), y

    xtr, ytr = make(n_train, 0)
    xte, yte = make(n_test, 1)
    return xtr, ytr, xte, yte


def dataset(cfg: dict, n_train: int | None = None, n_test: int | None = None, seed: int = DATA_SEED):
    """Dataset dict for a workload config; sizes default to the config's."""
    n_train = cfg["n_train"] if n_train is None else n_train
    n_test = cfg["n_test"] if n_test is None else n_test
    gen = cifar_like if cfg["data"] == "cifar" else mnist_like
    xtr, ytr, xte, yte = gen(n_train, n_test, seed)
    return dict(x_train=xtr, y_train=ytr, x_test=xte, y_test=yte)


# The convolutional prediction workload: P variants of a depthwise-separable
# (MobileNet-like) net, each run over a CIFAR-shaped test split (section 4.3's
# prediction fitness; Table 1's MobileNet is the paper's convolutional case).
CNN_CONFIGS = {
    "full": dict(name="p64-dwsep-cnn32x32x3-32-128-128-256-512-10-bf16", P=64, H=32, W=32, C=3, stem=32,
                 blocks=[(1, 128), (2, 128), (2, 256), (2, 512)], classes=10, n_test=10000,
                 dens=(0.5, 1.0), noise_std=0.01, seed=POP_SEED_BASE + 6),
    "small": dict(name="p6-dwsep-cnn8x8x3-32-128-128-10-bf16", P=6, H=8, W=8, C=3, stem=32,
                  blocks=[(1, 128), (2, 128)], classes=10, n_test=150,
                  dens=(0.5, 1.0), noise_std=0.01, seed=POP_SEED_BASE + 7),
}


def cnn_config(key: str, **overrides) -> dict:
    c = dict(CNN_CONFIGS[key])
    c.update(overrides)
    return c


def cnn_tensor_shapes(cfg: dict):
    """[(K, N)] of the net's weight tensors in canonical order: stem (9 C x
    stem), then per block depthwise (9 x C_in) and pointwise (C_in x C_out),
    then the head (C_last x classes)."""
    out = [(9 * cfg["C"], cfg["stem"])]
    c = cfg["stem"]
    for _, co in cfg["blocks"]:
        out += [(9, c), (c, co)]
        c = co
    return out + [(c, cfg["classes"])]


def cnn_inputs(cfg: dict, n_test: int | None = None, seed: int = DATA_SEED):
    """(base parameters float32 canonical, images float32 [n][H][W][C],
    labels int32 [n]).

    The base model stands in for a pretrained one: weights are normal with
    variance 2 / fan_in (fan_in = 9 C for the stem, 9 for a depthwise filter,
    C_in for a pointwise layer and the head), biases normal with s.d. 0.05.
    Images are the CIFAR-shaped stand-in, cropped (top-left) to H x W when
    smaller than 32 x 32, with C of its 3 channels (C <= 3) or the first
    channel repeated (C = 4).  Labels are the stand-in's ten classes taken
    modulo the net's class count."""
    n = cfg["n_test"] if n_test is None else n_test
    r = np.random.default_rng([seed + 5, cfg["seed"]])
    parts = []
    for K, N in cnn_tensor_shapes(cfg):
        parts.append(r.normal(0.0, np.sqrt(2.0 / K), size=K * N))     # fan_in = K
        parts.append(r.normal(0.0, 0.05, size=N))
    base = np.concatenate(parts).astype(np.float32)
    H, W, C = cfg["H"], cfg["W"], cfg["C"]
    assert H <= 32 and W <= 32 and 1 <= C <= 4
    _, _, x, y = cifar_like(0, n, seed)
    img = x.reshape(n, 32, 32, 3)[:, :H, :W, :]
    img = img[..., :C] if C <= 3 else np.concatenate([img, img[..., :1]], axis=3)
    return base, np.ascontiguousarray(img, np.float32), (y % cfg["classes"]).astype(np.int32)
