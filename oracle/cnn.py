"""CPU oracle of the convolutional prediction workload (GEVO-ML, arXiv
2310.10211, section 4.3: the prediction workload runs a model over a dataset
and records its error; Table 1's MobileNet is the paper's convolutional
case).

TEST INFRASTRUCTURE ONLY: plain numpy in fp64, imported only by the tests,
the smoke check and the CPU-baseline leg of the benchmark.

The net, CIFAR-shaped and MobileNet-like (depthwise-separable blocks):
  stem   3x3 convolution, stride 1, zero padding 1, C -> c_stem, bias, ReLU
  block  3x3 depthwise convolution, stride s (1 or 2), padding 1, bias, ReLU;
         then 1x1 pointwise convolution C_in -> c_out, bias, ReLU
  head   global average pooling, fully connected C_last -> classes, softmax
Per image the result is the cross-entropy against its label and whether the
argmax (lowest index on ties) equals it.

Weight tensors are K x N matrices, in this order (their index is the layer
index of the population's random draws):
  stem   K = 9 C, k = (3 dy + dx) C + c,  N = c_stem
  dw_i   K = 9,   k = 3 dy + dx,          N = C_in (one filter per channel)
  pw_i   K = C_in,                         N = c_out
  fc     K = C_last,                       N = classes
each followed by its N biases; the canonical parameter vector is their
concatenation ([K][N] row-major, then the biases), like the fully connected
nets' layers.  Variants are built as in the workload-4 population: base
weights times fl(1 + fl(std eps)) under a Bernoulli(rho_v) mask
(``tensor_init``, the C oracle's per-tensor draws).

Mode "bf16" rounds the input, every weight and every activation after ReLU
(and after pooling) to bfloat16, as the GPU path does, and sums in fp64;
mode "f64" rounds nothing.

Parity status: conv3x3 pinned against scipy.signal.correlate2d and an
identity filter; the stem against brute-force loops; pooling and the
pointwise layer by their definitions; the whole forward against a
brute-force per-pixel implementation on a tiny net; tensor_init against the
chain initialisation of the fully connected nets; removed layers (skip plus
repair) against the same layers with identity weights (the centre tap, or
the truncated identity matrix with bias 1 on appended channels, and zero
biases otherwise).
"""
from __future__ import annotations

import ctypes

import numpy as np

from . import bf16_round, lib, variant_hparams


def tensors(cfg):
    """[(name, K, N)] of the net described by cfg (keys C, stem, blocks, classes)."""
    out = [("stem", 9 * cfg["C"], cfg["stem"])]
    c = cfg["stem"]
    for i, (s, co) in enumerate(cfg["blocks"]):
        out.append((f"dw{i}", 9, c))
        out.append((f"pw{i}", c, co))
        c = co
    out.append(("fc", c, cfg["classes"]))
    return out


def param_count(cfg):
    return sum(K * N + N for _, K, N in tensors(cfg))


def unpack(params, cfg):
    """{name: (W [K][N], b [N])} views of a canonical parameter vector."""
    out, off = {}, 0
    for name, K, N in tensors(cfg):
        W = params[off:off + K * N].reshape(K, N)
        b = params[off + K * N:off + K * N + N]
        out[name] = (W, b)
        off += K * N + N
    return out


def tensor_init(seed, v, li, K, N, thresh, base_w=None, base_b=None, noise_std=0.0):
    """(W [K][N], b [N], mask [K][N]) of tensor li of variant v (C oracle)."""
    L = lib()
    W = np.zeros((K, N), np.float64)
    b = np.zeros(N, np.float64)
    M = np.zeros((K, N), np.uint8)
    kind = 1 if base_w is not None else 0
    bw = np.ascontiguousarray(base_w, np.float64) if base_w is not None else None
    bb = np.ascontiguousarray(base_b, np.float64) if base_b is not None else None
    f64p = ctypes.POINTER(ctypes.c_double)
    rc = L.or_tensor_init(seed, v, li, K, N, thresh, kind,
                          bw.ctypes.data_as(f64p) if bw is not None else None,
                          bb.ctypes.data_as(f64p) if bb is not None else None, float(noise_std),
                          W.ctypes.data_as(f64p), b.ctypes.data_as(f64p),
                          M.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)))
    assert rc == 0
    return W, b, M


def thresholds(cfg, variants):
    """Mask thresholds T_v = round(rho_v 2^24) of the variants (rho_v drawn as
    for the fully connected populations, from cfg["dens"])."""
    return [variant_hparams(cfg["seed"], v, (1e-3, 1e-3), cfg.get("dens", (1.0, 1.0)))[2] for v in variants]


def variant_params(cfg, base, v, thresh):
    """Canonical parameters and mask of variant v from the base parameters."""
    parts, masks = [], []
    for li, ((name, K, N), (Wb, bb)) in enumerate(zip(tensors(cfg), unpack(base, cfg).values())):
        W, b, M = tensor_init(cfg["seed"], v, li, K, N, thresh, Wb, bb, cfg.get("noise_std", 0.0))
        parts += [W.ravel(), b]
        masks.append(M.ravel())
    return np.concatenate(parts), np.concatenate(masks)


def _r(x, mode):
    # to bfloat16 (through binary32; the GPU rounds binary32 accumulators)
    return bf16_round(x).astype(np.float64) if mode == "bf16" else np.asarray(x, np.float64)


def softmax_stats(z, y):
    """(sum of cross-entropies lse(z) - z_y, number of rows whose first maximal
    logit is the label) of logits z [n][classes], fp64."""
    z = np.asarray(z, np.float64)
    m = z.max(axis=1)
    lse = np.log(np.exp(z - m[:, None]).sum(axis=1)) + m
    ce = lse - z[np.arange(len(y)), y]
    return float(ce.sum()), int((z.argmax(axis=1) == y).sum())


def conv3x3_depthwise(a, w, stride):
    """a [n][H][W][C], w [9][C] (tap 3 dy + dx): zero padding 1, stride s;
    out[n][yo][xo][c] = sum_{dy,dx} a[n][s yo + dy - 1][s xo + dx - 1][c] w[3 dy + dx][c]."""
    n, H, Wd, C = a.shape
    Ho, Wo = (H - 1) // stride + 1, (Wd - 1) // stride + 1
    ap = np.zeros((n, H + 2, Wd + 2, C), np.float64)
    ap[:, 1:H + 1, 1:Wd + 1, :] = a
    out = np.zeros((n, Ho, Wo, C), np.float64)
    for dy in range(3):
        for dx in range(3):
            win = ap[:, dy:dy + stride * (Ho - 1) + 1:stride, dx:dx + stride * (Wo - 1) + 1:stride, :]
            out += win * w[3 * dy + dx]
    return out


def conv3x3_full(a, w):
    """a [n][H][W][C], w [9C][N] (row (3 dy + dx) C + c): stride 1, zero
    padding 1; out[n][y][x][m] = sum_{dy,dx,c} a[n][y+dy-1][x+dx-1][c] w[(3dy+dx)C + c][m]."""
    n, H, Wd, C = a.shape
    ap = np.zeros((n, H + 2, Wd + 2, C), np.float64)
    ap[:, 1:H + 1, 1:Wd + 1, :] = a
    out = np.zeros((n, H, Wd, w.shape[1]), np.float64)
    for dy in range(3):
        for dx in range(3):
            t = 3 * dy + dx
            out += ap[:, dy:dy + H, dx:dx + Wd, :] @ w[t * C:(t + 1) * C, :]
    return out


def removed_depthwise(a, stride):
    """A removed depthwise layer (section 6.1 removes a convolution layer of
    MobileNet): its output is its input, repaired to the shape the next layer
    expects (section 4.1 shrinks or pads tensors) -- at stride s, the pixels
    (s yo, s xo), the centres of the windows the layer would have read."""
    return a[:, ::stride, ::stride, :]


def removed_pointwise(a, c_out):
    """A removed pointwise layer: its output is its input, repaired to c_out
    channels -- the first c_out channels kept (values dropped at the tensor's
    far edge), or channels of value 1 appended (section 4.1 pads with 1)."""
    n, H, Wd, C = a.shape
    if C >= c_out:
        return a[..., :c_out]
    return np.concatenate([a, np.ones((n, H, Wd, c_out - C), a.dtype)], axis=3)


def forward_logits(cfg, params, x, mode="bf16", removed=()):
    """Logits [n][classes] of images x [n][H][W][C] (values as given, fp32).
    removed: names ("dw<i>", "pw<i>") of the block layers taken out of the
    net (their parameters are then ignored)."""
    p = unpack(np.asarray(params, np.float64), cfg)
    a = _r(x.astype(np.float32), mode)
    W, b = p["stem"]
    a = _r(np.maximum(conv3x3_full(a, _r(W, mode)) + b, 0.0), mode)
    for i, (s, co) in enumerate(cfg["blocks"]):
        if f"dw{i}" in removed:
            a = removed_depthwise(a, s)
        else:
            W, b = p[f"dw{i}"]
            a = _r(np.maximum(conv3x3_depthwise(a, _r(W, mode), s) + b, 0.0), mode)
        if f"pw{i}" in removed:
            a = removed_pointwise(a, co)
        else:
            W, b = p[f"pw{i}"]
            a = _r(np.maximum(a @ _r(W, mode) + b, 0.0), mode)
    h = _r(a.mean(axis=(1, 2)), mode)
    W, b = p["fc"]
    return h @ _r(W, mode) + b


def evaluate(cfg, base, x, y, variants, mode="bf16", chunk=256, removed=None):
    """{v: (test CE sum, correct count)} over images x [n][H][W][C], labels y.
    removed: optional {v: names of the block layers variant v has removed}."""
    out = {}
    for v in variants:
        th = thresholds(cfg, [v])[0]
        params, _ = variant_params(cfg, base, v, th)
        gone = (removed or {}).get(v, ())
        ce, corr = 0.0, 0
        for c0 in range(0, len(y), chunk):
            z = forward_logits(cfg, params, x[c0:c0 + chunk], mode, gone)
            c, k = softmax_stats(z, y[c0:c0 + chunk])
            ce += c
            corr += k
        out[v] = (ce, corr)
    return out
