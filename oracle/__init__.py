"""CPU oracle for population-batched fitness evaluation (GEVO-ML, arXiv 2310.10211).

TEST INFRASTRUCTURE ONLY.  A plain, slow, obviously correct CPU implementation
(``gevo_oracle.c``, built with gcc, loaded with ctypes) of what the GPU library
computes.  Only the test-suite, the smoke check and the CPU-baseline leg of the
benchmark may import it.  It shares no code with the HIP library and imports
nothing from the product package.

Everything here is argument marshalling around the C functions; each C function
cites the passage of the paper it follows (section 4 for the population,
section 4.3 for the two fitness workloads, section 6.2 for the SGD update).

Parity status per function:
  philox                pinned by the published known-answer vectors of
                        Philox4x32-10 (tests/golden/philox4x32_10_kat.txt)
  variant_hparams/init  pinned by distribution tests (binomial density band,
                        log-uniform range, Xavier bound), by the KAT-pinned RNG
  permutation           pinned: is a permutation, Fisher-Yates brute-force
                        replay in pure Python on small n
  batch_grad            pinned by finite differences (fp64), by the
                        hand-computed 2-3-2 example (tests/golden), by PyTorch
                        CPU autograd in fp64
  train_steps           pinned by the 2-3-2 example after one step, by lr=0,
                        mask, batch-size-1 and mean-vs-sum invariants and by a
                        PyTorch CPU SGD replay in fp64
  predict               pinned by a brute-force numpy forward and constructed
                        argmax ties
  bf16 emulation        pinned by exhaustive/edge-value checks against the
                        definition of round-to-nearest-even
  bf16 rounding points  one hand-built net per point (X, W in the forward and
                        in G_l W_l^T, A after ReLU, G_l as an operand, hidden
                        bias gradient from the rounded G_l), each with only
                        that value off the bf16 grid; a mutation test rebuilds
                        the oracle with each point removed and checks that a
                        pin fails (tests/test_oracle_bf16_points.py)
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gevo_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libgevo_oracle.so")

F64, F32, BF16 = 0, 1, 2
MODES = {"f64": F64, "f32": F32, "bf16": BF16}

_lib = None
_lock = threading.Lock()


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no fast-math, no FMA contraction)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-ffp-contract=off", "-fno-fast-math",
               "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    with _lock:
        if _lib is None:
            build(force=False)
            L = ctypes.CDLL(_LIB_PATH)
            u32p = ctypes.POINTER(ctypes.c_uint32)
            f64p = ctypes.POINTER(ctypes.c_double)
            f32p = ctypes.POINTER(ctypes.c_float)
            i32p = ctypes.POINTER(ctypes.c_int32)
            u8p = ctypes.POINTER(ctypes.c_uint8)
            u64p = ctypes.POINTER(ctypes.c_uint64)
            L.or_philox4x32_10.argtypes = [u32p, u32p, u32p]
            L.or_philox4x32_10.restype = None
            L.or_bf16_round_array.argtypes = [f32p, f32p, ctypes.c_size_t]
            L.or_bf16_round_array.restype = None
            L.or_param_count.argtypes = [ctypes.c_int, u32p]
            L.or_param_count.restype = ctypes.c_size_t
            L.or_weight_count.argtypes = [ctypes.c_int, u32p]
            L.or_weight_count.restype = ctypes.c_size_t
            L.or_variant_hparams.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_float, ctypes.c_float,
                                             ctypes.c_float, ctypes.c_float, f32p, ctypes.c_uint32,
                                             f32p, f32p, u32p]
            L.or_variant_init.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int, u32p, ctypes.c_uint32,
                                          ctypes.c_int, f64p, ctypes.c_float, f64p, u8p]
            L.or_tensor_init.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32,
                                         ctypes.c_uint32, ctypes.c_uint32, ctypes.c_int, f64p, f64p, ctypes.c_float,
                                         f64p, f64p, u8p]
            L.or_genome_mask.argtypes = [ctypes.c_uint64, ctypes.c_int, u32p, ctypes.c_uint32, u32p, u32p, u8p]
            L.or_permutation.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32, u32p]
            L.or_permutation.restype = None
            L.or_batch_grad.argtypes = [ctypes.c_int, ctypes.c_int, u32p, f64p, f32p, i32p, ctypes.c_uint32,
                                        ctypes.c_double, f32p, f64p, f64p, f64p, f64p]
            L.or_structure_masks.argtypes = [ctypes.c_int, u32p, u32p, u8p, u8p, u8p]
            L.or_train_steps.argtypes = [ctypes.c_int, ctypes.c_int, u32p, f64p, u8p, u8p, ctypes.c_uint32,
                                         ctypes.c_float, f32p, i32p,
                                         ctypes.c_uint32, u32p, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32,
                                         f32p, f64p, u64p]
            L.or_predict.argtypes = [ctypes.c_int, ctypes.c_int, u32p, f64p, f32p, i32p, ctypes.c_uint32,
                                     f64p, u64p]
            _lib = L
    return _lib


def _p(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _dims(dims):
    return np.ascontiguousarray(np.asarray(dims, dtype=np.uint32))


def _mode(mode):
    return MODES[mode] if isinstance(mode, str) else int(mode)


# --------------------------------------------------------------------------- RNG
def philox(ctr, key):
    c = np.ascontiguousarray(np.asarray(ctr, dtype=np.uint32))
    k = np.ascontiguousarray(np.asarray(key, dtype=np.uint32))
    out = np.zeros(4, dtype=np.uint32)
    lib().or_philox4x32_10(_p(c, ctypes.c_uint32), _p(k, ctypes.c_uint32), _p(out, ctypes.c_uint32))
    return out


def bf16_round(x):
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    out = np.empty_like(x)
    lib().or_bf16_round_array(_p(x, ctypes.c_float), _p(out, ctypes.c_float), x.size)
    return out


def param_count(dims):
    d = _dims(dims)
    return int(lib().or_param_count(len(d) - 1, _p(d, ctypes.c_uint32)))


def weight_count(dims):
    d = _dims(dims)
    return int(lib().or_weight_count(len(d) - 1, _p(d, ctypes.c_uint32)))


def unpack(params, dims):
    """Views [(W_1, b_1), ...] of a canonical parameter vector (W_l is in x out)."""
    out, off = [], 0
    for l in range(1, len(dims)):
        din, dout = int(dims[l - 1]), int(dims[l])
        W = params[off:off + din * dout].reshape(din, dout)
        off += din * dout
        b = params[off:off + dout]
        off += dout
        out.append((W, b))
    return out


def unpack_mask(mask, dims):
    out, off = [], 0
    for l in range(1, len(dims)):
        din, dout = int(dims[l - 1]), int(dims[l])
        out.append(mask[off:off + din * dout].reshape(din, dout))
        off += din * dout
    return out


def variant_hparams(seed, v, lr_range, dens_range=(1.0, 1.0), dens_list=None):
    lr = ctypes.c_float()
    dens = ctypes.c_float()
    th = ctypes.c_uint32()
    if dens_list is not None and len(dens_list) > 0:
        dl = np.ascontiguousarray(np.asarray(dens_list, dtype=np.float32))
        dlp, nl = _p(dl, ctypes.c_float), len(dl)
    else:
        dl, dlp, nl = None, None, 0
    rc = lib().or_variant_hparams(ctypes.c_uint64(seed), v, float(lr_range[0]), float(lr_range[1]),
                                  float(dens_range[0]), float(dens_range[1]), dlp, nl,
                                  ctypes.byref(lr), ctypes.byref(dens), ctypes.byref(th))
    assert rc == 0
    return np.float32(lr.value), np.float32(dens.value), int(th.value)


def variant_init(seed, v, dims, thresh, init_kind=0, base=None, noise_std=0.0):
    """Returns (params float64 canonical, mask uint8 over weights)."""
    d = _dims(dims)
    params = np.zeros(param_count(dims), dtype=np.float64)
    mask = np.zeros(weight_count(dims), dtype=np.uint8)
    bp = None
    if base is not None:
        base = np.ascontiguousarray(np.asarray(base, dtype=np.float64))
        assert base.size == params.size
        bp = _p(base, ctypes.c_double)
    rc = lib().or_variant_init(ctypes.c_uint64(seed), v, len(d) - 1, _p(d, ctypes.c_uint32), thresh,
                               init_kind, bp, float(noise_std), _p(params, ctypes.c_double),
                               _p(mask, ctypes.c_uint8))
    assert rc == 0
    return params, mask


def genome_mask(seed, dims, edit_ids, thresholds):
    """Mask (uint8 over weights, canonical order) of an individual whose pruning
    edits are (edit_ids[i], thresholds[i]): a weight is kept when every edit keeps it."""
    d = _dims(dims)
    ids = np.ascontiguousarray(np.asarray(edit_ids, dtype=np.uint32))
    th = np.ascontiguousarray(np.asarray(thresholds, dtype=np.uint32))
    assert ids.shape == th.shape
    mask = np.zeros(weight_count(dims), dtype=np.uint8)
    rc = lib().or_genome_mask(ctypes.c_uint64(seed), len(d) - 1, _p(d, ctypes.c_uint32), len(ids),
                              _p(ids, ctypes.c_uint32), _p(th, ctypes.c_uint32), _p(mask, ctypes.c_uint8))
    assert rc == 0
    return mask


def permutation(seed, epoch, n):
    out = np.zeros(n, dtype=np.uint32)
    lib().or_permutation(ctypes.c_uint64(seed), epoch, n, _p(out, ctypes.c_uint32))
    return out


# ------------------------------------------------------------------ train / eval
def _gscale(gscale, rows, C):
    if gscale is None:
        return None, None
    g = np.ascontiguousarray(np.asarray(gscale, dtype=np.float32))
    assert g.shape == (rows, C), g.shape
    return g, _p(g, ctypes.c_float)


def batch_grad(mode, dims, params, X, y, scale=0.0, gscale=None):
    """Loss sum, gradients (canonical layout), logits and probabilities of one
    batch; gscale ([b][C], optional) replaces the scalar gradient scale."""
    d = _dims(dims)
    X = np.ascontiguousarray(np.asarray(X, dtype=np.float32))
    y = np.ascontiguousarray(np.asarray(y, dtype=np.int32))
    params = np.ascontiguousarray(np.asarray(params, dtype=np.float64))
    b = y.shape[0]
    grads = np.zeros_like(params)
    ce = ctypes.c_double()
    logits = np.zeros((b, int(d[-1])), dtype=np.float64)
    probs = np.zeros((b, int(d[-1])), dtype=np.float64)
    gs, gsp = _gscale(gscale, b, int(d[-1]))
    rc = lib().or_batch_grad(_mode(mode), len(d) - 1, _p(d, ctypes.c_uint32), _p(params, ctypes.c_double),
                             _p(X, ctypes.c_float), _p(y, ctypes.c_int32), b, float(scale), gsp,
                             _p(grads, ctypes.c_double), ctypes.byref(ce), _p(logits, ctypes.c_double),
                             _p(probs, ctypes.c_double))
    assert rc == 0, rc
    return ce.value, grads, logits, probs


def structure_masks(dims, widths, bias_keep, mask=None):
    """(weight mask, bias mask) of structural edits: layer l keeps its first
    widths[l] units and its bias when bias_keep[l-1]; mask (optional) is the
    weight mask to narrow."""
    d = _dims(dims)
    L = len(d) - 1
    w = np.ascontiguousarray(np.asarray(widths, dtype=np.uint32))
    bk = np.ascontiguousarray(np.asarray(bias_keep, dtype=np.uint8))
    assert w.size == L + 1 and bk.size == L
    m = np.ones(weight_count(dims), np.uint8) if mask is None else np.array(mask, dtype=np.uint8, copy=True)
    bm = np.zeros(int(sum(d[1:])), np.uint8)
    rc = lib().or_structure_masks(L, _p(d, ctypes.c_uint32), _p(w, ctypes.c_uint32), _p(bk, ctypes.c_uint8),
                                  _p(m, ctypes.c_uint8), _p(bm, ctypes.c_uint8))
    assert rc == 0
    return m, bm


def removed_layer_form(dims, widths, l):
    """The identity form of hidden layer l removed from a net whose layers
    keep widths[0..L] units (sections 6.1 and 4.1): (W [d_{l-1}][d_l], b
    [d_l], mask uint8 [d_{l-1}][d_l]).  Unit n passes kept input n on
    (W[n][n] = 1, n < min(widths[l-1], widths[l])); units widths[l-1] ..
    widths[l]-1, when the layer is wider than its kept input, hold the value
    1 (no weights, bias 1: the repair pads with 1); everything else is +0.
    With ReLU on non-negative inputs the layer passes its input on exactly."""
    d = [int(x) for x in dims]
    K, N = d[l - 1], d[l]
    W = np.zeros((K, N), np.float64)
    b = np.zeros(N, np.float64)
    m = min(int(widths[l - 1]), int(widths[l]))
    W[np.arange(m), np.arange(m)] = 1.0
    b[int(widths[l - 1]):int(widths[l])] = 1.0
    return W, b, (W != 0).astype(np.uint8)


def train_steps(mode, dims, params, mask, lr, X, y, perm, batch, t0, t1, gscale=None, bmask=None, frozen=0):
    """In-place SGD steps [t0, t1) on ``params``; returns (ce_sum, correct).
    gscale ([batch][C], optional): row i scales the output gradient of row i of
    every batch in place of fl(1/b_t).  bmask (over all biases, optional):
    biases with 0 stay +0.  frozen: bit l-1 set -> layer l updates with
    learning rate 0 (a removed layer)."""
    d = _dims(dims)
    assert params.dtype == np.float64 and params.flags.c_contiguous
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    X = np.ascontiguousarray(X, dtype=np.float32)
    y = np.ascontiguousarray(y, dtype=np.int32)
    perm = np.ascontiguousarray(perm, dtype=np.uint32)
    ce = ctypes.c_double(0.0)
    corr = ctypes.c_uint64(0)
    gs, gsp = _gscale(gscale, batch, int(d[-1]))
    bm = None if bmask is None else np.ascontiguousarray(bmask, dtype=np.uint8)
    rc = lib().or_train_steps(_mode(mode), len(d) - 1, _p(d, ctypes.c_uint32), _p(params, ctypes.c_double),
                              _p(mask, ctypes.c_uint8), None if bm is None else _p(bm, ctypes.c_uint8), int(frozen),
                              float(lr), _p(X, ctypes.c_float), _p(y, ctypes.c_int32),
                              y.shape[0], _p(perm, ctypes.c_uint32), batch, t0, t1, gsp,
                              ctypes.byref(ce), ctypes.byref(corr))
    assert rc == 0, rc
    return ce.value, corr.value


def predict(mode, dims, params, X, y):
    d = _dims(dims)
    params = np.ascontiguousarray(params, dtype=np.float64)
    X = np.ascontiguousarray(X, dtype=np.float32)
    y = np.ascontiguousarray(y, dtype=np.int32)
    ce = ctypes.c_double(0.0)
    corr = ctypes.c_uint64(0)
    rc = lib().or_predict(_mode(mode), len(d) - 1, _p(d, ctypes.c_uint32), _p(params, ctypes.c_double),
                          _p(X, ctypes.c_float), _p(y, ctypes.c_int32), y.shape[0],
                          ctypes.byref(ce), ctypes.byref(corr))
    assert rc == 0, rc
    return ce.value, corr.value


# ------------------------------------------------------------ whole population
def population(cfg, variants=None, base=None):
    """Per-variant (lr, density, threshold, params, mask) for a config dict with
    keys dims, seed, lr, and dens or dens_list, optional init/noise_std."""
    P = cfg["P"]
    variants = range(P) if variants is None else variants
    init_kind = 1 if cfg.get("init", "xavier") == "base_noise" else 0
    out = {}
    for v in variants:
        lr, dens, th = variant_hparams(cfg["seed"], v, cfg["lr"], cfg.get("dens", (1.0, 1.0)),
                                       cfg.get("dens_list"))
        params, mask = variant_init(cfg["seed"], v, cfg["dims"], th, init_kind, base,
                                    cfg.get("noise_std", 0.0))
        out[v] = dict(lr=lr, density=dens, thresh=th, params=params, mask=mask)
    return out


def evaluate(cfg, data, variants=None, epochs=None, mode=None, threads=None, steps=None, base=None,
             do_predict=True):
    """Fitness evaluation of the listed variants, one variant per thread.

    Training configs: ``epochs`` epochs of SGD (``steps`` limits epoch 0 to its
    first steps, for bounded samples), then prediction on the test split.
    Returns {v: dict(train_loss=[per epoch], train_acc=[...], test_loss, test_acc,
    params, mask, lr, density)}.
    """
    mode = _mode(mode if mode is not None else cfg["dtype"])
    pop = population(cfg, variants, base)
    epochs = cfg.get("epochs", 1) if epochs is None else epochs
    Xtr, ytr, Xte, yte = data["x_train"], data["y_train"], data["x_test"], data["y_test"]
    n = ytr.shape[0]
    B = cfg.get("batch", 1)
    T = (n + B - 1) // B
    perms = [permutation(cfg["seed"], e, n) for e in range(epochs)]

    def run(v):
        st = pop[v]
        tl, ta = [], []
        for e in range(epochs):
            t1 = T if steps is None else min(T, steps)
            ce, corr = train_steps(mode, cfg["dims"], st["params"], st["mask"], st["lr"], Xtr, ytr,
                                   perms[e], B, 0, t1)
            nrows = min(n, t1 * B)
            tl.append(ce / nrows)
            ta.append(corr / nrows)
        st["train_loss"], st["train_acc"] = tl, ta
        if do_predict:
            ce, corr = predict(mode, cfg["dims"], st["params"], Xte, yte)
            st["test_loss"] = ce / yte.shape[0]
            st["test_acc"] = corr / yte.shape[0]
        return v

    threads = threads or min(len(pop), os.cpu_count() or 1)
    if threads <= 1:
        for v in pop:
            run(v)
    else:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            list(ex.map(run, list(pop)))
    return pop
