"""Python binding of libgevo: population-batched fitness evaluation on MI355X.

Argument marshalling only.  Every step of evaluation runs in the HIP kernels of
``libgevo.so`` behind the C-ABI declared in ``include/gevo.h``; PyTorch is used
for device memory (datasets, workspace) and the stream.  There is no CPU
fallback: without the built library, importing ``Population`` fails loudly.

GEVO-ML (arXiv 2310.10211) evaluates every individual of its population by
retraining its model on the dataset or by running it over the dataset, scoring
time and error (section 4.3).  A ``Population`` holds P variants of a small
fully-connected classifier, each the original model with its own learning rate
and weight-pruning mask (the effects the paper attributes to its mutations,
section 6.2 and the abstract).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

__all__ = ["Population", "lib", "epoch_permutation", "check_bf16_rounding", "GevoError", "config_struct",
           "workspace_bytes", "nsga2_rank", "nsga2_select", "genomes_initial", "genomes_breed", "EDIT_LR",
           "EDIT_PRUNE", "EDIT_WIDTH", "EDIT_BIAS_OFF", "EDIT_LAYER_OFF"]

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgevo.so")

GEVO_ABI_VERSION = 1
MAX_LAYERS = 3
F32, BF16 = 0, 1
INIT_XAVIER, INIT_BASE_NOISE = 0, 1

EXPORTED = [
    "gevo_pop_workspace_bytes", "gevo_pop_init", "gevo_pop_train_epoch", "gevo_pop_train_steps",
    "gevo_pop_steps_per_epoch", "gevo_pop_predict", "gevo_pop_predict_noalloc", "gevo_pop_scores",
    "gevo_pop_last_time",
    "gevo_pop_export", "gevo_pop_import", "gevo_pop_epoch_labels", "gevo_epoch_permutation",
    "gevo_pop_set_profiling", "gevo_pop_kernel_stats", "gevo_pop_destroy", "gevo_status_str",
    "gevo_check_bf16_rounding", "gevo_nsga2_rank", "gevo_nsga2_select", "gevo_genomes_initial",
    "gevo_genomes_breed", "gevo_pop_set_genomes", "gevo_pop_set_grad_scale",
    "gevo_cnn_param_count", "gevo_cnn_workspace_bytes", "gevo_cnn_init", "gevo_cnn_predict", "gevo_cnn_scores",
    "gevo_cnn_export", "gevo_cnn_remove_layer", "gevo_cnn_destroy", "gevo_cnn_set_profiling", "gevo_cnn_kernel_stats",
]
CNN_MAX_BLOCKS = 4
CNN_KERNEL_KINDS = ["stem", "depthwise", "pointwise", "pool", "head", "reduce", "pw_dw"]
KERNEL_KINDS = ["init", "gather", "layer_train", "layer_fwd", "out_train", "out_predict", "bwd", "aux",
                "fused_train", "weight_copy", "fwd_out"]


class GevoError(RuntimeError):
    pass


class GevoEdit(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_uint32), ("id", ctypes.c_uint32), ("value", ctypes.c_uint32)]


EDIT_LR, EDIT_PRUNE, EDIT_WIDTH, EDIT_BIAS_OFF, EDIT_LAYER_OFF = 0, 1, 2, 3, 4


class GevoCnnConfig(ctypes.Structure):
    _fields_ = [
        ("abi_version", ctypes.c_uint32), ("P", ctypes.c_uint32),
        ("height", ctypes.c_uint32), ("width", ctypes.c_uint32), ("channels", ctypes.c_uint32),
        ("stem_channels", ctypes.c_uint32), ("n_blocks", ctypes.c_uint32),
        ("block_stride", ctypes.c_uint32 * CNN_MAX_BLOCKS), ("block_channels", ctypes.c_uint32 * CNN_MAX_BLOCKS),
        ("classes", ctypes.c_uint32), ("seed", ctypes.c_uint64),
        ("dens_lo", ctypes.c_float), ("dens_hi", ctypes.c_float), ("noise_rel_std", ctypes.c_float),
    ]


def cnn_config_struct(cfg: dict) -> GevoCnnConfig:
    """cfg keys: P, H, W, C, stem, blocks [(stride, channels)], classes, seed,
    dens (lo, hi), noise_std."""
    c = GevoCnnConfig()
    c.abi_version = 1
    c.P = cfg["P"]
    c.height, c.width, c.channels = cfg["H"], cfg["W"], cfg["C"]
    c.stem_channels = cfg["stem"]
    c.n_blocks = len(cfg["blocks"])
    for i, (st, ch) in enumerate(cfg["blocks"][:CNN_MAX_BLOCKS]):
        c.block_stride[i], c.block_channels[i] = st, ch
    c.classes = cfg["classes"]
    c.seed = cfg["seed"]
    c.dens_lo, c.dens_hi = cfg.get("dens", (1.0, 1.0))
    c.noise_rel_std = cfg.get("noise_std", 0.0)
    return c


class GevoPopConfig(ctypes.Structure):
    _fields_ = [
        ("abi_version", ctypes.c_uint32),
        ("n_layers", ctypes.c_uint32),
        ("dims", ctypes.c_uint32 * (MAX_LAYERS + 1)),
        ("P", ctypes.c_uint32),
        ("batch", ctypes.c_uint32),
        ("dtype", ctypes.c_int),
        ("seed", ctypes.c_uint64),
        ("lr_lo", ctypes.c_float),
        ("lr_hi", ctypes.c_float),
        ("dens_lo", ctypes.c_float),
        ("dens_hi", ctypes.c_float),
        ("dens_list", ctypes.POINTER(ctypes.c_float)),
        ("n_dens_list", ctypes.c_uint32),
        ("init", ctypes.c_int),
        ("base_params", ctypes.POINTER(ctypes.c_float)),
        ("noise_rel_std", ctypes.c_float),
        ("n_train", ctypes.c_int64),
        ("n_test", ctypes.c_int64),
    ]


_lib = None


def lib():
    """Load libgevo.so (built by __graft_entry__.build()); raises if missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        vp, u32, i64 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_int64
        f32p = ctypes.POINTER(ctypes.c_float)
        cfgp = ctypes.POINTER(GevoPopConfig)
        L.gevo_pop_workspace_bytes.argtypes = [cfgp, ctypes.POINTER(ctypes.c_size_t)]
        L.gevo_pop_init.argtypes = [cfgp, vp, ctypes.c_size_t, vp, vp, vp, vp, vp, ctypes.POINTER(vp)]
        L.gevo_pop_train_epoch.argtypes = [vp, u32]
        L.gevo_pop_train_steps.argtypes = [vp, u32, u32, u32]
        L.gevo_pop_steps_per_epoch.argtypes = [vp, ctypes.POINTER(u32)]
        L.gevo_pop_predict.argtypes = [vp]
        L.gevo_pop_predict_noalloc.argtypes = [vp]
        L.gevo_pop_scores.argtypes = [vp, f32p, f32p, f32p, f32p, f32p]
        L.gevo_pop_last_time.argtypes = [vp, ctypes.POINTER(ctypes.c_double)]
        L.gevo_pop_export.argtypes = [vp, u32, f32p, ctypes.POINTER(ctypes.c_uint8), f32p, f32p]
        L.gevo_pop_import.argtypes = [vp, u32, f32p]
        L.gevo_pop_epoch_labels.argtypes = [vp, ctypes.POINTER(ctypes.c_int32), i64]
        L.gevo_epoch_permutation.argtypes = [ctypes.c_uint64, u32, u32, ctypes.POINTER(u32)]
        L.gevo_pop_set_profiling.argtypes = [vp, ctypes.c_int]
        L.gevo_pop_kernel_stats.argtypes = [vp, ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                            ctypes.POINTER(ctypes.c_uint64)]
        L.gevo_check_bf16_rounding.argtypes = [vp, vp]
        u32p, f64p = ctypes.POINTER(u32), ctypes.POINTER(ctypes.c_double)
        editp = ctypes.POINTER(GevoEdit)
        L.gevo_nsga2_rank.argtypes = [u32, u32, f64p, u32p, f64p]
        L.gevo_nsga2_select.argtypes = [u32, u32p, f64p, u32, u32, ctypes.c_uint64, u32, u32p]
        L.gevo_genomes_initial.argtypes = [u32, u32, ctypes.c_uint64, ctypes.c_double, u32, ctypes.c_double, u32,
                                           u32p, editp]
        L.gevo_genomes_breed.argtypes = [u32, u32p, editp, ctypes.c_uint64, u32, ctypes.c_double, ctypes.c_double,
                                         ctypes.c_double, u32, u32, ctypes.c_double, u32, u32p, u32p, editp,
                                         ctypes.c_size_t]
        L.gevo_pop_set_genomes.argtypes = [vp, ctypes.c_float, u32p, editp, f32p, f64p]
        L.gevo_pop_set_grad_scale.argtypes = [vp, f32p]
        ccfgp = ctypes.POINTER(GevoCnnConfig)
        L.gevo_cnn_param_count.argtypes = [ccfgp, ctypes.POINTER(ctypes.c_size_t)]
        L.gevo_cnn_workspace_bytes.argtypes = [ccfgp, i64, ctypes.POINTER(ctypes.c_size_t)]
        L.gevo_cnn_init.argtypes = [ccfgp, vp, ctypes.c_size_t, f32p, vp, vp, i64, vp, ctypes.POINTER(vp)]
        L.gevo_cnn_predict.argtypes = [vp]
        L.gevo_cnn_scores.argtypes = [vp, f32p, f32p, f32p]
        L.gevo_cnn_export.argtypes = [vp, u32, f32p, ctypes.POINTER(ctypes.c_uint8), f32p]
        L.gevo_cnn_remove_layer.argtypes = [vp, u32, u32]
        L.gevo_cnn_set_profiling.argtypes = [vp, ctypes.c_int]
        L.gevo_cnn_kernel_stats.argtypes = [vp, ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                            ctypes.POINTER(ctypes.c_uint64)]
        L.gevo_cnn_destroy.argtypes = [vp]
        L.gevo_cnn_destroy.restype = None
        L.gevo_pop_destroy.argtypes = [vp]
        L.gevo_pop_destroy.restype = None
        L.gevo_status_str.argtypes = [ctypes.c_int]
        L.gevo_status_str.restype = ctypes.c_char_p
        for name in EXPORTED:
            if name not in ("gevo_pop_destroy", "gevo_status_str"):
                getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(rc, what):
    if rc != 0:
        raise GevoError(f"{what}: {lib().gevo_status_str(rc).decode()} ({rc})")


def _fp(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def config_struct(cfg: dict, n_train: int, n_test: int, keep: list):
    """GevoPopConfig from a workload dict (keys: dims, P, batch, dtype, seed, lr,
    dens or dens_list, init, noise_std, base_params)."""
    c = GevoPopConfig()
    dims = list(cfg["dims"])
    c.abi_version = GEVO_ABI_VERSION
    c.n_layers = len(dims) - 1
    for i in range(min(len(dims), MAX_LAYERS + 1)):
        c.dims[i] = dims[i]
    c.P = cfg["P"]
    c.batch = cfg.get("batch", 1)
    c.dtype = BF16 if cfg.get("dtype", "f32") == "bf16" else F32
    c.seed = cfg["seed"]
    c.lr_lo, c.lr_hi = cfg.get("lr", (0.0, 0.0))
    if cfg.get("dens_list"):
        dl = np.ascontiguousarray(np.asarray(cfg["dens_list"], np.float32))
        keep.append(dl)
        c.dens_list = _fp(dl)
        c.n_dens_list = dl.size
    else:
        c.dens_lo, c.dens_hi = cfg.get("dens", (1.0, 1.0))
    c.init = INIT_BASE_NOISE if cfg.get("init", "xavier") == "base_noise" else INIT_XAVIER
    if cfg.get("base_params") is not None:
        bp = np.ascontiguousarray(np.asarray(cfg["base_params"], np.float32))
        keep.append(bp)
        c.base_params = _fp(bp)
    c.noise_rel_std = cfg.get("noise_std", 0.0)
    c.n_train = n_train
    c.n_test = n_test
    return c


def workspace_bytes(cfg: dict, n_train: int, n_test: int) -> int:
    keep = []
    c = config_struct(cfg, n_train, n_test, keep)
    out = ctypes.c_size_t()
    _check(lib().gevo_pop_workspace_bytes(ctypes.byref(c), ctypes.byref(out)), "gevo_pop_workspace_bytes")
    return out.value


def epoch_permutation(seed: int, epoch: int, n: int) -> np.ndarray:
    out = np.zeros(n, np.uint32)
    _check(lib().gevo_epoch_permutation(seed, epoch, n, out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))),
           "gevo_epoch_permutation")
    return out


def check_bf16_rounding(stream=None) -> list:
    """Per operand pairing, the number of binary32 encodings whose kernel bf16
    rounding differs from round-to-nearest-even (see gevo_check_bf16_rounding)."""
    import torch
    counts = torch.zeros(2, dtype=torch.int64, device="cuda")
    st = stream if stream is not None else torch.cuda.current_stream()
    _check(lib().gevo_check_bf16_rounding(ctypes.c_void_p(st.cuda_stream), ctypes.c_void_p(counts.data_ptr())),
           "gevo_check_bf16_rounding")
    return [int(c) for c in counts.cpu()]


def _u32p(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_uint32))


def _f64p(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _pack_genomes(genomes):
    """Flat (offsets, edits) of a list of edit lists [(kind, id, value), ...]."""
    offsets = np.zeros(len(genomes) + 1, np.uint32)
    flat = [e for g in genomes for e in g]
    edits = (GevoEdit * max(len(flat), 1))()
    for i, (kind, eid, value) in enumerate(flat):
        edits[i].kind, edits[i].id, edits[i].value = kind, eid, value
    offsets[1:] = np.cumsum([len(g) for g in genomes], dtype=np.uint64).astype(np.uint32)
    return offsets, edits


def _unpack_genomes(offsets, edits):
    return [[(edits[i].kind, edits[i].id, edits[i].value) for i in range(int(offsets[v]), int(offsets[v + 1]))]
            for v in range(len(offsets) - 1)]


def nsga2_rank(objs):
    """NSGA-II front index and crowding distance of each row of objs [n][m] (minimised)."""
    o = np.ascontiguousarray(np.asarray(objs, np.float64))
    n, m = o.shape
    rank = np.zeros(n, np.uint32)
    crowd = np.zeros(n, np.float64)
    _check(lib().gevo_nsga2_rank(n, m, _f64p(o), _u32p(rank), _f64p(crowd)), "gevo_nsga2_rank")
    return rank, crowd


def nsga2_select(rank, crowding, n_elite, n_select, seed, gen):
    """Elites (best first) followed by binary-tournament winners."""
    r = np.ascontiguousarray(np.asarray(rank, np.uint32))
    c = np.ascontiguousarray(np.asarray(crowding, np.float64))
    out = np.zeros(n_select, np.uint32)
    _check(lib().gevo_nsga2_select(len(r), _u32p(r), _f64p(c), n_elite, n_select, seed, gen, _u32p(out)),
           "gevo_nsga2_select")
    return [int(i) for i in out]


def _dims_arg(dims):
    if dims is None:
        return 0, None, None
    d = np.ascontiguousarray(np.asarray(dims, np.uint32))
    return len(d) - 1, d, _u32p(d)


def genomes_initial(n, seed, rho_lo, n_mut=3, id_base=0, struct_p=0.0, dims=None):
    """n individuals with n_mut drawn edits each (structural with probability struct_p)."""
    edits = (GevoEdit * max(n * n_mut, 1))()
    nl, keep, dp = _dims_arg(dims)
    _check(lib().gevo_genomes_initial(n, n_mut, seed, rho_lo, id_base, struct_p, nl, dp, edits),
           "gevo_genomes_initial")
    return [[(edits[n_mut * i + j].kind, edits[n_mut * i + j].id, edits[n_mut * i + j].value) for j in range(n_mut)]
            for i in range(n)]


def genomes_breed(parents, seed, gen, cxpb, mutpb, rho_lo, id_base, max_edits, struct_p=0.0, dims=None):
    """Children of the tournament winners (messy one-point crossover, mutation)."""
    off, edits = _pack_genomes(parents)
    cap = int(off[-1]) + len(parents)
    out_off = np.zeros(len(parents) + 1, np.uint32)
    out = (GevoEdit * max(cap, 1))()
    nl, keep, dp = _dims_arg(dims)
    _check(lib().gevo_genomes_breed(len(parents), _u32p(off), edits, seed, gen, cxpb, mutpb, rho_lo, id_base,
                                    max_edits, struct_p, nl, dp, _u32p(out_off), out, cap), "gevo_genomes_breed")
    return _unpack_genomes(out_off, out)


def param_count(dims) -> int:
    return sum(dims[l - 1] * dims[l] + dims[l] for l in range(1, len(dims)))


class Population:
    """P variants on one GPU; all device memory comes from torch."""

    def __init__(self, cfg: dict, x_train, y_train, x_test, y_test, device="cuda", stream=None):
        import torch
        self.torch = torch
        self.cfg = dict(cfg)
        self.dims = list(cfg["dims"])
        self.P = cfg["P"]
        dev = torch.device(device)

        def dt(a, dtype):
            t = torch.as_tensor(a)
            return t.to(device=dev, dtype=dtype).contiguous()

        self.x_train = dt(x_train, torch.float32) if x_train is not None and len(x_train) else None
        self.y_train = dt(y_train, torch.int32) if y_train is not None and len(y_train) else None
        self.x_test = dt(x_test, torch.float32)
        self.y_test = dt(y_test, torch.int32)
        n_train = 0 if self.x_train is None else self.x_train.shape[0]
        n_test = self.x_test.shape[0]
        if self.x_train is not None:
            assert self.x_train.shape == (n_train, self.dims[0]) and self.y_train.shape == (n_train,)
        assert self.x_test.shape == (n_test, self.dims[0]) and self.y_test.shape == (n_test,)
        self.n_train, self.n_test = n_train, n_test
        self._keep = []
        self._cfg = config_struct(cfg, n_train, n_test, self._keep)
        nbytes = ctypes.c_size_t()
        _check(lib().gevo_pop_workspace_bytes(ctypes.byref(self._cfg), ctypes.byref(nbytes)),
               "gevo_pop_workspace_bytes")
        self.workspace = torch.empty(max(nbytes.value, 256), dtype=torch.uint8, device=dev)
        self.stream = stream if stream is not None else torch.cuda.current_stream(dev)
        h = ctypes.c_void_p()
        ptr = lambda t: None if t is None else ctypes.c_void_p(t.data_ptr())
        _check(lib().gevo_pop_init(ctypes.byref(self._cfg), ctypes.c_void_p(self.workspace.data_ptr()),
                                   nbytes.value, ptr(self.x_train), ptr(self.y_train), ptr(self.x_test),
                                   ptr(self.y_test), ctypes.c_void_p(self.stream.cuda_stream), ctypes.byref(h)),
               "gevo_pop_init")
        self._h = h

    # --------------------------------------------------------------- workloads
    def train_epoch(self, epoch: int):
        _check(lib().gevo_pop_train_epoch(self._h, epoch), "gevo_pop_train_epoch")

    def train_steps(self, epoch: int, s0: int, s1: int):
        _check(lib().gevo_pop_train_steps(self._h, epoch, s0, s1), "gevo_pop_train_steps")

    @property
    def steps_per_epoch(self) -> int:
        out = ctypes.c_uint32()
        _check(lib().gevo_pop_steps_per_epoch(self._h, ctypes.byref(out)), "gevo_pop_steps_per_epoch")
        return out.value

    def predict(self):
        _check(lib().gevo_pop_predict(self._h), "gevo_pop_predict")

    def predict_noalloc(self):
        """gevo_pop_predict with its scratch in the library's static device array."""
        _check(lib().gevo_pop_predict_noalloc(self._h), "gevo_pop_predict_noalloc")

    def scores(self) -> dict:
        arrs = {k: np.zeros(self.P, np.float32) for k in ("train_loss", "train_acc", "test_loss", "test_acc", "time_s")}
        _check(lib().gevo_pop_scores(self._h, *[_fp(arrs[k]) for k in
                                               ("train_loss", "train_acc", "test_loss", "test_acc", "time_s")]),
               "gevo_pop_scores")
        return arrs

    def last_time(self) -> float:
        s = ctypes.c_double()
        _check(lib().gevo_pop_last_time(self._h, ctypes.byref(s)), "gevo_pop_last_time")
        return s.value

    # ------------------------------------------------------------ state access
    def export(self, v: int):
        params = np.zeros(param_count(self.dims), np.float32)
        nw = sum(self.dims[l - 1] * self.dims[l] for l in range(1, len(self.dims)))
        mask = np.zeros(nw, np.uint8)
        lr, dens = ctypes.c_float(), ctypes.c_float()
        _check(lib().gevo_pop_export(self._h, v, _fp(params), mask.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)),
                                     ctypes.byref(lr), ctypes.byref(dens)), "gevo_pop_export")
        return dict(params=params, mask=mask, lr=np.float32(lr.value), density=np.float32(dens.value))

    def import_params(self, v: int, params):
        p = np.ascontiguousarray(np.asarray(params, np.float32))
        assert p.size == param_count(self.dims)
        _check(lib().gevo_pop_import(self._h, v, _fp(p)), "gevo_pop_import")

    def epoch_labels(self) -> np.ndarray:
        out = np.zeros(self.n_train, np.int32)
        _check(lib().gevo_pop_epoch_labels(self._h, out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                           self.n_train), "gevo_pop_epoch_labels")
        return out

    def set_profiling(self, on: bool = True):
        _check(lib().gevo_pop_set_profiling(self._h, 1 if on else 0), "gevo_pop_set_profiling")

    def kernel_stats(self) -> dict:
        """{kind: (total_ms, launches)} of kernels enqueued while profiling was on."""
        out = {}
        for i, name in enumerate(KERNEL_KINDS):
            ms, n = ctypes.c_double(), ctypes.c_uint64()
            _check(lib().gevo_pop_kernel_stats(self._h, i, ctypes.byref(ms), ctypes.byref(n)), "gevo_pop_kernel_stats")
            out[name] = (ms.value, n.value)
        return out

    def set_genomes(self, genomes, lr_base):
        """Rebuild every variant from its edit list; returns (learning rates,
        expected kept fractions).  Training restarts at epoch 0."""
        assert len(genomes) == self.P
        off, edits = _pack_genomes(genomes)
        lr = np.zeros(self.P, np.float32)
        dens = np.zeros(self.P, np.float64)
        _check(lib().gevo_pop_set_genomes(self._h, lr_base, _u32p(off), edits, _fp(lr), _f64p(dens)),
               "gevo_pop_set_genomes")
        return lr, dens

    def set_grad_scale(self, scale):
        """Per-element output-gradient scale [P][batch][classes] (None: the scalar 1/b)."""
        if scale is None:
            _check(lib().gevo_pop_set_grad_scale(self._h, None), "gevo_pop_set_grad_scale")
            return
        s = np.ascontiguousarray(np.asarray(scale, np.float32))
        assert s.shape == (self.P, self.cfg["batch"], self.dims[-1]), s.shape
        _check(lib().gevo_pop_set_grad_scale(self._h, _fp(s)), "gevo_pop_set_grad_scale")

    def reinit(self):
        """Destroy the handle and create a fresh population on the same workspace
        and datasets (a new fitness evaluation from the seed)."""
        self.close()
        h = ctypes.c_void_p()
        ptr = lambda t: None if t is None else ctypes.c_void_p(t.data_ptr())
        _check(lib().gevo_pop_init(ctypes.byref(self._cfg), ctypes.c_void_p(self.workspace.data_ptr()),
                                   self.workspace.numel(), ptr(self.x_train), ptr(self.y_train), ptr(self.x_test),
                                   ptr(self.y_test), ctypes.c_void_p(self.stream.cuda_stream), ctypes.byref(h)),
               "gevo_pop_init")
        self._h = h

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            lib().gevo_pop_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def cnn_param_count(cfg: dict) -> int:
    n = ctypes.c_size_t()
    c = cnn_config_struct(cfg)
    _check(lib().gevo_cnn_param_count(ctypes.byref(c), ctypes.byref(n)), "gevo_cnn_param_count")
    return n.value


class CnnPopulation:
    """P variants of the convolutional prediction workload on one GPU; all
    device memory comes from torch."""

    def __init__(self, cfg: dict, base_params, x_test, y_test, device="cuda", stream=None):
        import torch
        self.torch = torch
        self.cfg = dict(cfg)
        self.P = cfg["P"]
        dev = torch.device(device)
        self.x_test = torch.as_tensor(x_test).to(device=dev, dtype=torch.float32).contiguous()
        self.y_test = torch.as_tensor(y_test).to(device=dev, dtype=torch.int32).contiguous()
        n = self.x_test.shape[0]
        assert self.x_test.shape == (n, cfg["H"], cfg["W"], cfg["C"]) and self.y_test.shape == (n,)
        self.n_test = n
        self._cfg = cnn_config_struct(cfg)
        base = np.ascontiguousarray(np.asarray(base_params, dtype=np.float32))
        assert base.size == cnn_param_count(cfg)
        nbytes = ctypes.c_size_t()
        _check(lib().gevo_cnn_workspace_bytes(ctypes.byref(self._cfg), n, ctypes.byref(nbytes)),
               "gevo_cnn_workspace_bytes")
        self.workspace = torch.empty(max(nbytes.value, 256), dtype=torch.uint8, device=dev)
        self.stream = stream if stream is not None else torch.cuda.current_stream(dev)
        h = ctypes.c_void_p()
        _check(lib().gevo_cnn_init(ctypes.byref(self._cfg), ctypes.c_void_p(self.workspace.data_ptr()), nbytes.value,
                                   _fp(base), ctypes.c_void_p(self.x_test.data_ptr()),
                                   ctypes.c_void_p(self.y_test.data_ptr()), n,
                                   ctypes.c_void_p(self.stream.cuda_stream), ctypes.byref(h)), "gevo_cnn_init")
        self._h = h

    def predict(self):
        _check(lib().gevo_cnn_predict(self._h), "gevo_cnn_predict")

    def scores(self) -> dict:
        loss = np.zeros(self.P, np.float32)
        acc = np.zeros(self.P, np.float32)
        t = np.zeros(self.P, np.float32)
        _check(lib().gevo_cnn_scores(self._h, _fp(loss), _fp(acc), _fp(t)), "gevo_cnn_scores")
        return {"test_loss": loss, "test_acc": acc, "time_s": t}

    def set_profiling(self, on: bool):
        _check(lib().gevo_cnn_set_profiling(self._h, 1 if on else 0), "gevo_cnn_set_profiling")

    def kernel_stats(self) -> dict:
        """{kind: (total ms, launches)} of the kernels timed so far."""
        out = {}
        for i, k in enumerate(CNN_KERNEL_KINDS):
            ms, n = ctypes.c_double(), ctypes.c_uint64()
            _check(lib().gevo_cnn_kernel_stats(self._h, i, ctypes.byref(ms), ctypes.byref(n)), "gevo_cnn_kernel_stats")
            out[k] = (ms.value, n.value)
        return out

    def remove_layer(self, v: int, layer):
        """Variant v loses a block layer: its canonical tensor index, or its
        name "dw<i>" / "pw<i>" (the depthwise or pointwise layer of block i)."""
        if isinstance(layer, str):
            i = int(layer[2:])
            layer = 2 * i + (1 if layer.startswith("dw") else 2)
        _check(lib().gevo_cnn_remove_layer(self._h, v, layer), "gevo_cnn_remove_layer")

    def export(self, v: int) -> dict:
        n = cnn_param_count(self.cfg)
        params = np.zeros(n, np.float32)
        nw = n - _cnn_bias_count(self.cfg)
        mask = np.zeros(nw, np.uint8)
        dens = np.zeros(1, np.float32)
        _check(lib().gevo_cnn_export(self._h, v, _fp(params), mask.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)),
                                     _fp(dens)), "gevo_cnn_export")
        return {"params": params, "mask": mask, "density": float(dens[0])}

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            lib().gevo_cnn_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _cnn_bias_count(cfg: dict) -> int:
    n = cfg["stem"]
    c = cfg["stem"]
    for _, co in cfg["blocks"]:
        n += c + co
        c = co
    return n + cfg["classes"]
