#!/usr/bin/env python3
"""Benchmark of population-batched fitness evaluation on one MI355X.

One step = one full fitness evaluation of the population (GEVO-ML, arXiv
2310.10211, section 4.3): create the population from the seed (masks, initial
weights), retrain every variant for the workload's epochs of mini-batch SGD
over the training split (section 6.2), predict the test split, read the
scores.  The default workload is P=256 variants of a 784-256-10 classifier in
bf16 with fp32 master weights, 60,000 MNIST-shaped synthetic rows, batch 128,
2 epochs.

Prints one JSON line.  `value` = variant-samples/s of training over the whole
step (P * n_train * epochs / step time); inputs are resident in HBM before the
timed region.  `roofline` is for the kernel with the largest share of the
timed kernel time, from HIP events recorded by each launch's own dispatch.
`cpu_baseline` times the CPU oracle on a bounded sample of the same workload.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK = {"bf16": 2500.0, "f32": 157.3}        # dense MFMA TFLOP/s, MI355X
PREDICT_CHUNK = 2048                          # test rows per prediction launch (the library's chunk)
HBM_PEAK_GBS = 8000.0
CSRC = os.path.join(ROOT, "paper_2310_10211_amd", "csrc")
KERNEL_SOURCES = ["gevo_device.h", "gevo_internal.h", "gevo_kernels.hip", "gevo_fused.hip", "gevo_stream.hip",
                  "gevo_bwd.hip", "gevo_gemm.hip", "gevo_predict.hip"]
# rocprofv3 kernel-name stem -> kernel kind of gevo_pop_kernel_stats (training kind, predict kind)
KERNEL_KIND_OF = {"k_fused2": ("fused_train", None), "k_stream_layer": ("layer_train", "layer_fwd"),
                  "k_layer": ("layer_train", "layer_fwd"), "k_out_fwd": ("out_train", None),
                  "k_out_upd": ("out_train", None), "k_out": (None, "out_predict"),
                  "k_bwd_gemm": ("bwd", None), "k_bwd": ("bwd", None), "k_pred_gemm<true>": (None, "fwd_out"),
                  "k_pred_gemm<false>": (None, "layer_fwd"), "k_wt_bf16": (None, "weight_copy"),
                  "k_fwd_gemm": (None, "layer_fwd")}


def fused_workload(cfg):
    """Two-layer bf16 nets train in the fused per-variant kernel; the layer and
    output kernels then only run for prediction."""
    return len(cfg["dims"]) == 3 and cfg["dtype"] == "bf16"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_counters.json")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", type=int, default=3, help="workload 1..5 (default 3)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the CPU-oracle sample")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="time without per-kernel events")
    ap.add_argument("--cnn", action="store_true",
                    help="time the convolutional prediction workload (P=64 depthwise-separable nets on "
                         "32x32x3 images) instead")
    ap.add_argument("--search", type=int, default=0, metavar="G",
                    help="time G generations of the search loop on this workload instead")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device copy 3 times (reference for HBM counters) and exit")
    ap.add_argument("--mfma-from", metavar="DIR",
                    help="only summarise a rocprofv3 --pmc run of the MFMA counters (SQ_VALU_MFMA_BUSY_CYCLES, "
                         "SQ_INSTS_VALU_MFMA_MOPS_BF16/_F32, GRBM_GUI_ACTIVE, ...) as a markdown table and exit")
    ap.add_argument("--traffic-from", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR", "COPY_WRITE_DIR"),
                    help="only fold rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE runs of this workload and of "
                         "--calibrate-copy into profiles/traffic_counters.json and exit")
    return ap.parse_args()


def calibrate_copy():
    """A plain copy kernel of known size: 1 GiB read + 1 GiB written per launch."""
    import torch
    n = 1 << 28                                    # 2^28 float32 = 1 GiB
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read_per_launch": 4 * n, "copy_bytes_written_per_launch": 4 * n, "launches": 3}))


# ------------------------------------------------------------ algorithmic cost
def layer_costs(cfg):
    """Per-launch algorithmic bytes and flops of each kernel kind (real, unpadded
    dims; e = operand bytes).  Returns {kind: (bytes, flops)} per launch, averaged
    over the launches of one SGD step, plus per-step launch counts."""
    d, P, B = cfg["dims"], cfg["P"], cfg["batch"]
    e = 2 if cfg["dtype"] == "bf16" else 4
    L = len(d) - 1
    out = {}
    # hidden layers l = 1..L-1: weight gradient + masked update (+ next forward)
    lb, lf = [], []
    for l in range(1, L):
        K, N = d[l - 1], d[l]
        shared_in = l == 1
        per_v = N * K * 8 + N * K / 8 + N * B * e + 2 * B * N * e + N * 8   # W rd+wr, mask, G in, A out, bias
        in_b = (K * B * e) * 2                                             # A cols (dW) + A rows (next forward)
        byts = P * per_v + (in_b if shared_in else P * in_b)
        lb.append(byts)
        lf.append(P * 4.0 * B * K * N)                                      # dW + forward
    if lb:
        out["layer_train"] = (sum(lb) / len(lb), sum(lf) / len(lf), len(lb))
    # output layer
    K, C = d[L - 1], d[L]
    byts = P * (C * K * 8 + C * K / 8 + 2 * B * K * e + (K * B * e if L > 1 else 0))
    fl = P * 2.0 * B * K * C * (3 if L > 1 else 2)
    out["out_train"] = (byts, fl, 1)
    # hidden backward GEMMs
    bb, bf = [], []
    for l in range(2, L):
        K, N = d[l - 1], d[l]
        bb.append(P * (K * N * e + B * N * e + 2 * K * B * e))
        bf.append(P * 2.0 * B * K * N)
    if bb:
        out["bwd"] = (sum(bb) / len(bb), sum(bf) / len(bf), len(bb))
    if cfg["epochs"] == 0:
        out.update(predict_costs(cfg))
    if L == 2:
        # fused per-variant kernel: one launch = every SGD step of an epoch
        K, N = d[0], d[1]
        T = (cfg["n_train"] + B - 1) // B
        per_step = P * (N * K * 8 + N * K / 8 + C * N * 8 + C * N / 8 + (N + C) * 8) + 2 * B * K * e + B * 4
        fl_step = P * B * (4.0 * K * N + 6.0 * N * C)
        out["fused_train"] = (T * per_step, T * fl_step, 1)
    return out


def _pad(x, m=32):
    return (x + m - 1) // m * m


def predict_plan(cfg):
    """The library's prediction plan for bf16 nets: hidden layer l runs on the
    prediction GEMM when its padded width is a multiple of 256 (reading a bf16
    weight copy), and a last hidden layer exactly 256 wide also runs the output
    layer ('fwd_out'); other hidden layers run the older forward kernels
    ('layer_fwd' with fp32 weights) and the output layer on its own
    ('out_predict').  Returns [(kind, weight bytes per weight)] per hidden layer
    and whether the output layer is fused."""
    d = cfg["dims"]
    L = len(d) - 1
    plan, fused = [], False
    for l in range(1, L):
        pred = cfg["dtype"] == "bf16" and _pad(d[l]) % 256 == 0
        if pred and l == L - 1 and _pad(d[l]) == 256:
            plan.append(("fwd_out", 2))
            fused = True
        else:
            plan.append(("layer_fwd", 2 if pred else 4))
    return plan, fused


def predict_costs(cfg):
    """{kind: (bytes, flops, launches)} per launch of one pass over the test
    split, averaged over the kind's launches.  Per launch (one chunk of rows,
    all P variants): weights once (the bf16 copy or the fp32 master) plus
    biases; the layer's input rows (layer 1: shared by all variants); its
    output rows unless the output layer is fused; a fused launch adds the
    output layer's fp32 weights and the chunk's labels.  The weight copy
    reads the fp32 master and writes bf16."""
    d, P = cfg["dims"], cfg["P"]
    e = 2 if cfg["dtype"] == "bf16" else 4
    L = len(d) - 1
    C = d[L]
    n, R = cfg["n_test"], PREDICT_CHUNK
    chunks = [min(R, n - c) for c in range(0, n, R)]
    plan, fused = predict_plan(cfg)
    acc = {}

    def add(kind, b, f):
        a = acc.setdefault(kind, [0.0, 0.0, 0])
        a[0] += b
        a[1] += f
        a[2] += 1

    for l, (kind, wb) in enumerate(plan, start=1):
        K, N = d[l - 1], d[l]
        if wb == 2:
            add("weight_copy", P * K * N * (4 + 2), 0.0)
        for rows in chunks:
            a_in = rows * K * e if l == 1 else P * rows * K * e
            b = P * (K * N * wb + N * 4) + a_in
            f = P * 2.0 * rows * K * N
            if kind == "fwd_out":
                b += P * (C * N * 4 + C * 4) + rows * 4
                f += P * 2.0 * rows * N * C
            else:
                b += P * rows * N * e
            add(kind, b, f)
    if not fused:
        K = d[L - 1]
        for rows in chunks:
            add("out_predict", P * (C * K * 4 + C * 4) + (rows * K * e if L == 1 else P * rows * K * e) + rows * 4,
                P * 2.0 * rows * K * C)
    return {k: (v[0] / v[2], v[1] / v[2], v[2]) for k, v in acc.items()}


def train_flops_per_sample(dims):
    """fwd 2 + weight gradient 2 (+ input gradient 2 above the first layer) per weight."""
    f = 4 * dims[0] * dims[1]
    for l in range(2, len(dims)):
        f += 6 * dims[l - 1] * dims[l]
    return f


def predict_flops_per_sample(dims):
    return sum(2 * dims[l - 1] * dims[l] for l in range(1, len(dims)))


CNN_KERNEL_SOURCES = ["gevo_device.h", "gevo_internal.h", "gevo_kernels.hip", "gevo_gemm.hip", "gevo_cnn.hip"]
# rocprofv3 kernel-name stem -> kernel kind of the convolutional workload
CNN_KIND_OF = {"k_cnn_stem": "stem", "k_cnn_dw": "depthwise", "k_fwd_gemm": "pointwise", "k_cnn_pool": "pool",
               "k_out": "head", "k_cnn_pwdw": "pw_dw"}


def source_sha(sources=None):
    h = hashlib.sha256()
    for name in sources or KERNEL_SOURCES:
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _counter_rows(d, counter):
    """(kernel name, grid size, value KiB) of every dispatch in a rocprofv3 --pmc csv directory."""
    import csv
    import glob
    rows = []
    for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as f:
            for r in csv.DictReader(f):
                if r["Counter_Name"] == counter:
                    rows.append((r["Kernel_Name"], int(r["Grid_Size"]), float(r["Counter_Value"])))
    if not rows:
        raise SystemExit(f"bench.py: no {counter} rows under {d}")
    return rows


def fold_traffic(cfg, fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, command):
    """HBM bytes per launch of each kernel kind: FETCH_SIZE and WRITE_SIZE (KiB per
    dispatch) scaled by what the same counters read for a plain 1 GiB copy."""
    scale = copy_scales(copy_fetch_dir, copy_write_dir)
    trains = cfg["epochs"] > 0 and not fused_workload(cfg)
    per = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        groups = {}
        for name, grid, v in _counter_rows(d, counter):
            stem = next((k for k in KERNEL_KIND_OF if k in name), None)
            if stem:
                groups.setdefault((stem, grid), []).append(v)
        # a training kernel runs every SGD step (once per hidden layer of its
        # kind, one launch shape per layer); its prediction launches are a few
        # per call: launch shapes with at least half the top count are training
        top = {}
        for (stem, grid), vals in groups.items():
            top[stem] = max(top.get(stem, 0), len(vals))
        for (stem, grid), vals in groups.items():
            tr_kind, pr_kind = KERNEL_KIND_OF[stem]
            is_train = tr_kind and (stem == "k_fused2" or (trains and 2 * len(vals) >= top[stem]))
            kind = tr_kind if is_train else pr_kind
            if kind is None:
                continue
            # every launch of the kind: the average per launch, as the algorithmic bytes are
            cur = per.setdefault(kind, dict(grids=set(), n={}, kib={}))
            cur["grids"].add(grid)
            cur["n"][counter] = cur["n"].get(counter, 0) + len(vals)
            cur["kib"][counter] = cur["kib"].get(counter, 0.0) + sum(vals)
    for r in per.values():
        for c in r["kib"]:
            r["kib"][c] /= r["n"][c]
    try:
        with open(TRAFFIC_FILE) as f:
            table = json.load(f)
    except (OSError, ValueError):
        table = {}
    rec = table.setdefault(cfg["name"], {})
    sha = source_sha()
    for kind, r in per.items():
        if len(r["kib"]) != 2:
            continue
        rec[kind] = dict(kernel_source_sha=sha, grids=sorted(r["grids"]), dispatches=r["n"],
                         fetch_kib_per_dispatch=round(r["kib"]["FETCH_SIZE"], 3),
                         write_kib_per_dispatch=round(r["kib"]["WRITE_SIZE"], 3),
                         fetch_scale=round(scale["FETCH_SIZE"], 4), write_scale=round(scale["WRITE_SIZE"], 4),
                         hbm_bytes_per_launch=int(1024 * (r["kib"]["FETCH_SIZE"] * scale["FETCH_SIZE"]
                                                          + r["kib"]["WRITE_SIZE"] * scale["WRITE_SIZE"])),
                         command=command)
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(table, f, indent=1, sort_keys=True)
        f.write("\n")
    print(json.dumps(rec))


def copy_scales(copy_fetch_dir, copy_write_dir):
    """Bytes per counter unit: a plain 1 GiB copy's known bytes over its FETCH_SIZE
    and WRITE_SIZE readings."""
    n_copy = 4 << 28
    scale = {}
    for counter, d in (("FETCH_SIZE", copy_fetch_dir), ("WRITE_SIZE", copy_write_dir)):
        big = [v for name, _, v in _counter_rows(d, counter) if "copyBuffer" in name and v > 2 ** 19]
        if not big:
            raise SystemExit(f"bench.py: no 1 GiB copy dispatch in {d}")
        scale[counter] = n_copy / (1024.0 * sum(big) / len(big))
    return scale


def fold_traffic_cnn(cfg, fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, command):
    """Convolutional workload: mean HBM bytes per launch of each kernel kind over
    all its launches (the kinds launch with several shapes, one per layer)."""
    scale = copy_scales(copy_fetch_dir, copy_write_dir)
    per = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        for name, _, v in _counter_rows(d, counter):
            stem = next((k for k in CNN_KIND_OF if k in name), None)
            if stem:
                r = per.setdefault(CNN_KIND_OF[stem], {}).setdefault(counter, [0.0, 0])
                r[0] += v
                r[1] += 1
    try:
        with open(TRAFFIC_FILE) as f:
            table = json.load(f)
    except (OSError, ValueError):
        table = {}
    rec = table.setdefault(cfg["name"], {})
    sha = source_sha(CNN_KERNEL_SOURCES)
    for kind, r in per.items():
        if len(r) != 2:
            continue
        kib = {c: r[c][0] / r[c][1] for c in r}
        rec["cnn_" + kind] = dict(kernel_source_sha=sha, dispatches={c: r[c][1] for c in r},
                                  fetch_kib_per_dispatch=round(kib["FETCH_SIZE"], 3),
                                  write_kib_per_dispatch=round(kib["WRITE_SIZE"], 3),
                                  fetch_scale=round(scale["FETCH_SIZE"], 4), write_scale=round(scale["WRITE_SIZE"], 4),
                                  hbm_bytes_per_launch=int(1024 * (kib["FETCH_SIZE"] * scale["FETCH_SIZE"]
                                                                   + kib["WRITE_SIZE"] * scale["WRITE_SIZE"])),
                                  command=command)
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(table, f, indent=1, sort_keys=True)
        f.write("\n")
    print(json.dumps(rec))


def traffic_for(kernel, workload, sources=None):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or None
    if absent or taken on a different kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    rec = t.get(workload, {}).get(kernel)
    if not rec or rec.get("kernel_source_sha") != source_sha(sources):
        return None
    return rec.get("hbm_bytes_per_launch")


N_SIMD = 1024                                 # 256 CUs x 4 SIMDs
N_XCD = 8
MOP_FLOPS = 512                                # flops per MFMA "MOP" (SQ_INSTS_VALU_MFMA_MOPS_*)


def mfma_summary(d):
    """Per kernel of a rocprofv3 --pmc run: dispatches, cycles per dispatch
    (the dispatch timestamps), GPU clock (GRBM_GUI_ACTIVE, summed over the 8
    XCDs, over that time), MFMA busy fraction
    (SQ_VALU_MFMA_BUSY_CYCLES over all SIMD-cycles), MFMA flops per dispatch
    (MOPS x 512, padding included) and their rate at the measured cycles."""
    import collections
    import csv
    import glob
    acc = collections.defaultdict(lambda: collections.defaultdict(float))
    n = collections.Counter()
    dur = collections.defaultdict(float)
    for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as f:
            for r in csv.DictReader(f):
                k = r["Kernel_Name"].split("(")[0].replace("void ", "").replace("gevo::", "")
                acc[k][r["Counter_Name"]] += float(r["Counter_Value"])
                if r["Counter_Name"] == "GRBM_GUI_ACTIVE":
                    n[k] += 1
                    dur[k] += (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9
    lines = ["| Kernel | Dispatches | us per dispatch | GPU clock (GHz) | MFMA busy | MFMA TFLOP/s (bf16) | "
             "MFMA TFLOP/s (fp32) | LDS bank conflicts per LDS instruction |",
             "|---|---:|---:|---:|---:|---:|---:|---:|"]
    for k, v in sorted(acc.items(), key=lambda kv: -kv[1].get("GRBM_GUI_ACTIVE", 0.0)):
        if not n[k] or v.get("GRBM_GUI_ACTIVE", 0) <= 0 or dur[k] <= 0:
            continue
        cyc = v["GRBM_GUI_ACTIVE"] / N_XCD / n[k]
        t = dur[k] / n[k]
        busy = v.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / n[k] / (N_SIMD * cyc)
        bf = v.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) * MOP_FLOPS / n[k] / t / 1e12
        f32 = v.get("SQ_INSTS_VALU_MFMA_MOPS_F32", 0.0) * MOP_FLOPS / n[k] / t / 1e12
        lds = v.get("SQ_INSTS_LDS", 0.0)
        conf = v.get("SQ_LDS_BANK_CONFLICT", 0.0) / lds if lds else 0.0
        if busy < 1e-4 and cyc < 1e5:
            continue
        lines.append(f"| {k} | {n[k]} | {t * 1e6:,.1f} | {cyc / t / 1e9:.2f} | {100 * busy:.1f}% | {bf:,.1f} | "
                     f"{f32:,.1f} | {conf:.3f} |")
    return "\n".join(lines)


# ------------------------------------------------------------------ CPU oracle
def host_threads():
    """(threads to use, CPUs this process may run on): the machine's CPU share
    (OMP_NUM_THREADS where the environment sets it) within the affinity mask."""
    avail = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    try:
        share = int(os.environ.get("OMP_NUM_THREADS", "0"))
    except ValueError:
        share = 0
    return (min(share, avail) if share > 0 else avail), avail


def cpu_baseline(cfg, data, budget_s):
    import oracle
    threads, nproc = host_threads()
    V = threads
    variants = list(range(0, cfg["P"], max(1, cfg["P"] // V)))[:V]
    if cfg["epochs"] == 0:                   # prediction workload
        rows = 256
        sub = dict(data, y_test=data["y_test"][:rows], x_test=data["x_test"][:rows])
        t0 = time.perf_counter()
        oracle.evaluate(cfg, sub, variants=variants[:1], epochs=0, threads=1)
        one = time.perf_counter() - t0
        rows = int(max(256, min(len(data["y_test"]), rows * budget_s / max(one, 1e-3) * 0.8)))
        sub = dict(data, y_test=data["y_test"][:rows], x_test=data["x_test"][:rows])
        t0 = time.perf_counter()
        oracle.evaluate(cfg, sub, variants=variants, epochs=0, threads=threads)
        wall = time.perf_counter() - t0
        return dict(value=len(variants) * rows / wall, unit="variant-samples/s", cores=threads, nproc=nproc,
                    kind="oracle",
                    sample=f"{len(variants)} variants x {rows} test rows, prediction, {cfg['dtype']} oracle, "
                           f"one variant per thread, {threads} threads of {nproc} CPUs, {wall:.1f} s")
    B = cfg["batch"]
    t0 = time.perf_counter()
    oracle.evaluate(cfg, data, variants=variants[:1], epochs=1, steps=1, threads=1, do_predict=False)
    one = time.perf_counter() - t0
    steps = int(max(1, min((len(data["y_train"]) + B - 1) // B, budget_s / max(one, 1e-3) * 0.8)))
    t0 = time.perf_counter()
    oracle.evaluate(cfg, data, variants=variants, epochs=1, steps=steps, threads=threads, do_predict=False)
    wall = time.perf_counter() - t0
    return dict(value=len(variants) * steps * B / wall, unit="variant-samples/s", cores=threads, nproc=nproc,
                kind="oracle",
                sample=f"{len(variants)} variants x {steps} SGD steps of batch {B} (epoch 0), {cfg['dtype']} "
                       f"oracle, one variant per thread, {threads} threads of {nproc} CPUs, {wall:.1f} s")


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py: this build evaluates a population on exactly one GPU (asked for {max(args.gpus, world)}); "
              "variants would shard across GPUs with no exchange of weights.", file=sys.stderr)
        sys.exit(2)

    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.mfma_from:
        print(mfma_summary(args.mfma_from))
        return
    if args.traffic_from and args.cnn:
        import synthetic
        fold_traffic_cnn(synthetic.cnn_config("full"), *args.traffic_from,
                         command="rocprofv3 --pmc FETCH_SIZE|WRITE_SIZE --output-format csv -- python3 bench.py "
                                 "--cnn --steps 1 --warmup 0 --no-cpu --no-profile")
        return
    if args.traffic_from:
        import synthetic
        fold_traffic(synthetic.config(args.config), *args.traffic_from,
                     command=f"rocprofv3 --pmc FETCH_SIZE|WRITE_SIZE --output-format csv -- python3 bench.py "
                             f"--config {args.config} --steps 1 --warmup 0 --no-cpu --no-profile")
        return

    if args.cnn:
        cnn_bench(args)
        return

    import torch
    import paper_2310_10211_amd as g
    import synthetic

    cfg = synthetic.config(args.config)
    print(f"[bench] workload {cfg['name']}: generating synthetic data", file=sys.stderr, flush=True)
    data = synthetic.dataset(cfg)
    dev = torch.device("cuda:0")
    pop = g.Population(cfg, data["x_train"], data["y_train"], data["x_test"], data["y_test"], device=dev)
    torch.cuda.synchronize()

    if args.search:
        search_bench(pop, cfg, args.search)
        return

    def step(profile):
        pop.reinit()
        if profile:
            pop.set_profiling(True)
        for ep in range(cfg["epochs"]):
            pop.train_epoch(ep)
        pop.predict()
        s = pop.scores()
        stats = pop.kernel_stats() if profile else None
        return s, stats

    for i in range(args.warmup):
        step(False)
        print(f"[bench] warmup {i + 1}/{args.warmup} done", file=sys.stderr, flush=True)

    profile = not args.no_profile
    kstats = {}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        s, st = step(profile)
        if st:
            for k, (ms, n) in st.items():
                a = kstats.setdefault(k, [0.0, 0])
                a[0] += ms
                a[1] += n
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    print(f"[bench] timed {args.steps} steps", file=sys.stderr, flush=True)
    ms_step = (t1 - t0) * 1e3 / args.steps

    P, n_tr, n_te, E = cfg["P"], cfg["n_train"], cfg["n_test"], cfg["epochs"]
    if E > 0:
        value = P * n_tr * E / (ms_step / 1e3)
        work_flops = P * n_tr * E * train_flops_per_sample(cfg["dims"]) + P * n_te * predict_flops_per_sample(cfg["dims"])
    else:
        value = P * n_te / (ms_step / 1e3)
        work_flops = P * n_te * predict_flops_per_sample(cfg["dims"])
    peak = PEAK[cfg["dtype"]]

    roofline = None
    kernel_ms = {k: round(v[0] / args.steps, 3) for k, v in kstats.items() if v[1]}
    if kstats:
        dom = max((k for k in kstats if kstats[k][1] > 0), key=lambda k: kstats[k][0])
        avg_s = kstats[dom][0] / kstats[dom][1] / 1e3
        costs = layer_costs(cfg)
        if dom in costs:
            byts, fl, _ = costs[dom]
            ridge = peak * 1e12 / (HBM_PEAK_GBS * 1e9)
            if fl / byts < ridge:
                ach = byts / avg_s / 1e9
                roofline = dict(bound="hbm", achieved=round(ach, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                                frac=round(ach / HBM_PEAK_GBS, 4))
            else:
                ach = fl / avg_s / 1e12
                roofline = dict(bound="mfma", achieved=round(ach, 1), peak=peak, unit="TFLOP/s",
                                frac=round(ach / peak, 4))
            roofline.update(kernel=dom, avg_launch_us=round(avg_s * 1e6, 2), launches=kstats[dom][1],
                            algorithmic_bytes_per_launch=int(byts), algorithmic_flops_per_launch=int(fl),
                            traffic=traffic_for(dom, cfg["name"]))

    cpu = None
    if not args.no_cpu:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        cpu = cpu_baseline(cfg, data, args.cpu_seconds)

    out = {
        "metric": "variant-samples/sec (train fwd+bwd+SGD) at P variants; % bf16 MFMA peak",
        "value": round(value, 1),
        "unit": "variant-samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg["dtype"],
        "data": "synthetic",
        "config": {"workload": cfg["name"], "P": P, "dims": cfg["dims"], "batch": cfg["batch"], "epochs": E,
                   "n_train": n_tr, "n_test": n_te, "step": "init + all epochs + test prediction + scores",
                   "parallelism": "population (one GPU)"},
        "mfma_frac_of_step": round(work_flops / (ms_step / 1e3) / (peak * 1e12), 4),
        "kernel_ms_per_step": kernel_ms,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))


# ------------------------------------------------------- convolutional workload
def cnn_fuse_rows(cin, cout, w, s, ho):
    """Strip rows of the fused pointwise + depthwise kernel for one block pair,
    or 0 when the library runs the pair unfused (the library's rule: Cin <= 128
    and Cout 128 or 256; a strip's S (R - 1) + 3 rows of inputs and outputs
    and the tap pairs within 64 KiB of LDS, its inputs within 2,048 pieces of
    16 bytes)."""
    if cin % 32 or cin > 128 or cout not in (128, 256):
        return 0
    best = 0
    for r in range(1, ho + 1):
        px = (s * (r - 1) + 3) * w
        lds = (px * (cin + 8) + 7) // 8 * 8 * 2 + (px * (cout + 8) + 7) // 8 * 8 * 2 + 24 * cout
        if lds <= 64 * 1024 and px * cin // 8 <= 2048:
            best = r
    return best


def cnn_costs(cfg, n):
    """{kernel kind: (algorithmic HBM bytes, flops)} of one prediction pass over
    n test images for all P variants.  Per image and variant every activation
    map that goes through memory is written once by its producer and read once
    by its consumer (bf16); a fused pointwise + depthwise pair keeps the
    pointwise map on chip.  The input image is read once for all variants
    (fp32); every launch reads its variants' fp32 weights and biases once per
    64-image chunk."""
    P, H, W, C, cls = cfg["P"], cfg["H"], cfg["W"], cfg["C"], cfg["classes"]
    chunks = (n + 63) // 64
    stem = cfg["stem"]
    out = {"stem": [n * H * W * C * 4 + P * n * H * W * stem * 2 + P * chunks * (9 * C * stem + stem) * 4,
                    2.0 * P * n * H * W * 9 * C * stem]}
    blocks = cfg["blocks"]
    sizes = [(H, W)]
    for s_, _ in blocks:
        h, w = sizes[-1]
        sizes.append(((h - 1) // s_ + 1, (w - 1) // s_ + 1))
    chans = [stem] + [co for _, co in blocks]          # input channels of block i = chans[i]
    dw, pw, fu = [0.0, 0.0], [0.0, 0.0], [0.0, 0.0]

    def dw_cost(i):
        (h, w), (ho, wo), c = sizes[i], sizes[i + 1], chans[i]
        return P * n * (h * w + ho * wo) * c * 2 + P * chunks * 10 * c * 4, 2.0 * P * n * ho * wo * c * 9

    b0, f0 = dw_cost(0)
    dw[0] += b0
    dw[1] += f0
    i = 0
    while i < len(blocks):
        (h, w), ci, co = sizes[i + 1], chans[i], chans[i + 1]
        pw_fl = 2.0 * P * n * h * w * ci * co
        if i + 1 < len(blocks) and cnn_fuse_rows(ci, co, w, blocks[i + 1][0], sizes[i + 2][0]):
            (ho, wo) = sizes[i + 2]
            fu[0] += P * n * (h * w * ci + ho * wo * co) * 2 + P * chunks * (ci * co + co + 10 * co) * 4
            fu[1] += pw_fl + 2.0 * P * n * ho * wo * co * 9
        else:
            pw[0] += P * n * h * w * (ci + co) * 2 + P * chunks * (ci * co + co) * 4
            pw[1] += pw_fl
            if i + 1 < len(blocks):
                b, f = dw_cost(i + 1)
                dw[0] += b
                dw[1] += f
        i += 1
    out["depthwise"] = dw
    if pw[0]:
        out["pointwise"] = pw
    if fu[0]:
        out["pw_dw"] = fu
    h, w = sizes[-1]
    ch = chans[-1]
    out["pool"] = [P * n * (h * w * ch + ch) * 2, float(P * n * h * w * ch)]
    out["head"] = [P * n * ch * 2 + P * chunks * (ch * cls + cls) * 4, 2.0 * P * n * ch * cls]
    return {k: tuple(v) for k, v in out.items()}


def cnn_cpu_baseline(cfg, base, x, y, budget_s):
    from oracle import cnn
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = 1
    n0 = 64
    t0 = time.perf_counter()
    cnn.evaluate(cfg, base, x[:n0], y[:n0], [0], mode="bf16")
    one = time.perf_counter() - t0
    n = int(max(n0, min(len(y), n0 * budget_s / max(one, 1e-3) * 0.8)))
    t0 = time.perf_counter()
    cnn.evaluate(cfg, base, x[:n], y[:n], [0], mode="bf16")
    wall = time.perf_counter() - t0
    return dict(value=n / wall, unit="variant-images/s", cores=cores, kind="oracle",
                sample=f"variant 0 x {n} test images, prediction, bf16-rounding fp64 oracle (numpy, {cores} BLAS "
                       f"threads), {wall:.1f} s")


def cnn_bench(args):
    import numpy as np
    import torch
    import paper_2310_10211_amd as g
    import synthetic

    cfg = synthetic.cnn_config("full")
    print(f"[bench] workload {cfg['name']}: generating synthetic inputs", file=sys.stderr, flush=True)
    base, x, y = synthetic.cnn_inputs(cfg)
    dev = torch.device("cuda:0")
    t0 = time.perf_counter()
    pop = g.CnnPopulation(cfg, base, x, y, device=dev)
    torch.cuda.synchronize()
    init_ms = (time.perf_counter() - t0) * 1e3

    def step():
        pop.predict()
        return pop.scores()

    for i in range(args.warmup):
        step()
        print(f"[bench] warmup {i + 1}/{args.warmup} done", file=sys.stderr, flush=True)
    profile = not args.no_profile
    if profile:
        before = pop.kernel_stats()
        pop.set_profiling(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        s = step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    print(f"[bench] timed {args.steps} steps", file=sys.stderr, flush=True)
    ms_step = (t1 - t0) * 1e3 / args.steps
    P, n = cfg["P"], len(y)
    value = P * n / (ms_step / 1e3)
    costs = cnn_costs(cfg, n)
    roofline, kernel_ms = None, {}
    if profile:
        after = pop.kernel_stats()
        pop.set_profiling(False)
        kst = {k: (after[k][0] - before[k][0], after[k][1] - before[k][1]) for k in after}
        kernel_ms = {k: round(v[0] / args.steps, 3) for k, v in kst.items() if v[1]}
        dom = max((k for k in kst if kst[k][1] and k in costs), key=lambda k: kst[k][0])
        byts, fl = costs[dom]
        tot_s = kst[dom][0] / 1e3 / args.steps
        launches = kst[dom][1] // args.steps
        ach = byts / tot_s / 1e9
        roofline = dict(bound="hbm", achieved=round(ach, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                        frac=round(ach / HBM_PEAK_GBS, 4), kernel=dom,
                        avg_launch_us=round(tot_s / launches * 1e6, 2), launches=launches,
                        algorithmic_bytes_per_launch=int(byts / launches),
                        algorithmic_flops_per_launch=int(fl / launches),
                        traffic=traffic_for("cnn_" + dom, cfg["name"], CNN_KERNEL_SOURCES))
    cpu = None
    if not args.no_cpu:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        cpu = cnn_cpu_baseline(cfg, base.astype(np.float64), x, y, args.cpu_seconds)
    total_flops = sum(v[1] for v in costs.values())
    out = {
        "metric": "variant-images/sec (prediction fitness) at P variants",
        "value": round(value, 1),
        "unit": "variant-images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": cfg["name"], "P": P, "image": [cfg["H"], cfg["W"], cfg["C"]], "stem": cfg["stem"],
                   "blocks": cfg["blocks"], "classes": cfg["classes"], "n_test": n,
                   "step": "test prediction of every variant + scores (variants built once, outside)",
                   "init_ms": round(init_ms, 1), "parallelism": "population (one GPU)"},
        "mfma_frac_of_step": round(total_flops / (ms_step / 1e3) / (PEAK["bf16"] * 1e12), 4),
        "kernel_ms_per_step": kernel_ms,
        "mean_test_loss": round(float(np.mean(s["test_loss"])), 4),
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))


def search_bench(pop, cfg, generations):
    """Generations of the GEVO-ML search on one population: each generation is
    a genome rebuild, a full fitness evaluation (all epochs, prediction,
    scores) and the host's ranking, selection and breeding."""
    import torch
    import paper_2310_10211_amd as g
    from paper_2310_10211_amd.search import Search
    lr_base = 0.05
    s = Search(pop, lr_base=lr_base, seed=cfg["seed"], epochs=cfg["epochs"], n_elite=min(16, pop.P))
    s.start()                                                  # generation 0 (untimed)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(generations):
        s.step()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    cur = s.history[-1]
    h0 = time.perf_counter()
    reps = 10
    for r in range(reps):                                      # the host part of one step, alone
        rank, crowd = g.nsga2_rank(cur.objectives)
        chosen = g.nsga2_select(rank, crowd, s.n_elite, pop.P, s.seed, 1 + r)
        g.genomes_breed([cur.genomes[i] for i in chosen[s.n_elite:]], s.seed, 1 + r, s.cxpb, s.mutpb, s.rho_lo,
                        10**6, s.max_edits)
    host_ms = (time.perf_counter() - h0) / reps * 1e3
    front = Search.front(cur)
    out = {
        "metric": "search generations/s (genome rebuild + fitness evaluation + NSGA-II step)",
        "value": round(generations / dt, 4),
        "unit": "generations/s",
        "n_gpus": 1,
        "generations": generations,
        "ms_per_generation": round(dt / generations * 1e3, 3),
        "host_select_breed_ms": round(host_ms, 3),
        "higher_is_better": True,
        "data": "synthetic",
        "config": {"workload": cfg["name"], "P": pop.P, "dims": cfg["dims"], "batch": cfg["batch"],
                   "epochs": cfg["epochs"], "lr_base": lr_base, "n_elite": s.n_elite, "cxpb": s.cxpb,
                   "mutpb": s.mutpb, "rho_lo": s.rho_lo},
        "front": [{"train_error": round(float(cur.objectives[i][0]), 5),
                   "kept_fraction": round(float(cur.objectives[i][1]), 5),
                   "test_error": round(float(cur.test_error[i]), 5), "lr": float(cur.lr[i])} for i in front[:8]],
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
