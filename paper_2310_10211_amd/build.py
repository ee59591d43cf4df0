"""Build libgevo.so (HIP for gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libgevo.so")
SOURCES = [os.path.join(HERE, "csrc", n)
           for n in ("gevo_kernels.hip", "gevo_fused.hip", "gevo_resident.hip", "gevo_gemm.hip", "gevo_predict.hip", "gevo_stream.hip", "gevo_bwd.hip", "gevo_cnn.hip", "gevo_search.hip", "gevo_capi.hip")]
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off",                                   # elementwise fp32 ops round one at a time
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


# kernels whose master prefetches are explicit loads with explicit waits
PREFETCH_CHECKED = (("gevo_fused.hip", "_ZN4gevo8k_fused2"), ("gevo_stream.hip", "_ZN4gevo14k_stream_layer"))


# kernels whose direct-to-LDS loads read scalar registers from inline assembly
# (SGPR hazard check only; they stage no prefetch registers)
DMA_CHECKED = (("gevo_predict.hip", "_ZN4gevo11k_pred_gemm"), ("gevo_resident.hip", "_ZN4gevo6k_res2"),
               ("gevo_bwd.hip", "_ZN4gevo10k_bwd_gemm"))


def _device_asm(d: str, src: str) -> str:
    out = os.path.join(d, src[:-4] + ".s")
    cmd = [hipcc(), *[f for f in FLAGS if f not in ("-fPIC", "-shared")], "--cuda-device-only", "-S",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc"),
           "-o", out, os.path.join(HERE, "csrc", src)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc -S failed: " + res.stderr[-2000:])
    with open(out) as f:
        return f.read()


def check_fused_prefetch() -> dict:
    """Compile the kernels with explicit prefetches or direct-to-LDS loads to
    gfx950 assembly and verify their register discipline (check_prefetch.py)."""
    import tempfile

    from . import check_prefetch
    found = {}
    with tempfile.TemporaryDirectory() as d:
        for src, prefix in PREFETCH_CHECKED:
            found.update(check_prefetch.check_assembly(_device_asm(d, src), prefix))
        for src, prefix in DMA_CHECKED:
            found.update(check_prefetch.check_scalar_operands(_device_asm(d, src), prefix))
    return found


def build(verbose: bool = False) -> str:
    check_fused_prefetch()
    tmp = LIB + ".tmp"
    cmd = [hipcc(), *FLAGS, "-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc"),
           "-o", tmp, *SOURCES]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if verbose or res.returncode != 0:
        out = "\n".join(l for l in (res.stdout + res.stderr).splitlines()
                        if "packed-fp32-ops" not in l)            # the host pass does not know the feature
        if out.strip():
            print(out)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed: " + " ".join(cmd))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
