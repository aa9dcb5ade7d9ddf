"""Build libprr.so for gfx950 with hipcc, in the package directory.

Each source is compiled to an object of its own in parallel (the device code of the
fused step and of the separate kernels dominates the build time), then the objects are
linked into the shared library."""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCES = ["csrc/prr_kernels.hip", "csrc/prr_fused_bf16.hip", "csrc/prr_fused_f16.hip", "csrc/prr_fused_p64.hip",
           "csrc/prr_api.cpp", "csrc/prr_calibrate.cpp", "csrc/prr_budget.cpp",
           "csrc/prr_noalloc.hip"]
OUT = os.path.join(HERE, "libprr.so")
OBJ_DIR = os.path.join(ROOT, "_build", "obj")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # no packed fp32 instructions (v_pk_*_f32) anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in res.stderr.splitlines() if "packed-fp32-ops" not in l)
    return res.returncode, err


def build(verbose: bool = True) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    os.makedirs(OBJ_DIR, exist_ok=True)
    inc = ["-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(HERE, "csrc")]
    sources = [s for s in SOURCES if os.path.exists(os.path.join(HERE, s))]
    jobs = []
    for s in sources:
        obj = os.path.join(OBJ_DIR, os.path.basename(s) + ".o")
        jobs.append((obj, [hipcc, *HIPCC_FLAGS, *inc, "-c", os.path.join(HERE, s), "-o", obj]))
    if verbose:
        for _, cmd in jobs:
            print("[build]", " ".join(cmd), flush=True)
    with cf.ThreadPoolExecutor(max_workers=min(len(jobs), os.cpu_count() or 1)) as ex:
        results = list(ex.map(lambda j: _run(j[1]), jobs))
    for (obj, _), (rc, err) in zip(jobs, results):
        if rc != 0:
            raise RuntimeError(f"hipcc failed ({rc}) for {obj}:\n{err}")
        if err.strip() and verbose:
            print(err, file=sys.stderr)
    tmp = OUT + ".tmp"
    link = [hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", *[o for o, _ in jobs], "-o", tmp]
    if verbose:
        print("[build]", " ".join(link), flush=True)
    rc, err = _run(link)
    if rc != 0:
        raise RuntimeError(f"link failed ({rc}):\n{err}")
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    build()
