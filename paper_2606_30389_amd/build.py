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


# The fused kernel's roles hand results to each other, so it must keep its occupancy (two
# 512-thread workgroups per CU for 16-token pages; one for 64-token pages, whose grids hold
# at most ~170 workgroups) and no stack: a change that makes the compiler spill to scratch
# or cut occupancy slows every launch several-fold, so the build reports the kernel's
# resources and fails on either.
FUSED_MAX_SCRATCH = 64  # bytes per lane
FUSED_MIN_WAVES = {"ELi16E": 4, "ELi64E": 2}  # waves per SIMD by page size (mangled template argument)
RESOURCE_REMARKS = ["-Rpass-analysis=kernel-resource-usage"]


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in res.stderr.splitlines()
                    if "packed-fp32-ops" not in l and "kernel-resource-usage" not in l)
    return res.returncode, err, res.stderr


def fused_resources(stderr: str):
    """(kernel, scratch bytes per lane, waves per SIMD) of each fused_step_kernel instance
    in the compiler's resource remarks."""
    out, name = [], None
    scratch = occ = None
    for line in stderr.splitlines():
        if "Function Name:" in line:
            name = line.split("Function Name:")[1].split("[")[0].strip()
            scratch = occ = None
        elif name and "fused_step_kernel" in name and "ScratchSize [bytes/lane]:" in line:
            scratch = int(line.split(":")[-1].split("[")[0])
        elif name and "fused_step_kernel" in name and "Occupancy [waves/SIMD]:" in line:
            occ = int(line.split(":")[-1].split("[")[0])
            out.append((name, scratch, occ))
    return out


def build(verbose: bool = True) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    os.makedirs(OBJ_DIR, exist_ok=True)
    inc = ["-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(HERE, "csrc")]
    sources = [s for s in SOURCES if os.path.exists(os.path.join(HERE, s))]
    jobs = []
    for s in sources:
        obj = os.path.join(OBJ_DIR, os.path.basename(s) + ".o")
        extra = RESOURCE_REMARKS if "prr_fused_" in s else []
        jobs.append((obj, [hipcc, *HIPCC_FLAGS, *extra, *inc, "-c", os.path.join(HERE, s), "-o", obj]))
    if verbose:
        for _, cmd in jobs:
            print("[build]", " ".join(cmd), flush=True)
    with cf.ThreadPoolExecutor(max_workers=min(len(jobs), os.cpu_count() or 1)) as ex:
        results = list(ex.map(lambda j: _run(j[1]), jobs))
    for (obj, _), (rc, err, raw) in zip(jobs, results):
        if rc != 0:
            raise RuntimeError(f"hipcc failed ({rc}) for {obj}:\n{err}")
        if err.strip() and verbose:
            print(err, file=sys.stderr)
        for name, scratch, occ in fused_resources(raw):
            if verbose:
                print(f"[build] {name}: scratch {scratch} B/lane, {occ} waves/SIMD", flush=True)
            need = next((v for k, v in FUSED_MIN_WAVES.items() if k in name), 4)
            if scratch is None or scratch > FUSED_MAX_SCRATCH or occ < need:
                raise RuntimeError(f"{name}: scratch {scratch} B/lane, {occ} waves/SIMD (the fused kernel must not "
                                   f"spill beyond {FUSED_MAX_SCRATCH} B/lane and must keep {need} waves/SIMD)")
    tmp = OUT + ".tmp"
    link = [hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", *[o for o, _ in jobs], "-o", tmp]
    if verbose:
        print("[build]", " ".join(link), flush=True)
    rc, err, _ = _run(link)
    if rc != 0:
        raise RuntimeError(f"link failed ({rc}):\n{err}")
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    build()
