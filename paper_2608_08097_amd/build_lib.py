"""Build liboasis.so (all HIP kernels + the C ABI) for gfx950 with hipcc, in-tree."""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
LIB_PATH = os.path.join(PKG_DIR, "liboasis.so")


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build liboasis.so)")


def sources() -> list[str]:
    return sorted(glob.glob(os.path.join(PKG_DIR, "csrc", "*.hip")))


BUILD_DIR = os.path.join(ROOT, "_build")


def flags() -> list[str]:
    return [
        "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
        # packed-FP32 VALU ops stay disabled in every kernel
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-Wall", "-Wno-unused-function",
        "-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG_DIR, "csrc"),
    ]


# Extra compiler flags of single sources. attn.hip: keep MFMA accumulators and
# results in VGPRs; otherwise the compiler parks the attention's accumulators in
# AGPRs and copies all 64 of them to VGPRs on every unit for the rare rescale
# path.
FILE_FLAGS = {"attn.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def _run(cmd: list[str]) -> str:
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}): {' '.join(cmd)}\n{err}")
    return err


def build(verbose: bool = False) -> str:
    """Compile every HIP source (one hipcc process per file, in parallel) and link liboasis.so next
    to this file; returns its path."""
    from concurrent.futures import ThreadPoolExecutor
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = sources()
    objs = [os.path.join(BUILD_DIR, os.path.splitext(os.path.basename(f))[0] + ".o") for f in srcs]
    cmds = [[hipcc(), *flags(), *FILE_FLAGS.get(os.path.basename(f), []), "-c", f, "-o", o]
            for f, o in zip(srcs, objs)]
    try:
        jobs = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        jobs = os.cpu_count() or 1
    with ThreadPoolExecutor(max_workers=max(1, min(16, jobs))) as ex:
        errs = list(ex.map(_run, cmds))
    tmp = LIB_PATH + ".tmp"
    link = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    errs.append(_run(link))
    if verbose:
        for c in cmds + [link]:
            print(" ".join(c), flush=True)
        err = "\n".join(e for e in errs if e.strip())
        if err:
            print(err, file=sys.stderr)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
