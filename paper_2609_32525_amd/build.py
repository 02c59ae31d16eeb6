"""Builds libflashslice.so (HIP kernels + C ABI) in-tree for gfx950 with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libflashslice.so")
OBJDIR = os.path.join(HERE, "_build")
SOURCES = [os.path.join(HERE, "csrc", f) for f in (
    "fs_pass_bwd_b.hip", "fs_pass_slice.hip", "fs_pass_deslice.hip", "fs_pass_bwd_a.hip",
    "fs_pass_point.hip", "fs_pass_linearno.hip", "fs_pass_bwd_b2.hip",
    "fs_kernels.hip", "fs_tokens.hip", "fs_tokmix.hip", "fs_noalloc.hip", "fs_api.cpp")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# Per-source flags: MFMA results in VGPRs rather than accumulation registers measured faster
# for the slice and deslice passes (less accumulator traffic around the softmax) and slower
# for backward pass B (higher register pressure), so it is applied per translation unit.
SOURCE_FLAGS = {
    "fs_pass_slice.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
    "fs_pass_deslice.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
}

# -packed-fp32-ops: no v_pk_{add,mul,fma}_f32 in the generated code.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-Wno-unused-result"]


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}): {' '.join(cmd)}\n{err}")
    return err


def build(verbose: bool = False, extra=None) -> str:
    """Compiles every source to an object (in parallel), then links the shared library."""
    os.makedirs(OBJDIR, exist_ok=True)
    cflags = [f for f in FLAGS if f != "-shared"] + (extra or [])
    objs, cmds = [], []
    for src in SOURCES:
        obj = os.path.join(OBJDIR, os.path.basename(src) + ".o")
        objs.append(obj)
        cmds.append([HIPCC] + cflags + SOURCE_FLAGS.get(os.path.basename(src), [])
                    + ["-c", src, "-o", obj])
    with ThreadPoolExecutor(max_workers=min(len(cmds), os.cpu_count() or 1)) as ex:
        errs = list(ex.map(_run, cmds))
    tmp = LIB + ".tmp"
    errs.append(_run([HIPCC] + FLAGS + (extra or []) + objs + ["-o", tmp]))
    if verbose:
        for c in cmds:
            print(" ".join(c), flush=True)
        for e in errs:
            if e.strip():
                print(e, file=sys.stderr)
    # the wide-store wait states the compiler leaves out after raw buffer stores
    if __package__:
        from .isa_check import WAIT_STATES, check_library
    else:  # run as a script from the package directory
        from isa_check import WAIT_STATES, check_library
    nstores, bad = check_library(tmp)
    if bad:
        lines = "\n".join("  " + " | ".join(b) for b in bad[:20])
        raise RuntimeError(f"{len(bad)} of {nstores} wide stores have their data registers "
                           f"overwritten within {WAIT_STATES} wait states:\n{lines}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
