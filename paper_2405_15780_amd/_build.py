"""Compile the HIP attention library for gfx950 into an in-tree shared object."""
from __future__ import annotations

import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB_PATH = os.path.join(HERE, "libvitattn.so")
SOURCES = ["vitattn_api.hip", "vitattn_fwd.hip", "vitattn_bwd.hip", "vitattn_merge.hip", "vitattn_ulysses.hip", "vitattn_agg.hip"]
ARCH = "gfx950"

HIP_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-Wall", "-Wextra",
    # packed fp32 VALU forms stay disabled on this target
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # keep matrix-core accumulators in VGPR form: otherwise the allocator
    # parks loop-carried accumulators in AGPRs and copies them every trip
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: cannot build the gfx950 attention library")


# Debug variant for the tests: every kernel first fills its LDS with NaN bytes,
# so a read of LDS that nothing wrote shows up as NaN (never used by the
# package itself; tests load it explicitly).
LDS_POISON_LIB_PATH = os.path.join(HERE, "libvitattn_ldspoison.so")


def _command(out: str, extra=()) -> list:
    return [hipcc(), *HIP_FLAGS, *extra, "-o", out, *[os.path.join(CSRC, s) for s in SOURCES]]


def build(verbose: bool = False, lds_poison: bool = True) -> str:
    """Always recompiles; writes LIB_PATH (and, with lds_poison, the LDS-poison
    debug variant, compiled alongside) atomically and returns LIB_PATH."""
    jobs = [(LIB_PATH, ())]
    if lds_poison:
        jobs.append((LDS_POISON_LIB_PATH, ("-DVITATTN_DEBUG_LDS_POISON",)))
    procs = []
    for path, extra in jobs:
        tmp = path + f".tmp{os.getpid()}"
        cmd = _command(tmp, extra)
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((path, tmp, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)))
    failed = []
    for path, tmp, p in procs:
        out, err = p.communicate()
        if p.returncode != 0:
            failed.append(f"{os.path.basename(path)}: hipcc failed ({p.returncode}):\n{out}\n{err}")
        else:
            os.replace(tmp, path)
    if failed:
        raise RuntimeError("\n".join(failed))
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
