"""Compile the HIP sources in ``csrc/`` into ``libkvx.so`` for gfx950.

Usage: ``python -m paper_2608_30963_amd.build`` (or ``build()`` from Python).
The library is built in-tree so it travels with the source tree.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libkvx.so")
ARCH = "gfx950"


def hipcc() -> str:
    for c in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


NOISE = "is not a recognized feature for this target"


def _flags():
    return [
        f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
        # keep the compiler from forming packed fp32 instructions
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-I", os.path.join(ROOT, "include"), "-I", CSRC,
    ]


def _check(r, what):
    err = "\n".join(x for x in r.stderr.splitlines() if NOISE not in x)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {what} ({r.returncode}):\n{err}")
    return err


def build(out: str = LIB, verbose: bool = False) -> str:
    """Compile the host library, the translator fit, the translator-variant
    composition, the staged (unfused) translation and the fused kernel's
    three precision variants as separate objects (in parallel), then link
    libkvx.so."""
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    units = [("kvx", os.path.join(CSRC, "kvx.hip"), []),
             ("fit", os.path.join(CSRC, "fit.hip"), []),
             ("compose", os.path.join(CSRC, "compose.hip"), []),
             ("staged", os.path.join(CSRC, "staged.hip"), [])]
    for i, name in enumerate(("bf16x2", "bf16", "f16")):
        units.append((f"fused_{name}", os.path.join(CSRC, "fused_launch.hip"),
                      [f"-DKVX_LAUNCH_PREC={i}"]))
    procs = []
    for name, src, extra in units:
        obj = os.path.join(objdir, name + ".o")
        cmd = [hipcc()] + _flags() + extra + ["-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((name, obj, subprocess.Popen(cmd, stdout=subprocess.PIPE,
                                                  stderr=subprocess.PIPE, text=True)))
    objs = []
    for name, obj, p in procs:
        stdout, stderr = p.communicate()
        err = _check(subprocess.CompletedProcess(p.args, p.returncode, stdout, stderr), name)
        if err.strip() and verbose:
            print(err, file=sys.stderr)
        objs.append(obj)
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC"] + objs + ["-o", out + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    _check(subprocess.run(cmd, capture_output=True, text=True), "link")
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
