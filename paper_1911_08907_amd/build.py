"""Build libaps.so (HIP kernels + C ABI) for gfx950 with hipcc, in-tree.

Each kernel file under csrc/ is compiled to an object in parallel; the
objects are then linked into one shared library.  The benchmark's
measurement probes (probe/*.hip, the path's access patterns without its
arithmetic) are linked into a library of their own, libaps_probe.so."""
from __future__ import annotations

import glob
import os
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libaps.so")
PROBE_DIR = os.path.join(PKG, "probe")
PROBE_LIB = os.path.join(PKG, "libaps_probe.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    # no hand-rolled or compiler-formed packed fp32 arithmetic
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # IEEE behaviour: keep fp32 denormals, no contraction into fma
    "-fno-fast-math",
    "-ffp-contract=off",
    "-Wall",
]


def sources() -> list:
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if cand and (os.path.sep not in cand or os.path.exists(cand)):
            return cand
    return "hipcc"


def _noise(stderr: str) -> list:
    # the host pass does not know the gpu-only target feature; that warning is expected
    return [ln for ln in stderr.splitlines()
            if ln.strip() and "packed-fp32-ops" not in ln and "warning generated" not in ln]


def build(verbose: bool = False, jobs: int | None = None) -> str:
    """Compile every csrc/*.hip file and link libaps.so next to this file,
    then the probes into libaps_probe.so."""
    _link(sources(), LIB, "libaps.so", verbose, jobs)
    _link(sorted(glob.glob(os.path.join(PROBE_DIR, "*.hip"))), PROBE_LIB, "libaps_probe.so", verbose, jobs)
    return LIB


def _link(srcs: list, lib: str, name: str, verbose: bool, jobs: int | None) -> None:
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    jobs = jobs or min(8, os.cpu_count() or 1)
    with tempfile.TemporaryDirectory(prefix="aps_build_") as tmp:
        objs, pending = [], []
        for src in srcs:
            obj = os.path.join(tmp, os.path.basename(src) + ".o")
            cmd = [hipcc(), *HIPCC_FLAGS, *inc, "-c", "-o", obj, src]
            if verbose:
                print(" ".join(cmd), flush=True)
            pending.append((src, cmd))
            objs.append(obj)
        running = []
        failed = []
        while pending or running:
            while pending and len(running) < jobs:
                src, cmd = pending.pop(0)
                running.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)))
            src, proc = running.pop(0)
            _, err = proc.communicate()
            if proc.returncode != 0:
                failed.append((src, err))
            elif verbose and _noise(err):
                sys.stderr.write("\n".join(_noise(err)) + "\n")
        if failed:
            for src, err in failed:
                sys.stderr.write(f"--- {src}\n{err}")
            raise RuntimeError(f"hipcc failed building {name}")
        tmp_lib = lib + ".tmp"
        cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp_lib, *objs]
        if verbose:
            print(" ".join(cmd), flush=True)
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            sys.stderr.write(res.stderr)
            raise RuntimeError(f"linking {name} failed")
        os.replace(tmp_lib, lib)


if __name__ == "__main__":
    print(build(verbose=True))
