"""Build libpvconv.so (HIP, gfx950) in-tree with hipcc, and libpvpeak.so (the
measured-peak probes the benchmark uses, csrc/peak/).

Usage: python -m paper_1907_03739_amd.build [--verbose]
"""
from __future__ import annotations

import concurrent.futures
import glob
import os
import re
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libpvconv.so")
PEAK_LIB = os.path.join(PKG, "libpvpeak.so")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# Packed fp32 ops are disabled for all device code; the host pass warns that
# it does not know the feature, which is harmless.
FLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wno-unused-command-line-argument", f"-I{INCLUDE}", f"-I{CSRC}"]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def peak_sources():
    return sorted(glob.glob(os.path.join(CSRC, "peak", "*.hip")))


# Every kernel's resource usage is reported by the compiler; a kernel with
# scratch (private memory, i.e. register spills or stack arrays) fails the
# build, since scratch traffic goes to HBM and no kernel here is designed to
# use it.
RESOURCE_REMARKS = "-Rpass-analysis=kernel-resource-usage"
_FN = re.compile(r"remark: Function Name: (\S+)")
_SCRATCH = re.compile(r"remark:\s+ScratchSize \[bytes/lane\]: (\d+)")


def scratch_kernels(remarks: str):
    """(kernel, bytes per lane) for every function the remarks give scratch."""
    bad, fn = [], None
    for line in remarks.splitlines():
        m = _FN.search(line)
        if m:
            fn = m.group(1)
            continue
        m = _SCRATCH.search(line)
        if m and int(m.group(1)) > 0:
            bad.append((fn, int(m.group(1))))
    return bad


def _compile(src, verbose):
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC, *FLAGS, RESOURCE_REMARKS, "-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    lines = (r.stdout + r.stderr).splitlines()
    out = "\n".join(l for l in lines
                    if "packed-fp32-ops" not in l and "is not a recognized feature" not in l
                    and "kernel-resource-usage" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{out}")
    bad = scratch_kernels("\n".join(lines))
    if bad:
        listing = "\n".join(f"  {fn}: {n} bytes/lane" for fn, n in bad)
        raise RuntimeError(f"kernels in {src} use scratch memory:\n{listing}")
    if verbose and out.strip():
        print(out)
    return obj


def _link(objs, lib, verbose):
    tmp = lib + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    """Compile every csrc/*.hip for gfx950 and link libpvconv.so, and the probes
    of csrc/peak/ into libpvpeak.so (always rebuilds)."""
    os.makedirs(BUILD, exist_ok=True)
    srcs, peak = sources(), peak_sources()
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs) + len(peak))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), srcs + peak))
    _link(objs[:len(srcs)], LIB, verbose)
    if peak:
        _link(objs[len(srcs):], PEAK_LIB, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose="--verbose" in sys.argv))
