"""Build the native libraries in-tree for gfx950.

libtaskpress.so   the eviction path (HIP kernels + C ABI), from csrc/
libtpsynth_*.so   the seeded input generator (host build with gcc, device build with hipcc)
libtprates.so     microbenchmarks of the machine's ceilings (bench.py --rates), not the path
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIBDIR = os.path.join(PKG, "lib")
BUILD = os.path.join(ROOT, "_build")
SYNTH = os.path.join(ROOT, "synth")

ARCH = os.environ.get("TP_OFFLOAD_ARCH", "gfx950")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 instructions stay off (see the design notes)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]
SOURCES = ["abi.cpp", "guide_scores.hip", "guide_attention.hip", "quantize.hip", "select.hip", "compact.hip"]
# The score passes see finite inputs only (the ABI's precondition; -inf marks masked logits),
# so max() need not quiet NaNs: this drops the canonicalising moves before every v_max.
EXTRA_FLAGS = {"guide_scores.hip": ["-fno-honor-nans"]}


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l and "warning generated" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build failed: {' '.join(cmd)}\n{out}")
    return out


def build_taskpress(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    os.makedirs(LIBDIR, exist_ok=True)
    objs = []
    cmds = []
    for src in SOURCES:
        obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        cmds.append([HIPCC, *HIP_FLAGS, *EXTRA_FLAGS.get(src, []), *lang, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(cmds))) as ex:
        for out in ex.map(_run, cmds):
            if verbose and out.strip():
                print(out)
    lib = os.path.join(LIBDIR, "libtaskpress.so")
    tmp = lib + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, lib)
    return lib


def build_rates() -> str:
    os.makedirs(LIBDIR, exist_ok=True)
    lib = os.path.join(LIBDIR, "libtprates.so")
    _run([HIPCC, *HIP_FLAGS, "-shared", "-x", "hip", os.path.join(CSRC, "microbench.hip"), "-o", lib + ".tmp"])
    os.replace(lib + ".tmp", lib)
    return lib


def build_synth() -> list[str]:
    host = os.path.join(SYNTH, "libtpsynth_host.so")
    dev = os.path.join(SYNTH, "libtpsynth_dev.so")
    _run(["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared",
          os.path.join(SYNTH, "synth_host.c"), "-o", host + ".tmp"])
    os.replace(host + ".tmp", host)
    _run([HIPCC, f"--offload-arch={ARCH}", "-O3", "-ffp-contract=off", "-fPIC", "-shared",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          os.path.join(SYNTH, "synth_dev.hip"), "-o", dev + ".tmp"])
    os.replace(dev + ".tmp", dev)
    return [host, dev]


def build_all(verbose: bool = False) -> list[str]:
    with cf.ThreadPoolExecutor(max_workers=3) as ex:
        f1 = ex.submit(build_taskpress, verbose)
        f2 = ex.submit(build_synth)
        f3 = ex.submit(build_rates)
        return [f1.result(), *f2.result(), f3.result()]


if __name__ == "__main__":
    for p in build_all(verbose=True):
        print("built", p)
