"""Build libpard.so (gfx950) from the HIP sources in this directory.

Usage: python -m paper_2504_18583_amd.csrc.build   (or call build()).
Objects go to ``_build/`` beside the package; the shared library is written
into the package directory, where the binding loads it from.  The same call
links ``gemm_counters`` (a stand-alone launch of the gate/up GEMM) and
``layer_counters`` (stand-alone launches of the one-launch decode layer) from
the GEMM object, and ``step_counters`` (whole decode steps through the C ABI)
against the library, for hardware-counter runs, and ``mfma_peak`` (the
attainable rate of the GEMMs' MFMA instructions).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
PKG = os.path.dirname(HERE)
ROOT = os.path.dirname(PKG)
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libpard.so")
COUNTERS_EXE = os.path.join(PKG, "gemm_counters")
LAYER_EXE = os.path.join(PKG, "layer_counters")
STEP_EXE = os.path.join(PKG, "step_counters")
MFMA_EXE = os.path.join(PKG, "mfma_peak")

SOURCES = ["engine.hip", "gemm.hip", "attention.hip", "device_init.hip", "cod.hip", "gemm_counters.hip",
           "layer_counters.hip", "step_counters.hip", "mfma_peak.hip"]
LIB_SOURCES = SOURCES[:5]

HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-function",
    # packed fp32 VALU ops are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{os.path.join(ROOT, 'include')}",
]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *CFLAGS, "-c", os.path.join(HERE, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    noise = "is not a recognized feature for this target"
    warn = "\n".join(l for l in res.stderr.splitlines() if noise not in l and l.strip())
    if warn:
        print(warn, file=sys.stderr)
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(len(SOURCES)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    obj = dict(zip(SOURCES, objs))
    _link(LIB, ["-shared", "-fPIC"], [obj[s] for s in LIB_SOURCES])
    _link(COUNTERS_EXE, [], [obj["gemm_counters.hip"], obj["gemm.hip"]])
    _link(LAYER_EXE, [], [obj["layer_counters.hip"], obj["gemm.hip"]])
    _link(STEP_EXE, [f"-L{PKG}", "-Wl,-rpath,$ORIGIN"], [obj["step_counters.hip"], "-lpard"])
    _link(MFMA_EXE, [], [obj["mfma_peak.hip"]])
    if verbose:
        print(f"built {LIB}, {COUNTERS_EXE}, {LAYER_EXE}, {STEP_EXE} and {MFMA_EXE}")
    return LIB


def _link(out: str, flags: list, objs: list) -> None:
    tmp = out + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", *flags, "-o", tmp, *objs]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"linking {os.path.basename(out)} failed:\n{' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, out)


if __name__ == "__main__":
    build(verbose=True)
