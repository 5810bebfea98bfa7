"""Build the gfx950 HIP libraries in-tree with hipcc: ``libapb.so`` (the C
ABI of ``include/apb.h``) and ``libapb_probe.so`` (the matrix-core ceiling
probe of ``include/apb_probe.h``, used by the benchmark only).

Usage: ``python -m paper_2502_12085_amd.build`` (or ``build()`` from
Python).  Always recompiles.
"""
from __future__ import annotations

import os
import shutil
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libapb.so")
SOURCES = ["apb_api.hip", "apb_attention.hip", "apb_compress.hip", "apb_decode.hip", "apb_scorer.hip",
           "apb_layer.hip"]
PROBE_LIB = os.path.join(PKG, "libapb_probe.so")
PROBE_SOURCES = ["probe_mfma.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the APB library needs ROCm's hipcc")


def compile_command(out: str = LIB, sources=None) -> list:
    sources = SOURCES if sources is None else sources
    return [
        hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
        # packed fp32 VALU forms stay off: ordinary scalar fp32 code only
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-Wall", "-Wno-unused-function",
        "-I", os.path.join(ROOT, "include"),
        "-o", out,
    ] + [os.path.join(CSRC, src) for src in sources]


def _build_one(out: str, sources, verbose: bool) -> str:
    tmp = out + ".tmp"
    cmd = compile_command(tmp, sources)
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + res.stdout + res.stderr)
    os.replace(tmp, out)
    return out


def build(verbose: bool = False) -> str:
    _build_one(PROBE_LIB, PROBE_SOURCES, verbose)
    return _build_one(LIB, SOURCES, verbose)


if __name__ == "__main__":
    print(build(verbose=True))
