"""Compile libdlfp.so (HIP for gfx950) in-tree.

Usage: ``python -m paper_2609_38386_amd.build`` or ``build_library()``.
Always recompiles; the result lands next to this file.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_PATH = os.path.join(HERE, "libdlfp.so")
ARCH = "gfx950"

SOURCES = ["dlfp_host.cpp", "dlfp_timer.cpp", "kv_append.hip", "attention_mixed.hip", "stream_hold.hip",
           "linear.hip"]

# Packed FP32 instructions are kept out of device code.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", f"-I{INCLUDE}", f"-I{CSRC}",
          "-Wall", "-Wno-unused-function"]


def _hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found; the HIP library cannot be built")


PROBE_SOURCES = ["probes.hip"]
PROBE_LIB_PATH = os.path.join(HERE, "libdlfp_probe.so")


def build_probes(verbose: bool = False) -> str:
    """libdlfp_probe.so: the achievable-ceiling probes (measurement only)."""
    return _build(PROBE_SOURCES, PROBE_LIB_PATH, verbose, 1)


def build_library(verbose: bool = False, jobs: int = 3) -> str:
    return _build(SOURCES, LIB_PATH, verbose, jobs)


def _build(sources, lib_path, verbose: bool, jobs: int) -> str:
    hipcc = _hipcc()
    tmp = tempfile.mkdtemp(prefix="dlfp_build_")
    try:
        objs, procs = [], []
        for src in sources:
            obj = os.path.join(tmp, src + ".o")
            lang = ["-x", "hip"]
            cmd = [hipcc, *COMMON, *DEVICE_FLAGS, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE,
                                                stderr=subprocess.STDOUT, text=True)))
            objs.append(obj)
            if len(procs) >= jobs:
                _drain(procs, verbose)
        _drain(procs, verbose)
        out_tmp = lib_path + ".tmp"
        cmd = [hipcc, "-shared", f"--offload-arch={ARCH}", *objs, "-o", out_tmp]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
        if r.returncode != 0:
            raise RuntimeError("link failed:\n" + r.stdout)
        os.replace(out_tmp, lib_path)
        return lib_path
    finally:
        shutil.rmtree(tmp, ignore_errors=True)


def _drain(procs, verbose):
    while procs:
        src, p = procs.pop(0)
        out, _ = p.communicate()
        msg = "\n".join(line for line in out.splitlines()
                        if "packed-fp32-ops" not in line and "--hip-link" not in line)
        if p.returncode != 0:
            raise RuntimeError(f"compiling {src} failed:\n{msg}")
        if verbose and msg.strip():
            print(msg, flush=True)


if __name__ == "__main__":
    path = build_library(verbose="-v" in sys.argv)
    print(path)
    print(build_probes(verbose="-v" in sys.argv))
