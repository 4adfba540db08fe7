"""Builds ``libams.so`` (HIP kernels + host engine + C ABI) for gfx950 with hipcc.

Usage: ``python -m paper_2508_10259_amd.build`` (or ``__graft_entry__.build()``).
Objects go to ``_build/`` at the repository root; the shared library is
written next to this file, where the binding loads it from.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libams.so")
PROBE_LIB = os.path.join(PKG, "libams_probe.so")

ARCH = "gfx950"
HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-result",
    # gfx950 packed fp32 arithmetic stays disabled (plain fp32 VALU instead)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}", f"-I{os.path.join(CSRC, 'host')}", f"-I{os.path.join(CSRC, 'kernels')}",
]


def hipcc() -> str:
    p = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(p):
        raise RuntimeError("hipcc not found")
    return p


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "kernels", "*.hip"))) + \
        sorted(glob.glob(os.path.join(CSRC, "host", "*.cpp")))


def _spills(remarks: str):
    """Kernels whose register allocation spills to scratch (from the resource-usage remarks).
    SGPR spills that land in VGPR lanes (scratch size 0) stay in registers and pass."""
    bad, name = [], None
    for line in remarks.splitlines():
        if "Function Name:" in line:
            name = line.split("Function Name:")[1].split("[")[0].strip()
        for key in ("VGPRs Spill:", "ScratchSize [bytes/lane]:"):
            if key in line:
                v = line.split(key)[1].split("[")[0].strip()
                if v.isdigit() and int(v) > 0:
                    bad.append(f"{name}: {key} {v}")
    return bad


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD, os.path.relpath(src, CSRC).replace(os.sep, "_") + ".o")
    cmd = [hipcc()] + HIP_FLAGS + ["-c", src, "-o", obj]
    if src.endswith(".hip"):
        cmd.append("-Rpass-analysis=kernel-resource-usage")
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    lines = [l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l]
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {src}\n" + "\n".join(lines))
    # every kernel must run from registers: a spill to scratch is a build error
    spills = _spills("\n".join(lines))
    if spills:
        raise RuntimeError(f"register spills in {src}:\n" + "\n".join(spills))
    other = [l for l in lines if "kernel-resource-usage" not in l]
    if other and verbose:
        print("\n".join(other))
    return obj


def _link(objs, lib: str) -> None:
    tmp = lib + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed\n" + r.stdout)
    os.replace(tmp, lib)


def build(verbose: bool = False, jobs: int = 8) -> str:
    """Compile every source and link ``libams.so`` (and the test-only
    ``libams_probe.so`` over the same kernel objects); always rebuilds."""
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    probe = sorted(glob.glob(os.path.join(CSRC, "probe", "*.cpp")))
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), srcs + probe))
    main_objs, probe_objs = objs[:len(srcs)], objs[len(srcs):]
    _link(main_objs, LIB)
    kernel_objs = [o for o, s in zip(main_objs, srcs) if s.endswith(".hip")]
    _link(kernel_objs + probe_objs, PROBE_LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
