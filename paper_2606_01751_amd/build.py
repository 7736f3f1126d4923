"""Builds libsx.so (the C-ABI library declared in include/sx.h) for gfx950 with hipcc, and beside it
libsx_checked.so: the same library with the device-side validation of index arrays
(SX_DEVICE_CHECKS: row lists and cu_seqlens checked before any kernel reads them, SX_EDEVICE).

Usage: python -m paper_2606_01751_amd.build [--debug]
Objects go to _build/ at the repository root; the libraries land next to this file.  --debug builds
both without optimisation.
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
LIB = os.path.join(PKG, "libsx.so")
LIB_CHECKED = os.path.join(PKG, "libsx_checked.so")


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def common_flags(debug: bool = False):
    return [
        "--offload-arch=gfx950", "-std=c++17", "-fPIC", "-O0" if debug else "-O3",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-I", INCLUDE, "-I", CSRC, "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
    ]


def _compile(src: str, debug: bool, checked: bool = False) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + (".checked.o" if checked else ".o"))
    cmd = [hipcc(), "-x", "hip", "-c", src, "-o", obj] + common_flags(debug) + (["-DSX_DEVICE_CHECKS=1"] if checked else [])
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return obj


def build(debug: bool = False, jobs: int = 8) -> str:
    os.makedirs(BUILD, exist_ok=True)
    sources = sorted(glob.glob(os.path.join(CSRC, "*.hip"))) + sorted(glob.glob(os.path.join(CSRC, "*.cpp")))
    host = os.path.join(CSRC, "sx_host.cpp")   # the only source the device checks change
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, debug), sources))
        host_checked = ex.submit(_compile, host, debug, True).result()
    _link(objs, LIB)
    _link([host_checked if o.endswith("sx_host.cpp.o") else o for o in objs], LIB_CHECKED)
    return LIB


def _link(objs, out: str) -> None:
    tmp = out + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp] + objs
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    os.replace(tmp, out)


if __name__ == "__main__":
    print(build(debug="--debug" in sys.argv))
