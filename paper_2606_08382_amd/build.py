"""Build libstarkv.so (HIP for gfx950) in-tree with hipcc.

The decode split kernel is compiled once per (head_dim, cache precision) so the
translation units build in parallel.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libstarkv.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
         "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
         # packed fp32 arithmetic stays off (hipcc's host pass warns it does not know it)
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]

UNITS = [("starkv_host.cpp", []), ("append.hip", []), ("output.hip", []), ("stream.hip", []),
         ("decode.hip", ["-DSK_COMMON"])]
UNITS += [("decode.hip", [f"-DSK_D={d}", f"-DSK_QM={q}"]) for d in (64, 128) for q in (0, 1, 2, 3)]


def _obj_name(src: str, defs) -> str:
    tag = "_".join(d.replace("-D", "").replace("=", "") for d in defs)
    return os.path.join(BUILD, os.path.splitext(src)[0] + ("_" + tag if tag else "") + ".o")


def _compile(unit):
    src, defs = unit
    obj = _obj_name(src, defs)
    cmd = [HIPCC, *FLAGS, *defs, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src} {defs}:\n{msg}")
    return obj


def build(verbose: bool = False, jobs: int = 8) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, UNITS))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True, jobs=int(sys.argv[1]) if len(sys.argv) > 1 else 8)
