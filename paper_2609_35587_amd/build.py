"""Build libhwsel.so (the HIP kernels and the C ABI) for gfx950, in-tree.

Every translation unit is compiled with hipcc for gfx950 only; packed-fp32
instructions are disabled; the feature and evaluation units are also compiled
without multiply-add contraction (their binary64 sequences are part of their
contract).
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libhwsel.so")
# measured ceilings for the benchmark's rooflines: a library of its own
CEIL_SRC, CEIL_LIB = "ceilings.hip", os.path.join(HERE, "libhwsel_ceilings.so")
ARCH = "gfx950"
SOURCES = ["api.hip", "catalogue.hip", "evaluate.hip", "features.hip", "forest.hip", "mlp.hip", "scorers.hip",
           "select.hip"]
COMMON = ["-O3", "-std=c++20", "-fPIC", f"--offload-arch={ARCH}", "-fno-fast-math",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wall", "-Wno-unused-function", "-Wno-unknown-pragmas"]
PER_FILE = {"features.hip": ["-ffp-contract=off"], "evaluate.hip": ["-ffp-contract=off"]}


def hipcc() -> str:
    return os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, src.replace(".hip", ".o"))
    cmd = [hipcc(), *COMMON, *PER_FILE.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    if r.stderr.strip():
        sys.stderr.write(r.stderr)
    return obj


def build(jobs: int = 8) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(_compile, SOURCES + [CEIL_SRC]))
    ceil_obj = objs.pop()
    for out, parts in ((LIB, objs), (CEIL_LIB, [ceil_obj])):
        tmp = out + f".tmp{os.getpid()}"
        subprocess.run([hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", *parts, "-o", tmp], check=True)
        os.replace(tmp, out)
    return LIB


if __name__ == "__main__":
    print(build())
