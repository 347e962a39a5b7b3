"""Build libeldr_moe.so (gfx950) in-tree: csrc/*.hip with hipcc, and the
host-only csrc/*.cpp (the routing library) with the host C++ compiler.

    python -m paper_2607_00466_amd.build

Every call compiles: each source to an object under _build/ (in parallel),
then one shared library next to this file.
"""
from __future__ import annotations

import concurrent.futures as cf
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
LIB = os.path.join(PKG, "libeldr_moe.so")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CXX = os.environ.get("CXX_HOST", "g++")
CXXFLAGS = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-I", INCLUDE, "-I", CSRC]
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-Wno-unused-result",
    # keep the compiler from emitting packed-fp32 VALU instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
]


# The compiler reports every kernel's resources; the build fails on scratch
# or vector register spills in any kernel, and on an FFN kernel held to one
# wave a SIMD (its LDS allows two workgroups a CU, so more registers than two
# waves a SIMD leave halve its loads in flight).  Scalar spills go to vector
# register lanes, not memory, and are allowed.
RESOURCE_FLAG = "-Rpass-analysis=kernel-resource-usage"
_REMARK = re.compile(r"remark:\s+(Function Name|ScratchSize \[bytes/lane\]|VGPRs Spill|"
                     r"Occupancy \[waves/SIMD\]): (\S+)")


def _resource_problems(stderr: str) -> list[str]:
    problems, name = [], None
    for m in _REMARK.finditer(stderr):
        key, val = m.group(1), m.group(2)
        if key == "Function Name":
            name = val
        elif key.startswith("Occupancy"):
            if "ffn_" in (name or "") and int(val) < 2:
                problems.append(f"{name}: occupancy {val} wave a SIMD")
        elif int(val) != 0:
            problems.append(f"{name}: {key} {val}")
    return problems


def _run(cmd: list[str]) -> None:
    r = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass warns that it does not know the packed-fp32 feature; drop that line
    noise = "is not a recognized feature for this target"
    lines = [l for l in r.stderr.splitlines() if noise not in l]
    err = "\n".join(l for l in lines if "kernel-resource-usage" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{err}")
    problems = _resource_problems(r.stderr) if RESOURCE_FLAG in cmd else []
    if problems:
        raise RuntimeError("kernel resources: " + "; ".join(problems))
    # (the remarks' source excerpts and carets are dropped with them)
    err = "\n".join(l for l in err.splitlines() if l.strip() and not l.lstrip().startswith(("|", "^")) and
                    not re.match(r"\s*\d+ \|", l))
    if err.strip():
        print(err, file=sys.stderr)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    host = sorted(glob.glob(os.path.join(CSRC, "*.cpp")))
    objs = [os.path.join(BUILD, os.path.basename(s) + ".o") for s in srcs + host]
    jobs = [[HIPCC, *FLAGS, RESOURCE_FLAG, "-c", s, "-o", o] for s, o in zip(srcs, objs)]
    jobs += [[CXX, *CXXFLAGS, "-c", s, "-o", o] for s, o in zip(host, objs[len(srcs):])]
    with cf.ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        for f in [ex.submit(_run, j) for j in jobs]:
            f.result()
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
