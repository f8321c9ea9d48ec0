"""Build libvla.so (gfx950) in-tree.

    python paper_2609_22335_amd/build.py

hipcc cross-compiles for gfx950 without a GPU. The counter-based generator is
plain host C++ built by g++ without floating-point contraction, so its values
match the seeded generator of the tests bit for bit.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
ROOT = os.path.dirname(HERE)
OUT = os.path.join(HERE, "libvla.so")
BUILD = os.path.join(ROOT, "_build")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
HIP_FLAGS = [
    "-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC",
    "-I" + os.path.join(ROOT, "include"),
    # packed fp32 VALU forms stay off (hipcc -O3 would otherwise emit them)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result", "-Wno-unused-value",
]


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if p.returncode != 0:
        raise RuntimeError("build step failed:\n" + " ".join(cmd) + "\n" + p.stdout)
    return p.stdout


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    gen_o = os.path.join(BUILD, "gen.o")
    jobs = [
        ["g++", "-O2", "-std=c++17", "-fPIC", "-ffp-contract=off", "-c",
         os.path.join(CSRC, "gen.cpp"), "-o", gen_o],
    ]
    objs = [gen_o]
    for src in ("kernels.hip", "runtime.hip"):
        o = os.path.join(BUILD, src.replace(".hip", ".o"))
        jobs.append([HIPCC, *HIP_FLAGS, "-c", os.path.join(CSRC, src), "-o", o])
        objs.append(o)
    with ThreadPoolExecutor(len(jobs)) as ex:
        logs = list(ex.map(_run, jobs))
    tmp = OUT + ".tmp"
    logs.append(_run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp,
                      "-lpthread"]))
    shutil.move(tmp, OUT)
    if verbose:
        for l in logs:
            if l.strip():
                print(l)
    return OUT


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
