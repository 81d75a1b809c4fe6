"""Build the DAVET HIP library (libdavet.so) in-tree for gfx950.

Device sources (*.hip) and the HIP-runtime host sources are compiled with
hipcc for gfx950 only; the allocation policy is compiled with g++ and
-ffp-contract=off so its double arithmetic is never contracted into fused
multiply-adds.  Usage: ``python paper_2608_01821_amd/build.py`` (run by
path: importing the package would load the old library first).
"""

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INC = os.path.join(ROOT, "include")
OUT_DIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libdavet.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")

HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++17",
    # no packed-fp32 instructions anywhere in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + INC, "-I" + CSRC, "-Wno-unused-result",
]
POLICY_FLAGS = [
    "-O2", "-fPIC", "-std=c++17", "-ffp-contract=off",
    "-I" + INC, "-I" + os.path.join(ROCM, "include"),
    "-D__HIP_PLATFORM_AMD__",
]

HIP_SOURCES = ["views.hip", "realizers.hip", "unmask.hip", "rowops.hip", "gemm16.hip",
               "gemm_f32.hip", "attention.hip", "step.hip", "policy_dev.hip",
               "runtime.cpp",
               "schedule.cpp"]
POLICY_SOURCES = ["policy.cpp", "parser.cpp"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                       text=True)
    out = "\n".join(l for l in r.stdout.splitlines()
                    if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError("command failed: %s\n%s" % (" ".join(cmd), out))
    return out


def build(verbose: bool = False) -> str:
    """Compile every source and link libdavet.so; returns the library path."""
    os.makedirs(OUT_DIR, exist_ok=True)
    jobs = []
    for src in HIP_SOURCES:
        obj = os.path.join(OUT_DIR, src.rsplit(".", 1)[0] + ".o")
        cmd = [HIPCC] + HIP_FLAGS + ["-c", os.path.join(CSRC, src), "-o", obj]
        if src.endswith(".cpp"):
            cmd = [HIPCC] + HIP_FLAGS + ["-x", "hip", "-c",
                                         os.path.join(CSRC, src), "-o", obj]
        jobs.append((obj, cmd))
    for src in POLICY_SOURCES:
        obj = os.path.join(OUT_DIR, src.rsplit(".", 1)[0] + ".o")
        jobs.append((obj, ["g++"] + POLICY_FLAGS +
                     ["-c", os.path.join(CSRC, src), "-o", obj]))
    workers = min(len(jobs), max(1, min(8, os.cpu_count() or 1)))
    with cf.ThreadPoolExecutor(workers) as ex:
        outs = list(ex.map(lambda j: _run(j[1]), jobs))
    if verbose:
        for o in outs:
            if o.strip():
                print(o)
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] +
         [j[0] for j in jobs])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
