"""Build librbq.so (the HIP kernels + C ABI) in-tree for gfx950 with hipcc.

Usage: python -m paper_2606_31519_amd.build [-v]
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD_DIR = os.path.join(HERE, "_build")
LIB_PATH = os.path.join(HERE, "librbq.so")

HIP_SOURCES = ["api.hip", "score.hip", "quantize.hip", "encode.hip", "topp.hip", "decode.hip"]
CXX_SOURCES = ["validate.cpp"]          # plain C++ (no HIP): host-side argument checks

ARCH = "gfx950"


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build librbq.so)")


HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
    # no packed-fp32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]
CXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall"]
# per-source additions: the decode kernels keep their MFMA accumulators in
# ordinary VGPRs (the softmax rescales them with vector ALU ops; accumulation
# registers would cost copies and a wave per SIMD)
EXTRA_FLAGS = {"decode.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(line for line in r.stdout.splitlines() if "not a recognized feature" not in line)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out, flush=True)


def build(verbose: bool = False) -> str:
    """Compile every source and link librbq.so; returns the library path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    hipcc = _hipcc()
    jobs = []
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD_DIR, src.replace(".hip", ".o"))
        jobs.append([hipcc, *HIP_FLAGS, *EXTRA_FLAGS.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj])
    for src in CXX_SOURCES:
        obj = os.path.join(BUILD_DIR, src.replace(".cpp", ".o"))
        jobs.append(["g++", *CXX_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj])
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        list(ex.map(lambda c: _run(c, verbose), jobs))
    objs = [os.path.join(BUILD_DIR, s.rsplit(".", 1)[0] + ".o") for s in HIP_SOURCES + CXX_SOURCES]
    tmp = LIB_PATH + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs], verbose)
    os.replace(tmp, LIB_PATH)
    _write_build_info()
    return LIB_PATH


BUILD_INFO = os.path.join(HERE, "librbq.build.json")


def _write_build_info() -> None:
    """Beside the library: the commit it was built from (with whether the tree
    had uncommitted changes) and a hash of its sources, so that a run on a
    machine without the repository's history can still name what it ran."""
    import datetime
    import hashlib
    import json

    def git(*args):
        try:
            r = subprocess.run(["git", "-C", HERE, *args], capture_output=True, text=True, timeout=10)
            return r.stdout.strip() if r.returncode == 0 else None
        except Exception:
            return None

    h = hashlib.sha256()
    inc = os.path.join(os.path.dirname(HERE), "include")
    for d in (CSRC, inc):
        for name in sorted(os.listdir(d)):
            with open(os.path.join(d, name), "rb") as f:
                h.update(name.encode() + b"\0" + f.read())
    status = git("status", "--porcelain", "--", CSRC, inc)
    info = {"git": git("rev-parse", "--short=12", "HEAD"), "sources_dirty": bool(status) if status is not None else None,
            "sources_sha256": h.hexdigest(), "arch": ARCH,
            "built_utc": datetime.datetime.now(datetime.timezone.utc).strftime("%Y-%m-%dT%H:%M:%SZ")}
    with open(BUILD_INFO, "w") as f:
        json.dump(info, f)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
