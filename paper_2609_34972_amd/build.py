"""Build ``libdeltavision.so`` (gfx950) in-tree with hipcc.

Each source is compiled to an object in ``_build/`` in parallel, then linked.
Packed-fp32 VALU instructions are disabled for every device compilation.
"""
from __future__ import annotations

import hashlib
import json
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libdeltavision.so")
INFO = os.path.join(HERE, "build_info.json")
SOURCES = ["api.cpp", "build_kernels.hip", "attention.hip", "recurrent.hip", "delta_rule.hip",
           "probe.hip", "fused_kv.hip"]
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function"]
# The VGPR form of the MFMA instructions keeps accumulators out of the AGPR file. Kernels that
# work on their accumulators with VALU inside their main loops (online softmax, the delta-rule
# chain) otherwise pay a copy each way per element and step; the dense GEMM main loops compile
# to the same code either way.
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-mllvm", "-amdgpu-mfma-vgpr-form"]


def _compile(src: str) -> str:
    out = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC] + COMMON + DEVICE + ["-I", CSRC, "-c", os.path.join(CSRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"hipcc failed on {src}")
    # hipcc's host pass does not know the device feature flag; that warning is harmless
    noise = [ln for ln in (r.stderr or "").splitlines()
             if ln.strip() and "packed-fp32-ops" not in ln]
    if noise:
        sys.stderr.write("\n".join(noise) + "\n")
    return out


def sources_digest() -> str:
    """Short sha256 over the library's sources (and this build script)."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)) + [os.path.join("..", "build.py")]:
        path = os.path.join(CSRC, name)
        if os.path.isfile(path):
            with open(path, "rb") as f:
                h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def _write_build_info() -> None:
    """Record which sources the library was built from (read by the benchmark, which runs where
    no git metadata is available)."""
    def git(*a):
        try:
            r = subprocess.run(["git", *a], cwd=HERE, capture_output=True, text=True, timeout=10)
            return r.stdout.strip() if r.returncode == 0 else None
        except (OSError, subprocess.SubprocessError):
            return None
    info = {"git_rev": git("rev-parse", "HEAD"),
            "git_dirty": bool(git("status", "--porcelain", "--", "."))
            if git("rev-parse", "HEAD") else None,
            "sources_sha256_16": sources_digest(), "arch": ARCH}
    with open(INFO, "w") as f:
        json.dump(info, f)


def build() -> str:
    """Compile every HIP source for gfx950 and link the shared library. Returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(len(SOURCES)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    _write_build_info()
    return LIB


if __name__ == "__main__":
    print(build())
