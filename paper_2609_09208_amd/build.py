"""Build libpotattn.so (gfx950) in-tree with hipcc.

Flags: -O3 for gfx950 only; -ffp-contract=off so that every fp32 operation in
the exact parts (query quantiser, log2-domain score, encoder decisions) is one
correctly rounded IEEE operation; fp32 denormals preserved; packed-fp32
instructions disabled in code generation.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libpotattn.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-ffp-contract=off", "-fno-gpu-flush-denormals-to-zero",
    "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
]


def sources():
    csrc = os.path.join(PKG, "csrc")
    return sorted(glob.glob(os.path.join(csrc, "*.hip")) + glob.glob(os.path.join(csrc, "*.cpp")))


def _compile(src: str, obj: str) -> tuple[int, str]:
    cmd = [HIPCC, *FLAGS, "-c", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(PKG, "csrc"), "-o", obj, src]
    res = subprocess.run(cmd, capture_output=True, text=True)
    return res.returncode, res.stderr


def build(verbose: bool = False, jobs: int | None = None) -> str:
    """Compile every source (in parallel, one object each) and link
    libpotattn.so (always recompiles)."""
    from concurrent.futures import ThreadPoolExecutor
    srcs = sources()
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)
    objs = [os.path.join(objdir, os.path.basename(s) + ".o") for s in srcs]
    jobs = jobs or max(1, min(len(srcs), os.cpu_count() or 1, 16))
    with ThreadPoolExecutor(jobs) as ex:
        results = list(ex.map(_compile, srcs, objs))
    failed = False
    for src, (rc, err) in zip(srcs, results):
        errs = [ln for ln in err.splitlines() if "packed-fp32-ops" not in ln and ln.strip()]
        if rc != 0:
            failed = True
            sys.stderr.write(f"--- {os.path.basename(src)}\n{err}")
        elif verbose and errs:
            sys.stderr.write("\n".join(errs) + "\n")
    if failed:
        raise RuntimeError("hipcc failed building libpotattn.so")
    out_tmp = LIB + ".tmp"
    link = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", out_tmp, *objs]
    res = subprocess.run(link, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stderr)
        raise RuntimeError("linking libpotattn.so failed")
    os.replace(out_tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
