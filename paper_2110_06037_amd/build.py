"""Builds libsoftneuro.so (C ABI + HIP kernels for gfx950) in-tree.

Every source is compiled by hipcc with packed-FP32 instruction generation
disabled; objects go to ``_build/`` at the repository root and the shared
library next to this file.
"""

from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OBJ = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libsoftneuro.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-mllvm", "-amdgpu-mfma-vgpr-form=1",
         "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
         "-I" + os.path.join(ROOT, "include")]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.cpp")) + glob.glob(os.path.join(CSRC, "*.hip")) +
                  glob.glob(os.path.join(CSRC, "kernels", "*.hip")))


def _up_to_date(src, obj):
    """Whether obj is newer than src and every header its dependency file lists."""
    dep = obj + ".d"
    if not (os.path.exists(obj) and os.path.exists(dep)):
        return False
    t = os.path.getmtime(obj)
    with open(dep) as f:
        text = f.read().replace("\\\n", " ")
    files = text.split(":", 1)[1].split() if ":" in text else [src]
    return all(os.path.exists(p) and os.path.getmtime(p) <= t for p in files)


def _compile(src, incremental=False):
    rel = os.path.relpath(src, CSRC).replace(os.sep, "_")
    obj = os.path.join(OBJ, rel + ".o")
    if incremental and _up_to_date(src, obj):
        return src, obj, 0, ""
    cmd = [HIPCC] + FLAGS + ["-MMD", "-MF", obj + ".d", "-c", src, "-o", obj]
    if src.endswith(".hip"):
        cmd[1:1] = ["-x", "hip"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    return src, obj, r.returncode, err


def build(verbose=False, jobs=None, incremental=False):
    """Compiles every source (incremental=True skips objects newer than their
    source and headers) and links the library."""
    os.makedirs(OBJ, exist_ok=True)
    srcs = sources()
    jobs = jobs or min(len(srcs), max(1, (os.cpu_count() or 4)), 16)
    objs = []
    failed = []
    with cf.ThreadPoolExecutor(jobs) as ex:
        for src, obj, rc, err in ex.map(lambda s: _compile(s, incremental), srcs):
            objs.append(obj)
            if rc != 0:
                failed.append((src, err))
            elif verbose and err.strip():
                print(err, file=sys.stderr)
    if failed:
        msg = "\n\n".join(f"{s}:\n{e}" for s, e in failed)
        raise RuntimeError("HIP build failed:\n" + msg)
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True, incremental="--incremental" in sys.argv))
