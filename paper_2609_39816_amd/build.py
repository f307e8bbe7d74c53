"""Builds libfm.so (HIP, gfx950) in place: paper_2609_39816_amd/libfm.so.

Every call compiles.  Translation units are compiled in parallel and
linked into one shared library.  Flags: gfx950 only, -ffp-contract=off (the
only fused operations are explicit fmaf calls), fp32 denormals kept, packed
fp32 instructions disabled.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libfm.so")
OBJ = os.path.join(HERE, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = ["-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-ffp-contract=off",
         "-fno-gpu-flush-denormals-to-zero", "-Xclang", "-target-feature", "-Xclang",
         "-packed-fp32-ops", "-Wno-pass-failed"]


def sources():
    fixed = ["fm_scheme.cpp", "fm_patterns.cpp", "fm_api.cpp", "fm_kernels.hip", "fm_gemm.hip", "fm_int8.hip",
             "fm_noalloc.hip"]
    fams = sorted(os.path.basename(p) for p in glob.glob(os.path.join(CSRC, "fm_fam_*.hip")))
    return fixed + fams


def _compile(src, extra, verbose):
    obj = os.path.join(OBJ, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, *extra, "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-c",
           os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"compiling {src} failed")
    return obj


def _stale(src):
    """True if the object is older than the source or any header it may use."""
    obj = os.path.join(OBJ, os.path.splitext(src)[0] + ".o")
    if not os.path.exists(obj):
        return True
    deps = [os.path.join(CSRC, src)] + glob.glob(os.path.join(CSRC, "*.h")) + \
        glob.glob(os.path.join(CSRC, "*.inc")) + [os.path.join(ROOT, "include", "fm.h")]
    t = os.path.getmtime(obj)
    return any(os.path.getmtime(d) > t for d in deps)


def build(verbose: bool = False, extra=(), jobs: int | None = None,
          only_stale: bool = False) -> str:
    """Compile every translation unit (only the out-of-date ones with
    only_stale=True) and link libfm.so."""
    subprocess.run([sys.executable, os.path.join(CSRC, "gen_patterns.py")], check=True)
    os.makedirs(OBJ, exist_ok=True)
    srcs = sources()
    todo = [s for s in srcs if _stale(s)] if only_stale else srcs
    jobs = jobs or min(len(srcs), max(1, min(16, os.cpu_count() or 1)))
    with ThreadPoolExecutor(jobs) as ex:
        list(ex.map(lambda s: _compile(s, extra, verbose), todo))
    objs = [os.path.join(OBJ, os.path.splitext(s)[0] + ".o") for s in srcs]
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError("linking libfm failed")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, only_stale="--stale" in sys.argv))
