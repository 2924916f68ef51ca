"""Build libsd.so (HIP kernels + C ABI) for gfx950, in-tree.

Every .hip file under csrc/ is compiled by hipcc for gfx950, every .cpp file
(host-only code: the serving scheduler) by g++, and the objects are linked
into paper_2510_11331_amd/libsd.so.  The HIP runtime is recorded
as the unversioned ``libamdhip64.so`` (the name PyTorch-ROCm loads from its
own lib directory), so a process that already runs torch shares one HIP
runtime with libsd; outside such a process the rpath finds ROCm's copy.
"""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT = os.path.join(HERE, "libsd.so")
BUILD_DIR = os.path.join(HERE, "_build")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-fPIC", "-std=c++20",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
    "-I", INCLUDE, "-I", CSRC,
]


GXX_FLAGS = ["-O2", "-fPIC", "-std=c++17", "-Wall", "-I", INCLUDE, "-I", CSRC]


def _hip_runtime_dir() -> str:
    """Directory whose libamdhip64.so carries no soname (PyTorch's), so the
    link records the unversioned name; falls back to ROCm's."""
    try:
        import importlib.util
        spec = importlib.util.find_spec("torch")
        if spec and spec.origin:
            d = os.path.join(os.path.dirname(spec.origin), "lib")
            if os.path.exists(os.path.join(d, "libamdhip64.so")):
                return d
    except Exception:
        pass
    return os.path.join(ROCM, "lib")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"build step failed: {' '.join(cmd[:3])} ...")
    return r


def build(verbose: bool = False, jobs: int = 8) -> str:
    hipcc = shutil.which("hipcc") or os.path.join(ROCM, "bin", "hipcc")
    os.makedirs(BUILD_DIR, exist_ok=True)
    # HIP sources (kernels + host runtime) with hipcc; host-only C++ (the
    # serving scheduler) with g++
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip"))) + sorted(glob.glob(os.path.join(CSRC, "*.cpp")))
    objs = [os.path.join(BUILD_DIR, os.path.splitext(os.path.basename(s))[0] + ".o") for s in srcs]

    def compile_one(so):
        s, o = so
        if s.endswith(".cpp"):
            _run(["g++", *GXX_FLAGS, "-c", s, "-o", o], verbose)
        else:
            _run([hipcc, *HIPCC_FLAGS, "-c", s, "-o", o], verbose)

    with ThreadPoolExecutor(max_workers=max(1, min(jobs, len(srcs)))) as ex:
        list(ex.map(compile_one, zip(srcs, objs)))
    rt = _hip_runtime_dir()
    tmp = OUT + ".tmp"
    _run(["g++", "-shared", "-fPIC", "-o", tmp, *objs, f"-L{rt}", "-lamdhip64",
          f"-Wl,-rpath,{ROCM}/lib", "-Wl,--no-undefined"], verbose)
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
