"""Build the engine's shared library (HIP kernels + C++ host code) for gfx950.

    python -m paper_2609_27203_amd.build

Compiles every engine source under csrc/ with hipcc into libxlh.so next to
this file, and csrc/ceiling.hip (the measurement kernel bench.py prices the
frontier kernel against) into libxlh_ceiling.so.  Objects are cached under
_build/ and rebuilt when their source or any header changes.  hipcc
cross-compiles for gfx950 without a GPU present.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(os.path.dirname(HERE), "include")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libxlh.so")
# measurement kernels bench.py prices the engine's kernels against (not part of the engine)
CEILING_SRC, CEILING_LIB = "ceiling.hip", os.path.join(HERE, "libxlh_ceiling.so")
ARCH = os.environ.get("XLH_OFFLOAD_ARCH", "gfx950")

SOURCES = ["kernels.hip", "frontier.hip", "wcoj.hip", "coding.hip", "engine.cpp", "frontend.cpp", "api.cpp"]

COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # exact IEEE binary32 adds: no contraction, no packed-FP32 instruction forms
    "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}",
]


def _hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the engine is built with ROCm's hipcc for gfx950")


def _torch_lib_dir() -> str:
    """Directory of the HIP runtime that PyTorch loads (found without importing torch)."""
    import importlib.util
    spec = importlib.util.find_spec("torch")
    if spec is None or not spec.submodule_search_locations:
        raise RuntimeError("PyTorch (ROCm build) is required: it owns the device memory and streams")
    d = os.path.join(list(spec.submodule_search_locations)[0], "lib")
    if not os.path.exists(os.path.join(d, "libamdhip64.so")):
        raise RuntimeError(f"no libamdhip64.so under {d}: a ROCm build of PyTorch is required")
    return d


def _newest_header() -> float:
    paths = [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".h")]
    paths.append(os.path.join(INCLUDE, "xlh.h"))
    return max(os.path.getmtime(p) for p in paths)


def build(force: bool = False, verbose: bool = False) -> str:
    """Compile (incrementally unless force) and link libxlh.so; returns its path."""
    hipcc = _hipcc()
    os.makedirs(BUILD, exist_ok=True)
    hdr = _newest_header()
    objs, cmds = [], []
    for src in SOURCES + [CEILING_SRC]:
        s = os.path.join(CSRC, src)
        o = os.path.join(BUILD, src + ".o")
        objs.append(o)
        if not force and os.path.exists(o) and os.path.getmtime(o) >= max(os.path.getmtime(s), hdr):
            continue
        lang = [] if src.endswith(".hip") else ["-x", "hip"]
        cmds.append([hipcc, *COMMON, *lang, "-c", s, "-o", o])
    # the sources compile independently: one hipcc per source, in parallel
    jobs = max(1, min(len(cmds), int(os.environ.get("MAX_JOBS", os.cpu_count() or 1))))

    def compile_one(cmd):
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)

    if cmds:
        with ThreadPoolExecutor(jobs) as ex:
            list(ex.map(compile_one, cmds))
    # Link with the host linker against the exact HIP runtime PyTorch loads, so
    # the process holds one runtime and torch's streams and allocations are
    # valid in the library (hipcc would add /opt/rocm's runtime instead).
    tlib = _torch_lib_dir()
    for out, lib_objs in ((LIB, objs[:len(SOURCES)]), (CEILING_LIB, objs[len(SOURCES):])):
        tmp = out + ".tmp"
        cmd = ["g++", "-shared", "-fPIC", *lib_objs, "-o", tmp, f"-L{tlib}", "-l:libamdhip64.so",
               f"-Wl,-rpath,{tlib}", "-Wl,--no-undefined"]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        os.replace(tmp, out)
    return LIB


if __name__ == "__main__":
    print(build(force="--force" in sys.argv, verbose=True))
