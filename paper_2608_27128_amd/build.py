"""Compile libtwinkv.so (HIP kernels for gfx950 + the C ABI host layer) in-tree.

    python -m paper_2608_27128_amd.build

Kernels (csrc/kernels/*.hip) are compiled by hipcc for gfx950 with packed-fp32 VALU
instructions disabled; the host layer (csrc/api.cpp) is plain C++ against the HIP
runtime API.  Everything is linked into paper_2608_27128_amd/libtwinkv.so.  A second copy
built with -DTWINKV_DEBUG (kernels that poison their LDS between uses, with extra barriers)
goes to paper_2608_27128_amd/libtwinkv_debug.so; only the tests load it.
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
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libtwinkv.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
ARCH = "gfx950"

HIP_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # no packed fp32 VALU instructions anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA results in architectural VGPRs, where the VALU epilogues read them
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",
    "-Wall", "-Wno-unused-function",
    f"-I{CSRC}", f"-I{os.path.join(ROOT, 'include')}",
]
CXX_FLAGS = [
    "-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
    f"-I{os.path.join(ROCM, 'include')}", f"-I{CSRC}", f"-I{os.path.join(ROOT, 'include')}",
]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    # the host pass does not know the device-only feature flag; that warning is expected
    noise = [ln for ln in r.stderr.splitlines() if ln.strip() and "packed-fp32-ops" not in ln
             and "is not a recognized feature" not in ln and "warning: " not in ln]
    if verbose and noise:
        print("\n".join(noise), file=sys.stderr)


DEBUG_LIB = os.path.join(HERE, "libtwinkv_debug.so")


def _build_one(lib: str, objdir: str, extra: list, verbose: bool) -> str:
    hipcc = os.path.join(ROCM, "bin", "hipcc")
    cxx = shutil.which("g++") or "g++"
    os.makedirs(objdir, exist_ok=True)
    jobs = []
    objs = []
    for src in sorted(glob.glob(os.path.join(CSRC, "kernels", "*.hip"))):
        obj = os.path.join(objdir, os.path.basename(src) + ".o")
        jobs.append([hipcc, *HIP_FLAGS, *extra, "-c", src, "-o", obj])
        objs.append(obj)
    api_obj = os.path.join(objdir, "api.cpp.o")
    jobs.append([cxx, *CXX_FLAGS, "-c", os.path.join(CSRC, "api.cpp"), "-o", api_obj])
    objs.append(api_obj)
    with ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        list(ex.map(lambda c: _run(c, verbose), jobs))
    tmp = lib + ".tmp"
    _run([hipcc, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp,
          f"-L{os.path.join(ROCM, 'lib')}", "-lamdhip64"], verbose)
    os.replace(tmp, lib)
    return lib


CLIENT_SRC = os.path.join(HERE, "examples", "repair_client.c")
CLIENT = os.path.join(BUILD, "repair_client")


def _build_client(verbose: bool) -> str:
    """The plain C example client (examples/repair_client.c), linked against libtwinkv.so
    (found next to the _build folder at run time) and the HIP runtime."""
    cc = shutil.which("gcc") or "gcc"
    tmp = CLIENT + ".tmp"
    _run([cc, "-std=c11", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
          f"-I{os.path.join(ROCM, 'include')}", f"-I{os.path.join(ROOT, 'include')}",
          CLIENT_SRC, "-o", tmp, f"-L{HERE}", "-ltwinkv", f"-L{os.path.join(ROCM, 'lib')}",
          "-lamdhip64", "-Wl,-rpath,$ORIGIN/..", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}"],
         verbose)
    os.replace(tmp, CLIENT)
    return CLIENT


def build(verbose: bool = False) -> str:
    """Compile every source and link libtwinkv.so, plus libtwinkv_debug.so (the LDS-poisoning
    build the tests compare against it, -DTWINKV_DEBUG) and the C example client; returns the
    library path."""
    _build_one(LIB, BUILD, [], verbose)
    _build_one(DEBUG_LIB, os.path.join(BUILD, "debug"), ["-DTWINKV_DEBUG"], verbose)
    _build_client(verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
