"""Build liblora_mi355x.so (HIP for gfx950) in-tree with hipcc, and its debug
build liblora_mi355x_debug.so (the same sources with LORA_DEBUG=1: the ops'
output/input overlap checks and the kernels' bounds checks of plan values).

Every call recompiles.  Objects go to paper_2601_07376_amd/_build/ (release)
and _build/debug/; the shared libraries land next to this file, where the
binding loads them.
"""
import concurrent.futures
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "liblora_mi355x.so")
DEBUG_LIB = os.path.join(HERE, "liblora_mi355x_debug.so")
SOURCES = ["plan.hip", "fwd_mfma.hip", "fwd_valu.hip", "grad.hip", "adamw.hip", "losses.hip",
           "noalloc.hip", "linear.hip", "calib.hip", "api.cpp"]
ARCH = "gfx950"

# Packed fp32 VALU instructions are disabled for all device code.
COMMON = ["-O3", "-std=c++17", "-fPIC", f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}",
          "-Wall", "-Wno-unused-function"]
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build the HIP library)")


def _compile(hipcc, src, debug, verbose):
    out = os.path.join(BUILD, "debug") if debug else BUILD
    obj = os.path.join(out, os.path.splitext(src)[0] + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    flags = COMMON + (["-DLORA_DEBUG=1"] if debug else [])
    cmd = [hipcc] + flags + DEVICE + lang + ["-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{out}")
    if out.strip() and verbose:
        print(out, flush=True)
    return obj


def _link(hipcc, objs, lib, verbose):
    tmp = lib + ".tmp"
    cmd = [hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, lib)
    return lib


def build(verbose=False, jobs=None, debug=None):
    """Compile every HIP/C++ source for gfx950 and link the shared libraries:
    debug=None both, False the release library only, True the debug one only.
    Returns the path of the release library (the debug one's when debug=True)."""
    hipcc = _hipcc()
    kinds = [False, True] if debug is None else [bool(debug)]
    for k in kinds:
        os.makedirs(os.path.join(BUILD, "debug") if k else BUILD, exist_ok=True)
    work = [(s, k) for k in kinds for s in SOURCES]
    jobs = jobs or min(len(work), os.cpu_count() or 1, 8)
    with concurrent.futures.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda w: _compile(hipcc, w[0], w[1], verbose), work))
    libs = []
    for k in kinds:
        mine = [o for (s, kk), o in zip(work, objs) if kk == k]
        libs.append(_link(hipcc, mine, DEBUG_LIB if k else LIB, verbose))
    return libs[0]


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
