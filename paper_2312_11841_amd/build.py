"""Build the gfx950 HIP library libmixrt.so in-tree with hipcc, and record
the compiler version and flags beside it (libmixrt.build.json), so that a
benchmark can report them without starting the compiler."""
import json
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libmixrt.so")
SOURCES = ["mixrt_api.cpp", "mixrt_mesh.cpp", "mixrt_render.hip", "mixrt_stages.hip",
           "mixrt_raycast.hip", "mixrt_raster.hip"]
MB_LIB = os.path.join(PKG, "libmixrt_microbench.so")
MB_SOURCES = ["microbench.hip"]
BUILD_INFO = os.path.join(PKG, "libmixrt.build.json")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=fast",
    # MFMA results in VGPRs: the MLP's ReLU and partial sums read them directly
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    # packed fp32 instructions stay off: plain float code only
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def build(verbose: bool = False, extra=()) -> str:
    _build_one(LIB, SOURCES, verbose, extra)
    _build_one(MB_LIB, MB_SOURCES, verbose, extra)
    _write_build_info(extra)
    return LIB


def _write_build_info(extra):
    r = subprocess.run([HIPCC, "--version"], capture_output=True, text=True)
    version = next((l.strip() for l in r.stdout.splitlines() if "HIP version" in l), None)
    info = {"hipcc": version, "flags": FLAGS + list(extra)}
    with open(BUILD_INFO + ".tmp", "w") as f:
        json.dump(info, f)
    os.replace(BUILD_INFO + ".tmp", BUILD_INFO)


def build_info() -> dict:
    """The record written by the last build (empty if there is none)."""
    try:
        with open(BUILD_INFO) as f:
            return json.load(f)
    except (OSError, ValueError):
        return {}


def _build_one(lib, sources, verbose, extra):
    tmp = lib + ".tmp"
    srcs = [os.path.join(CSRC, s) for s in sources]
    cmd = [HIPCC, *FLAGS, *extra, "-I", INCLUDE, "-I", CSRC, "-x", "hip", *srcs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in r.stderr.splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    os.replace(tmp, lib)


if __name__ == "__main__":
    extra = [a for a in sys.argv[1:] if a != "-v"]
    print(build(verbose=True, extra=extra))
