"""Build the gfx950 HIP library libmixrt.so in-tree with hipcc, and record
the compiler version and flags beside it (libmixrt.build.json), so that a
benchmark can report them without starting the compiler.

Also built: libmixrt_microbench.so (roofline microbenchmarks) and the
profiling variants of libmixrt.so, which differ from it only in the render
kernel, compiled from the same source with one -D option (see
mixrt_render.hip): libmixrt_split_nodisp.so, libmixrt_split_nohash.so,
libmixrt_split_nomlp.so (a stage removed) and libmixrt_timer.so (per-phase
clock counters).  Objects go to _build/ and are compiled in parallel."""
import json
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJ_DIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libmixrt.so")
COMMON_SOURCES = ["mixrt_api.cpp", "mixrt_mesh.cpp", "mixrt_stages.hip", "mixrt_raycast.hip",
                  "mixrt_raster.hip"]
RENDER_SOURCE = "mixrt_render.hip"
SOURCES = COMMON_SOURCES + [RENDER_SOURCE]
MB_LIB = os.path.join(PKG, "libmixrt_microbench.so")
MB_SOURCES = ["microbench.hip"]
BUILD_INFO = os.path.join(PKG, "libmixrt.build.json")
# profiling variant -> the -D option its render kernel is compiled with
VARIANTS = {
    "split_nodisp": "MIXRT_SPLIT_NO_DISP",
    "split_nohash": "MIXRT_SPLIT_NO_HASH",
    "split_nomlp": "MIXRT_SPLIT_NO_MLP",
    "timer": "MIXRT_PHASE_TIMER",
}

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
LINK_FLAGS = ["--offload-arch=gfx950", "-fPIC", "-shared"]
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # a*b + c is fused into one fma within an expression only, so every
    # kernel that inlines a device function rounds it the same way (the
    # render kernel's two paths give bitwise-identical frames)
    "-ffp-contract=on",
    # MFMA results in VGPRs: the MLP's ReLU and partial sums read them directly
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    # packed fp32 instructions stay off: plain float code only
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def variant_lib(name: str) -> str:
    """Path of a profiling variant of libmixrt.so."""
    return os.path.join(PKG, f"libmixrt_{name}.so")


def build(verbose: bool = False, extra=(), variants: bool = True) -> str:
    os.makedirs(OBJ_DIR, exist_ok=True)
    jobs = [(s, ()) for s in COMMON_SOURCES + [RENDER_SOURCE] + MB_SOURCES]
    if variants:
        jobs += [(RENDER_SOURCE, (f"-D{d}",)) for d in VARIANTS.values()]
    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(lambda j: _compile(j[0], j[1], verbose, extra), jobs))
    obj = dict(zip([(s, d) for s, d in jobs], objs))
    common = [obj[(s, ())] for s in COMMON_SOURCES]
    _link(LIB, common + [obj[(RENDER_SOURCE, ())]], verbose, extra)
    _link(MB_LIB, [obj[(s, ())] for s in MB_SOURCES], verbose, extra)
    if variants:
        for name, d in VARIANTS.items():
            _link(variant_lib(name), common + [obj[(RENDER_SOURCE, (f"-D{d}",))]], verbose, extra)
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


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in r.stderr.splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)


def _compile(source, defines, verbose, extra):
    stem = os.path.splitext(source)[0] + "".join("_" + d[2:].lower() for d in defines)
    out = os.path.join(OBJ_DIR, stem + ".o")
    cmd = [HIPCC, *FLAGS, *extra, *defines, "-I", INCLUDE, "-I", CSRC, "-x", "hip", "-c",
           os.path.join(CSRC, source), "-o", out + ".tmp"]
    _run(cmd, verbose)
    os.replace(out + ".tmp", out)
    return out


def _link(lib, objs, verbose, extra):
    tmp = lib + ".tmp"
    _run([HIPCC, *LINK_FLAGS, *objs, "-o", tmp], verbose)
    os.replace(tmp, lib)


if __name__ == "__main__":
    extra = [a for a in sys.argv[1:] if a not in ("-v", "--no-variants")]
    print(build(verbose=True, extra=extra, variants="--no-variants" not in sys.argv))
