"""Builds libssm.so (every HIP source under csrc/) for gfx950 with hipcc.

Usage: python -m paper_2608_23167_amd.build   (or __graft_entry__.build()).
Objects go to _build/ next to this file; the library is written in place
(paper_2608_23167_amd/libssm.so) so that it travels with the source tree.

`--debug` builds libssm_debug.so next to libssm.so (objects in _build_debug/)
with SSM_DEBUG defined: the kernels then check on the device the invariants
the host validation promises (positions, capacities, ids, k) and abort with
the failed condition instead of skipping a write or producing a NaN row.

`--hostsan DIR` builds DIR/libssm_hostsan.so: the same library with its host
code instrumented by AddressSanitizer and UndefinedBehaviorSanitizer (device
code as usual, uninstrumented), for the CPU tests of the C ABI's validation
and closed-form host paths.

`--tuning` builds a separate library (libssm_tuning.so, objects in
_build_tuning/) with SSM_TUNING defined: its GEMM launch choices can be
overridden through the SSM_GEMM_CFG / SSM_GEMM_KROT environment variables
for tile sweeps.  The product library never reads them.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libssm.so")
OBJ = os.path.join(HERE, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 instructions are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result",
]


def _compile(src: str, obj_dir: str, extra) -> str:
    obj = os.path.join(obj_dir, os.path.basename(src) + ".o")
    cmd = [HIPCC, *FLAGS, *extra, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False, tuning: bool = False, debug: bool = False) -> str:
    variant = "_tuning" if tuning else "_debug" if debug else ""
    obj_dir = OBJ + variant
    out = os.path.join(HERE, f"libssm{variant}.so")
    extra = ["-DSSM_TUNING"] if tuning else ["-DSSM_DEBUG"] if debug else []
    os.makedirs(obj_dir, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda src: _compile(src, obj_dir, extra), srcs))
    tmp = out + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)
    if verbose:
        print("built", out)
    return out


# Sanitizer build: each -fsanitize= applies to the host compilation only.
HOSTSAN_FLAGS = [
    "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fno-omit-frame-pointer", "-Wno-unused-result",
    *"-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined".split(),
    *"-Xarch_host -fno-sanitize-recover=undefined".split(),
]


def build_hostsan(out_dir: str) -> str:
    """Builds out_dir/libssm_hostsan.so (see the module docstring)."""
    os.makedirs(out_dir, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))

    def one(src):
        obj = os.path.join(out_dir, os.path.basename(src) + ".o")
        r = subprocess.run([HIPCC, *HOSTSAN_FLAGS, "-c", src, "-o", obj], capture_output=True,
                           text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src}:\n{r.stdout}\n{r.stderr}")
        return obj
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(one, srcs))
    out = os.path.join(out_dir, "libssm_hostsan.so")
    r = subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-shared-libsan",
                        *"-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined".split(),
                        "-o", out, *objs], capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    return out


if __name__ == "__main__":
    if "--hostsan" in sys.argv[1:]:
        print("built", build_hostsan(sys.argv[sys.argv.index("--hostsan") + 1]))
        sys.exit(0)
    build(verbose=True, tuning="--tuning" in sys.argv[1:], debug="--debug" in sys.argv[1:])
    sys.exit(0)
