"""Build ``libpulse_stage.so`` (HIP for gfx950) in-tree.

    python -m paper_2606_19163_amd.build

Every source under ``csrc/`` is compiled by hipcc into ``_build/`` and linked
into ``paper_2606_19163_amd/libpulse_stage.so``.  Packed fp32 instructions are
disabled for all device code.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libpulse_stage.so")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")

CFLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-function",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE,
    "-I", CSRC,
]

SOURCES = ["igemm.hip", "igemm2.hip", "norm.hip", "misc.hip", "probe.hip", "attn.hip",
           "tnorm.hip", "stage.cpp", "tstage.cpp", "sched.cpp", "partition.cpp"]

# Attention's softmax takes maxima of MFMA results: with the IEEE mode bit
# off (and no NaN semantics to keep) fmaxf needs no quieting copy of each
# operand, which halves the VALU work of the row maxima.
SOURCE_FLAGS = {"attn.hip": ["-mno-amdgpu-ieee", "-fno-honor-nans"]}


# Host-only sanitizer build of the orchestration code (CPU tests only): each
# -fsanitize applies to the host pass alone; the kernels are not built with it.
ASAN_BUILD = os.path.join(ROOT, "_build_asan")
ASAN_LIB = os.path.join(ASAN_BUILD, "libpulse_stage_asan.so")
HOST_SOURCES = ["stage.cpp", "tstage.cpp", "sched.cpp", "partition.cpp"]
ASAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
              "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all",
              "-g"]


def _compile(src: str, out_dir: str = BUILD, extra=()) -> str:
    obj = os.path.join(out_dir, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *CFLAGS, *SOURCE_FLAGS.get(src, []), *extra, "-c", os.path.join(CSRC, src),
           "-o", obj]
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


def asan_runtime() -> str:
    """The compiler's shared AddressSanitizer runtime (preloaded into the
    Python process that loads the sanitizer build)."""
    import glob
    llvm = os.path.join(os.path.dirname(os.path.realpath(HIPCC)), "..", "llvm")
    hits = sorted(glob.glob(os.path.join(llvm, "lib", "clang", "*", "lib", "linux",
                                         "libclang_rt.asan-x86_64.so")))
    hits += sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not hits:
        raise RuntimeError("no libclang_rt.asan-x86_64.so next to hipcc")
    return hits[0]


def build_asan(verbose: bool = False) -> str:
    """libpulse_stage_asan.so: the host sources with AddressSanitizer and
    UndefinedBehaviorSanitizer, linked with the regular kernel objects (built
    first when missing).  For CPU tests of the host logic (dry runs,
    schedule, partitioner); it is never loaded on a GPU."""
    os.makedirs(ASAN_BUILD, exist_ok=True)
    kern = [s for s in SOURCES if s not in HOST_SOURCES]
    kobjs = [os.path.join(BUILD, os.path.splitext(s)[0] + ".o") for s in kern]
    if not all(os.path.exists(o) for o in kobjs):
        build()
    with ThreadPoolExecutor(max_workers=len(HOST_SOURCES)) as ex:
        hobjs = list(ex.map(lambda s: _compile(s, ASAN_BUILD, ASAN_FLAGS), HOST_SOURCES))
    tmp = ASAN_LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *hobjs, *kobjs, "-Xarch_host",
           "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-shared-libsan", "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, ASAN_LIB)
    if verbose:
        print(f"built {ASAN_LIB}")
    return ASAN_LIB


if __name__ == "__main__":
    if "--asan" in sys.argv:
        build_asan(verbose=True)
    else:
        build(verbose=True)
    sys.exit(0)
