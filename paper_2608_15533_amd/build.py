"""Build libdeltalog.so in-tree with hipcc for gfx950.

    python -m paper_2608_15533_amd.build        # compiles every source, links the library

Each translation unit is compiled in parallel into ``_build/`` and linked into
``paper_2608_15533_amd/libdeltalog.so``.  Packed fp32 VALU instructions are disabled
for device code (``-packed-fp32-ops``): every float operation is issued as an ordinary
scalar-per-lane VALU op.
"""

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libdeltalog.so")
ARCH = "gfx950"

SOURCES = ["abi.cpp", "dl_gdn.hip", "dl_kda.hip", "dl_rwkv6.hip", "dl_linattn.hip",
           "dl_retnet.hip", "dl_gla.hip", "dl_noalloc.hip"]

# No packed-fp32 instructions; MFMA accumulators in ordinary VGPRs (the merge's MFMA
# contraction accumulates into the state tile's own registers: AGPR accumulators would
# add 64 registers per lane and halve the occupancy).
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-mllvm", "-amdgpu-mfma-vgpr-form=1"]


def hipcc():
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def build_flags_string(extra=()):
    """The compiler flags that shape the kernels (the fixed device flags and any extra
    ones, e.g. -D tuning macros), as the library reports them through dl_build_flags()."""
    return " ".join([*DEVICE_FLAGS, *extra])


def _compile(src, extra):
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    flags_def = '-DDL_BUILD_FLAGS="' + build_flags_string(extra).replace('"', "'") + '"'
    cmd = [hipcc(), "-c", "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
           "-I", INCLUDE, "-I", CSRC, *DEVICE_FLAGS, *extra, flags_def,
           os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose=False, extra_flags=()):
    """Compile all sources and link ``libdeltalog.so``; returns the library path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    jobs = min(len(SOURCES), max(1, min(16, os.cpu_count() or 1)))
    with ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, list(extra_flags)), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


C_EXAMPLE_SRC = os.path.join(ROOT, "tests", "c_abi", "dl_example.c")
C_EXAMPLE_LIB = os.path.join(ROOT, "tests", "c_abi", "libdl_example.so")


def build_c_example(verbose=False):
    """Compile the pure-C ABI example (tests/c_abi/dl_example.c) with the host C compiler
    into a shared library linked against libdeltalog.so (found next to it at run time
    through the rpath).  The GPU tests load it with ctypes."""
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    rpath = os.path.relpath(PKG, os.path.dirname(C_EXAMPLE_LIB))
    cmd = ["gcc", "-std=c11", "-O2", "-fPIC", "-shared", "-Wall", "-Werror",
           "-D__HIP_PLATFORM_AMD__", "-I", INCLUDE, "-I", os.path.join(rocm, "include"),
           C_EXAMPLE_SRC, "-o", C_EXAMPLE_LIB, "-L", PKG, "-ldeltalog",
           "-L", os.path.join(rocm, "lib"), "-lamdhip64", "-lm",
           f"-Wl,-rpath,$ORIGIN/{rpath}", f"-Wl,-rpath,{os.path.join(rocm, 'lib')}"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"C example build failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    if verbose:
        print(f"built {C_EXAMPLE_LIB}")
    return C_EXAMPLE_LIB


if __name__ == "__main__":
    # python -m paper_2608_15533_amd.build [--out DIR] [hipcc flags, e.g. -DDL_MFMA_MERGE=1]
    # With --out the library (and its objects) go to DIR instead of the package: a build
    # variant that DELTALOG_LIB=DIR/libdeltalog.so selects at load time.
    args = sys.argv[1:]
    if args[:1] == ["--out"]:
        out = os.path.abspath(args[1])
        args = args[2:]
        BUILD_DIR = os.path.join(out, "obj")
        LIB = os.path.join(out, "libdeltalog.so")
    build(verbose=True, extra_flags=args)
