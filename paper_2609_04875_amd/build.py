"""Build libpgsr.so (HIP kernels + C ABI host runtime) for gfx950, in-tree.

Each source is compiled with hipcc to an object under ``_build/`` and the
objects are linked into ``paper_2609_04875_amd/lib/libpgsr.so``.  Packed fp32
instructions are disabled for all device code (-packed-fp32-ops).

``build_all`` also links the checked build, ``lib/libpgsr_checked.so``: the
same sources with PGSR_CHECKED, whose kernels validate every block id they
read from the block table or the free stack and whose pool calls then return
PGSR_ERANGE instead of touching memory outside the pool (a debugging aid for
device metadata written outside the library; same C ABI).
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(ROOT, "_build", "pgsr")
LIBDIR = os.path.join(PKG, "lib")
LIB = os.path.join(LIBDIR, "libpgsr.so")
CHECKED_LIB = os.path.join(LIBDIR, "libpgsr_checked.so")
ARCH = os.environ.get("PGSR_OFFLOAD_ARCH", "gfx950")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wall", "-Wno-unused-function", f"-I{INCLUDE}", f"-I{CSRC}"]


# Per-source options.  The pipelined prefill kernel reads every product's
# result with VALU instructions (softmax, rescale), so its matrix results must
# live in VGPRs: left to its heuristics the compiler
# places them in AGPRs and copies them back on every step.
EXTRA = {"attn_bf16_pipe.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))


def _compile(src: str, verbose: bool, objdir: str = OBJDIR, defines=()) -> str:
    obj = os.path.join(objdir, os.path.basename(src) + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    extra = EXTRA.get(os.path.basename(src), [])
    cmd = [HIPCC, *COMMON, *extra, *[f"-D{d}" for d in defines], *lang, "-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass warns that it does not know -packed-fp32-ops: harmless.
    noise = "not a recognized feature for this target"
    msgs = [ln for ln in (r.stdout + r.stderr).splitlines() if noise not in ln]
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n" + "\n".join(msgs))
    if msgs and verbose:
        print("\n".join(msgs), flush=True)
    return obj


def build(verbose: bool = False, lib: str = LIB, defines=()) -> str:
    """Compile and link; ``defines`` are extra -D options (variants for tuning)."""
    objdir = OBJDIR if lib == LIB else os.path.join(OBJDIR, "variant_" + os.path.basename(lib))
    os.makedirs(objdir, exist_ok=True)
    os.makedirs(os.path.dirname(lib), exist_ok=True)
    srcs = sources()
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, objdir, defines), srcs))
    tmp = lib + ".tmp"
    cmd = [HIPCC, "-shared", f"--offload-arch={ARCH}", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)
    return lib


def build_all(verbose: bool = False) -> tuple:
    """The default library and the checked build."""
    return build(verbose), build(verbose, lib=CHECKED_LIB, defines=("PGSR_CHECKED",))


if __name__ == "__main__":
    print(*build_all(verbose="-v" in sys.argv), sep="\n")
