"""Build libmocap_attn.so for gfx950 (in-tree, next to this file).

Every HIP source is compiled with hipcc for gfx950 only, with packed-fp32
instructions disabled in device code, then linked into one shared library.
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
LIB = os.path.join(PKG, "libmocap_attn.so")
SOURCES = ["api.cpp", "plan.cpp", "chunk_attn.hip", "kv_append.hip", "lse_merge.hip"]
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA results in VGPRs: the score accumulators feed the softmax VALU work
    # directly, with no copies out of accumulation registers.
    "-mllvm", "-amdgpu-mfma-vgpr-form=true",
    "-Wno-unused-command-line-argument",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


def _compile(src: str, verbose: bool, build_dir: str, extra_flags) -> str:
    obj = os.path.join(build_dir, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, *extra_flags, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed on {src}")
    return obj


def build(verbose: bool = False, extra_flags=(), lib_path: str = LIB, build_dir: str = BUILD_DIR) -> str:
    """Compile every source and link ``lib_path``.  ``extra_flags`` (e.g. -D
    tuning macros) and an alternative output location serve experiments."""
    os.makedirs(build_dir, exist_ok=True)
    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, build_dir, tuple(extra_flags)), SOURCES))
    tmp = lib_path + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    _check_stubs(tmp)
    os.replace(tmp, lib_path)
    return lib_path


def _check_stubs(lib: str) -> None:
    """Fail if a kernel's host launch stub was not emitted.

    If a kernel body does not compile for the host pass, clang can drop the
    template's stub without an error, leaving an undefined symbol that only
    shows up when the library is loaded."""
    out = subprocess.run(["nm", "-C", lib], check=True, capture_output=True, text=True).stdout
    missing = [ln.strip() for ln in out.splitlines() if " U " in ln and "__device_stub__" in ln]
    if missing:
        raise RuntimeError("kernel launch stubs missing from " + lib + ":\n" + "\n".join(missing))


DEBUG_LIB = os.path.join(PKG, "libmocap_attn_debug.so")


def build_debug(verbose: bool = False) -> str:
    """The library with host-side block-table checks before every launch
    (-DMOCAP_DEBUG_TABLES): libmocap_attn_debug.so, for debugging callers."""
    return build(verbose, extra_flags=("-DMOCAP_DEBUG_TABLES",), lib_path=DEBUG_LIB,
                 build_dir=os.path.join(BUILD_DIR, "debug"))


if __name__ == "__main__":
    if "--debug-tables" in sys.argv:
        print(build_debug(verbose="-v" in sys.argv))
    else:
        print(build(verbose="-v" in sys.argv))
