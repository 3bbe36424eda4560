"""Builds libprouter.so (the HIP kernels and the C ABI) for gfx950 with hipcc,
and libprtools.so (the seeded logit generator and the read probe that tests
and benchmarks use; not part of the verifier's interface).

Usage: python -m paper_2608_28726_amd.build   (or build() from Python)

       python -m paper_2608_28726_amd.build --sanitize
           builds _build/sanitize/libprouter.so with the host code (argument
           checks, state objects, launches) instrumented by AddressSanitizer
           and UndefinedBehaviorSanitizer; the device code is unchanged. Load
           it through PR_LIBRARY with the sanitizer runtime preloaded, e.g.
           LD_PRELOAD=$(hipcc's clang runtime dir)/libclang_rt.asan-x86_64.so
           ASAN_OPTIONS=detect_leaks=0 PR_LIBRARY=_build/sanitize/libprouter.so
           python -m pytest tests/test_abi_host.py
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJ_DIR = os.path.join(ROOT, "_build", "obj")
LIB = os.path.join(PKG, "libprouter.so")
TOOLS_LIB = os.path.join(PKG, "libprtools.so")
TOOLS_SOURCES = ["tools/prtools.hip"]

SOURCES = ["row_features.hip", "topp.hip", "aggregate.hip", "head.hip", "calibrate.hip", "api.hip"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    # The row state keeps its exponent reference as a rounded product and
    # rebases with exact residuals: every fused multiply-add is written out,
    # the compiler must not form others.
    "-ffp-contract=off",
    # Keep the compiler from forming packed fp32 instructions.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE,
    "-I", CSRC,
]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


# Host-only sanitizers: each -fsanitize= goes to the host compilation only.
SANITIZE_FLAGS = "-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined -Xarch_host -fno-omit-frame-pointer".split()
SANITIZE_DIR = os.path.join(ROOT, "_build", "sanitize")


def _compile(src: str, obj_dir: str = OBJ_DIR, extra=()) -> str:
    obj = os.path.join(obj_dir, os.path.splitext(src)[0].replace("/", "_") + ".o")
    cmd = [_hipcc(), *HIPCC_FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{res.stderr}")
    return obj


def _link(objs, lib: str, extra=()) -> None:
    tmp = lib + ".tmp"
    cmd = [_hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *extra, *objs, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link of {os.path.basename(lib)} failed:\n{res.stderr}")
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    """Compiles every source and links both shared libraries; returns the
    verifier library's path."""
    os.makedirs(OBJ_DIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(4, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(_compile, SOURCES + TOOLS_SOURCES))
    _link(objs[:len(SOURCES)], LIB)
    _link(objs[len(SOURCES):], TOOLS_LIB)
    if verbose:
        print(f"built {LIB} and {TOOLS_LIB}")
    return LIB


def sanitizer_runtime() -> str:
    """The shared AddressSanitizer runtime of hipcc's clang (it carries the
    UndefinedBehaviorSanitizer handlers too)."""
    res = subprocess.run([_hipcc(), "--print-runtime-dir"], capture_output=True, text=True)
    path = os.path.join(res.stdout.strip(), "libclang_rt.asan-x86_64.so")
    if not os.path.exists(path):
        import glob
        found = glob.glob(os.path.join(os.path.dirname(os.path.dirname(_hipcc())), "lib", "llvm", "lib", "clang", "*",
                                       "lib", "linux", "libclang_rt.asan-x86_64.so"))
        if not found:
            raise RuntimeError("the AddressSanitizer runtime of hipcc's clang was not found")
        path = found[0]
    return path


def build_sanitized(verbose: bool = False) -> str:
    """The verifier library with its host code under AddressSanitizer and
    UndefinedBehaviorSanitizer (see the module docstring); returns its path."""
    obj_dir = os.path.join(SANITIZE_DIR, "obj")
    os.makedirs(obj_dir, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(4, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(lambda f: _compile(f, obj_dir, SANITIZE_FLAGS), SOURCES))
    lib = os.path.join(SANITIZE_DIR, "libprouter.so")
    _link(objs, lib, [sanitizer_runtime()])
    if verbose:
        print(f"built {lib}")
    return lib


if __name__ == "__main__":
    if "--sanitize" in sys.argv[1:]:
        build_sanitized(verbose=True)
    else:
        build(verbose=True)
    sys.exit(0)
