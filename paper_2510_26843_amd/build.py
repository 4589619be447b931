"""Build the gfx950 HIP library in-tree with hipcc.

Three artefacts, all rebuilt on every call:
- libcas.so: the library;
- libcas_debug.so: the same sources with -DCAS_DEBUG (device checks of every
  bound that rests on values the kernels read from device memory);
- cas_runtime_check: csrc/runtime_check.c driving the C ABI, linked with the
  runtime's host code built under AddressSanitizer and
  UndefinedBehaviorSanitizer (host code only; the kernels are the release
  ones).
"""
from __future__ import annotations

import concurrent.futures as _fut
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libcas.so")
LIB_DEBUG = os.path.join(PKG, "libcas_debug.so")
RUNTIME_CHECK = os.path.join(PKG, "cas_runtime_check")
SOURCES = ("kernels.hip", "runtime.hip")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = os.environ.get("CAS_CLANG", "/opt/rocm/llvm/bin/clang")
ROCM_LIB = "/opt/rocm/lib"

FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC",
    "-fhip-fp32-correctly-rounded-divide-sqrt",
    # packed fp32 instructions stay off (plain scalar fp32 code only)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
    "-I" + INCLUDE, "-I" + CSRC,
]
# sanitizers for the host side of a HIP source: each flag applies to the host
# compilation only (device code cannot be built with them)
HOST_SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                 "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all"]
C_SANITIZE = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-fno-sanitize-recover=all"]


def _run(cmd, what: str) -> None:
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"{what} failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    if r.stderr.strip():
        lines = [l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l and l.strip()]
        if lines:
            sys.stderr.write("\n".join(lines) + "\n")


def _compile(src: str, obj: str, extra=()) -> None:
    _run([HIPCC, *FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj], f"hipcc on {src}")


def _link_lib(objs, out: str) -> None:
    tmp = out + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs], "link of " + os.path.basename(out))
    os.replace(tmp, out)


def _build_runtime_check(objdir: str, kernels_obj: str) -> str:
    """csrc/runtime_check.c + runtime.hip (host code sanitized) + the release kernels."""
    rt = os.path.join(objdir, "runtime_hostsan.o")
    drv = os.path.join(objdir, "runtime_check.o")
    _compile("runtime.hip", rt, ["-O1", "-g", *HOST_SANITIZE])
    _run([CLANG, "-std=c11", "-O1", "-g", *C_SANITIZE, "-I" + INCLUDE, "-c", os.path.join(CSRC, "runtime_check.c"),
          "-o", drv], "compile of runtime_check.c")
    tmp = RUNTIME_CHECK + ".tmp"
    _run([CLANG + "++", *C_SANITIZE, "-o", tmp, drv, rt, kernels_obj, "-L" + ROCM_LIB, "-lamdhip64",
          "-Wl,-rpath," + ROCM_LIB], "link of cas_runtime_check")
    os.replace(tmp, RUNTIME_CHECK)
    return RUNTIME_CHECK


def build_runtime_check(verbose: bool = False) -> str:
    """Only the sanitized runtime check (needs the release kernels object of a
    previous build())."""
    objdir = os.path.join(PKG, "_build")
    kobj = os.path.join(objdir, "kernels.o")
    if not os.path.exists(kobj):
        raise RuntimeError(f"{kobj} is missing: run build() first")
    out = _build_runtime_check(objdir, kobj)
    if verbose:
        print("built", out)
    return out


def build(verbose: bool = False) -> str:
    """Compile every HIP source for gfx950 and link libcas.so, libcas_debug.so
    and cas_runtime_check (always rebuilds)."""
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)
    jobs = []
    for src in SOURCES:
        base = src.replace(".hip", "")
        jobs.append((src, os.path.join(objdir, base + ".o"), ()))
        jobs.append((src, os.path.join(objdir, base + "_debug.o"), ("-DCAS_DEBUG",)))
    with _fut.ThreadPoolExecutor(max_workers=len(jobs)) as ex:
        list(ex.map(lambda a: _compile(*a), jobs))
    rel = [os.path.join(objdir, s.replace(".hip", ".o")) for s in SOURCES]
    dbg = [os.path.join(objdir, s.replace(".hip", "_debug.o")) for s in SOURCES]
    _link_lib(rel, LIB)
    _link_lib(dbg, LIB_DEBUG)
    _build_runtime_check(objdir, rel[0])
    if verbose:
        print("built", LIB, LIB_DEBUG, RUNTIME_CHECK)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
