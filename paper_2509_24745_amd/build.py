"""Build libproxyattn.so (HIP for gfx950) in-tree.

    python -m paper_2509_24745_amd.build             # the library
    python -m paper_2509_24745_amd.build --sanitize  # + its ASan/UBSan host build

Compiles every csrc/*.hip to an object with hipcc and links the shared
library next to this file.  Packed fp32 VALU instructions are disabled for
all device code.

The sanitized build (libproxyattn_san.so) instruments the HOST code only
(argument validation, problem resolution, workspace layout, launch
sequencing) with AddressSanitizer and UndefinedBehaviorSanitizer; device code
is compiled as usual.  It is for the host-only boundary tests, run in a
process that preloads the ASan runtime (see sanitizer_env()).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libproxyattn.so")
LIB_SAN = os.path.join(PKG, "libproxyattn_san.so")
BUILD_SAN = os.path.join(PKG, "_build_san")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-Wno-unused-function", "-Wno-unused-variable",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # no kernel produces or consumes NaN (masked scores are -inf, never NaN):
    # lets max/min skip the sNaN-quieting canonicalisations
    "-fno-honor-nans",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


# host-side instrumentation only: every sanitizer flag goes to the host
# compilation (-Xarch_host), never to device code
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host",
             "-fno-omit-frame-pointer", "-Xarch_host", "-g"]
CLANGXX = os.path.join(os.path.dirname(os.path.realpath(HIPCC)), "..", "llvm", "bin", "clang++")


def _compile(src: str, sanitize: bool = False) -> str:
    obj = os.path.join(BUILD_SAN if sanitize else BUILD, os.path.basename(src)[:-4] + ".o")
    cmd = [HIPCC, *FLAGS, *(SAN_FLAGS if sanitize else []), "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{out}")
    if out.strip():
        print(out, file=sys.stderr)
    return obj


def asan_runtime() -> str:
    """The clang ASan runtime (shared), which a sanitized process preloads."""
    r = subprocess.run([CLANGXX, "-print-file-name=libclang_rt.asan-x86_64.so"],
                       capture_output=True, text=True, check=True)
    return r.stdout.strip()


def sanitizer_env() -> dict:
    """Environment for a Python process that loads libproxyattn_san.so: the
    ASan runtime preloaded, leak checks off (the interpreter is not
    instrumented), every UBSan finding fatal."""
    env = dict(os.environ)
    env["LD_PRELOAD"] = asan_runtime()
    env["ASAN_OPTIONS"] = ("detect_leaks=0:detect_odr_violation=0:alloc_dealloc_mismatch=0:"
                           "verify_asan_link_order=0:abort_on_error=1")
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["PROXYATTN_LIBRARY"] = LIB_SAN
    return env


def build_sanitized(verbose: bool = True) -> str:
    """libproxyattn_san.so: host code under ASan + UBSan (see module doc)."""
    os.makedirs(BUILD_SAN, exist_ok=True)
    srcs = sources()
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, True), srcs))
    tmp = LIB_SAN + ".tmp"
    # link of host objects with the host compiler (the objects carry their
    # device code already); the ASan runtime stays a shared library
    cmd = [CLANGXX, "-shared", "-fPIC", "-shared-libasan", "-fsanitize=address,undefined",
           "-o", tmp, *objs, "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, LIB_SAN)
    if verbose:
        print(f"built {LIB_SAN}")
    return LIB_SAN


def build(verbose: bool = True, sanitize: bool = False) -> str:
    if sanitize:
        build_sanitized(verbose)
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(sanitize="--sanitize" in sys.argv[1:])
