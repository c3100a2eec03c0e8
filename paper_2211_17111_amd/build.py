"""Build libbevpool.so (HIP kernels + C ABI) for gfx950 with hipcc.

Every call compiles from source; objects go to ``_build/`` next to the
package and the shared library lands in the package directory, where the
Python binding loads it.
"""

from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB_NAME = "libbevpool.so"
LIB_PATH = os.path.join(PKG, LIB_NAME)

ARCH = "gfx950"
SOURCES = ["prepare.hip", "prepare_plan.hip", "schedule_local.hip", "forward.hip", "forward_strips.hip", "backward.hip", "softmax.hip",
           "geometry.hip",
           "api.cpp"]
# measurement probe for bench.py, built into a library of its own
PROBE_SOURCE = "stream_probe.hip"
PROBE_LIB = os.path.join(PKG, "libbevpool_probe.so")

# No fast-math and no flush-to-zero on the GPU path; packed fp32 ops off.
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wall", "-Wno-unused-function",
          f"-I{INCLUDE}", f"-I{CSRC}"]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = os.path.join(rocm, "bin", "hipcc")
    return path if os.path.exists(path) else "hipcc"


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in res.stdout.splitlines()
                    if "packed-fp32-ops" not in l and "is not a recognized feature" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"command failed ({res.returncode}): {' '.join(cmd)}\n{res.stdout}")
    if verbose and out.strip():
        print(out, flush=True)


def remove_stale_objects() -> list[str]:
    """Delete objects in the build folder that no source in SOURCES produces
    (left by renamed or deleted sources), so the folder holds only what the
    library links."""
    keep = {os.path.splitext(src)[0] + ".o" for src in SOURCES + [PROBE_SOURCE]}
    removed = []
    if os.path.isdir(BUILD):
        for name in sorted(os.listdir(BUILD)):
            if name.endswith(".o") and name not in keep:
                os.remove(os.path.join(BUILD, name))
                removed.append(name)
    return removed


def check_defined(lib: str) -> None:
    """Fail when the library leaves one of its own symbols undefined (a
    kernel whose launch stub the host pass did not emit links silently into
    a shared library and only fails when the library is loaded)."""
    res = subprocess.run(["nm", "-D", "--undefined-only", lib], stdout=subprocess.PIPE,
                         stderr=subprocess.STDOUT, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"nm failed on {lib}: {res.stdout}")
    own = [l.split()[-1] for l in res.stdout.splitlines() if "bevpool" in l]
    if own:
        raise RuntimeError(f"{lib} leaves {len(own)} of its own symbols undefined, e.g. {own[0]}")


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    for name in remove_stale_objects():
        if verbose:
            print(f"removed stale {name}", flush=True)
    cc = hipcc()

    def compile_one(src):
        obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        _run([cc, *COMMON, *lang, "-c", os.path.join(CSRC, src), "-o", obj], verbose)
        return obj

    with ThreadPoolExecutor(max_workers=min(4, len(SOURCES))) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = LIB_PATH + ".tmp"
    _run([cc, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp], verbose)
    check_defined(tmp)
    os.replace(tmp, LIB_PATH)
    # the measurement probe, a library of its own (bench.py loads it)
    pobj = os.path.join(BUILD, "stream_probe.o")
    _run([cc, *COMMON, "-x", "hip", "-c", os.path.join(CSRC, PROBE_SOURCE), "-o", pobj], verbose)
    _run([cc, "-shared", "-fPIC", f"--offload-arch={ARCH}", pobj, "-o", PROBE_LIB + ".tmp"], verbose)
    os.replace(PROBE_LIB + ".tmp", PROBE_LIB)
    return LIB_PATH


SAN_DIR = os.path.join(BUILD, "asan")
SAN_LIB = os.path.join(SAN_DIR, "libbevpool_asan.so")
# AddressSanitizer and UndefinedBehaviorSanitizer on the host code only (the
# device code is compiled as usual)
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-fno-omit-frame-pointer", "-g"]


def sanitizer_runtime() -> str:
    """The compiler's AddressSanitizer runtime, preloaded into a process that
    loads the sanitized library."""
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    res = subprocess.run([os.path.join(rocm, "llvm", "bin", "clang"),
                          "-print-file-name=libclang_rt.asan-x86_64.so"],
                         stdout=subprocess.PIPE, text=True)
    path = res.stdout.strip()
    if not os.path.isabs(path):  # (newer layouts name it per target)
        res = subprocess.run([os.path.join(rocm, "llvm", "bin", "clang"), "-print-runtime-dir"],
                             stdout=subprocess.PIPE, text=True)
        path = os.path.join(res.stdout.strip(), "libclang_rt.asan.so")
    return path


def build_sanitized(verbose: bool = False) -> str:
    """The same library with host-side ASan/UBSan instrumentation, for the
    ABI tests' argument-validation paths (no GPU needed).  Rebuilt only when
    a source or header is newer than it."""
    os.makedirs(SAN_DIR, exist_ok=True)
    inputs = [os.path.join(CSRC, f) for f in os.listdir(CSRC)] + [os.path.join(INCLUDE, "bevpool.h")]
    if os.path.exists(SAN_LIB) and os.path.getmtime(SAN_LIB) >= max(map(os.path.getmtime, inputs)):
        return SAN_LIB
    cc = hipcc()
    flags = [f if f != "-O3" else "-O1" for f in COMMON] + SAN_FLAGS

    def compile_one(src):
        obj = os.path.join(SAN_DIR, os.path.splitext(src)[0] + ".o")
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        _run([cc, *flags, *lang, "-c", os.path.join(CSRC, src), "-o", obj], verbose)
        return obj

    with ThreadPoolExecutor(max_workers=min(4, len(SOURCES))) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = SAN_LIB + ".tmp"
    _run([cc, "-shared", "-fPIC", f"--offload-arch={ARCH}", *SAN_FLAGS, *objs, "-o", tmp], verbose)
    os.replace(tmp, SAN_LIB)
    return SAN_LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
