"""Build libfdc.so in-tree with hipcc for gfx950.

Usage: python -m paper_2106_12736_amd.build   (or __graft_entry__.build()).
Always recompiles.  Objects are compiled in parallel and linked into
paper_2106_12736_amd/libfdc.so.
"""

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libfdc.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # packed fp32 instructions stay off (hipcc would otherwise form them from float2 code)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
    "-Wall", "-Wno-unused-function",
]


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp")))


def _compile(src):
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [HIPCC] + COMMON + lang + ["-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose=True):
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "-shared", f"--offload-arch={ARCH}", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    shutil.move(tmp, LIB)
    if verbose:
        print(f"built {LIB}", file=sys.stderr)
    return LIB


# Host sanitizers for the C ABI's host code (api.cpp only: argument validation, plan
# registry, workspace layout).  The device objects are the ones build() made; the
# sanitizer flags reach the host compilation only.
SAN_LIB = os.path.join(BUILD, "libfdc_hostsan.so")
SAN_FLAGS = [
    "-O1", "-g", "-fno-omit-frame-pointer",
    "-Xarch_host", "-fsanitize=address",
    "-Xarch_host", "-fsanitize=undefined",
    "-Xarch_host", "-fsanitize-trap=undefined",  # undefined behaviour traps, no separate runtime
]


def asan_runtime():
    """The compiler's AddressSanitizer runtime, to be preloaded into a process that
    loads SAN_LIB."""
    llvm = os.path.join(os.path.dirname(os.path.realpath(HIPCC)), "..", "llvm")
    out = subprocess.run([os.path.join(llvm, "bin", "clang"), "-print-file-name=libclang_rt.asan-x86_64.so"],
                         capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(out) or not os.path.exists(out):
        raise RuntimeError("AddressSanitizer runtime not found")
    return out


def build_host_sanitized(verbose=True):
    """SAN_LIB: the library with api.cpp compiled under AddressSanitizer and
    UndefinedBehaviorSanitizer (undefined behaviour traps), linked with the device
    objects of build() (made first if missing)."""
    os.makedirs(BUILD, exist_ok=True)
    dev = [s for s in sources() if s.endswith(".hip")]
    objs = [os.path.join(BUILD, os.path.basename(s) + ".o") for s in dev]
    hdrs = [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".h")] + [
        os.path.join(ROOT, "include", f) for f in os.listdir(os.path.join(ROOT, "include"))]
    newest_hdr = max(os.path.getmtime(h) for h in hdrs)

    def stale(src, obj):
        return not os.path.exists(obj) or os.path.getmtime(obj) < max(os.path.getmtime(src), newest_hdr)

    missing = [s for s, o in zip(dev, objs) if stale(s, o)]
    if missing:
        with ThreadPoolExecutor(max_workers=min(8, len(missing))) as ex:
            list(ex.map(_compile, missing))
    api = os.path.join(CSRC, "api.cpp")
    api_obj = os.path.join(BUILD, "api_hostsan.o")
    cmd = [HIPCC] + COMMON + SAN_FLAGS + ["-c", api, "-o", api_obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    rt = asan_runtime()
    cmd = [HIPCC, "-shared", f"--offload-arch={ARCH}", "-fPIC", "-Wl,-z,defs", "-o", SAN_LIB, api_obj] + objs + [
        rt, "-Wl,-rpath," + os.path.dirname(rt)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    if verbose:
        print(f"built {SAN_LIB}", file=sys.stderr)
    return SAN_LIB


if __name__ == "__main__":
    if len(sys.argv) > 1 and sys.argv[1] == "hostsan":
        build_host_sanitized()
    else:
        build()
