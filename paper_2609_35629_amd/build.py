"""Build libsantapp.so for gfx950 with hipcc (in-tree)."""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(ROOT, "_build", "santapp")
LIB = os.path.join(PKG, "libsantapp.so")
PROBE_LIB = os.path.join(PKG, "libsantapp_probe.so")  # streaming-read probe (measurement only)
SOURCES = ["api.hip", "build_kernels.hip", "route_kernels.hip", "decode_kernels.hip", "diag_kernels.hip",
           "kmeans_kernels.hip"]

ARCH = os.environ.get("SANTAPP_ARCH", "gfx950")
CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    # keep the compiler away from packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
]


def hipcc() -> str:
    p = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(p):
        raise RuntimeError("hipcc not found")
    return p


def _compile(src: str) -> str:
    obj = os.path.join(OBJDIR, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), *CFLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
    return obj


def _link(objs, out):
    tmp = out + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, out)


# AddressSanitizer and UndefinedBehaviorSanitizer for host code only (each
# option applies to the host pass; the device code is built as usual)
HOST_SANITIZE = [
    "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
    "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer",
]


def build_host_sanitized(out: str) -> str:
    """``out``: the library with the host code of ``api.hip`` (the entry
    points and their argument checks) built under HOST_SANITIZE, linked with
    the other files' regular objects (built first where missing).  For the
    host sanitizer test, which loads it with the ASan runtime preloaded."""
    os.makedirs(OBJDIR, exist_ok=True)
    others = [s for s in SOURCES if s != "api.hip"]
    objs = []
    for src in others:
        obj = os.path.join(OBJDIR, os.path.splitext(src)[0] + ".o")
        objs.append(obj if os.path.exists(obj) else _compile(src))
    san = os.path.splitext(out)[0] + "_api.o"
    cmd = [hipcc(), *CFLAGS, *HOST_SANITIZE, "-c", os.path.join(CSRC, "api.hip"), "-o", san]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on api.hip (sanitized):\n{r.stderr}")
    _link([san, *objs], out)
    return out


def build(verbose: bool = False) -> str:
    """Compile every kernel file and link ``libsantapp.so`` (and the
    streaming-read probe ``libsantapp_probe.so``) next to this file."""
    os.makedirs(OBJDIR, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(SOURCES) + 1) as ex:
        objs = list(ex.map(_compile, SOURCES + ["probe.hip"]))
    _link(objs[-1:], PROBE_LIB)
    objs = objs[:-1]
    _link(objs, LIB)
    if verbose:
        print(f"built {LIB}", file=sys.stderr)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
