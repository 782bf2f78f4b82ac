"""Build the host-bookkeeping test library: the real host layer (csrc/api.hip)
linked with the recording launch layer (fake_launch.hip) instead of the
kernels.  `sanitize=True` builds the host code with AddressSanitizer and
UndefinedBehaviorSanitizer (host only; no GPU code is instrumented)."""
from __future__ import annotations

import hashlib
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_2607_00760_amd", "csrc")
OUT = os.path.join(HERE, "_build")
SOURCES = [os.path.join(CSRC, "api.hip"), os.path.join(HERE, "fake_launch.hip")]
HEADERS = [os.path.join(CSRC, "mosaic_internal.h"), os.path.join(ROOT, "include", "mosaic.h")]
BASE = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", "-ffp-contract=off", "-w",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


def asan_runtime() -> str:
    """The clang AddressSanitizer runtime that a sanitized library needs preloaded."""
    import glob
    c = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not c:
        raise FileNotFoundError("libclang_rt.asan-x86_64.so not found under /opt/rocm/llvm")
    return c[-1]


def build(sanitize: bool = False) -> str:
    """Compile (when the sources changed) and return the library path."""
    h = hashlib.sha256()
    for f in SOURCES + HEADERS:
        h.update(open(f, "rb").read())
    h.update(b"san" if sanitize else b"plain")
    tag = h.hexdigest()[:12]
    lib = os.path.join(OUT, f"libmosaic_hostsim{'_san' if sanitize else ''}_{tag}.so")
    if os.path.exists(lib):
        return lib
    os.makedirs(OUT, exist_ok=True)
    cmd = ["/opt/rocm/bin/hipcc", *BASE, *(SAN if sanitize else []), "-shared", *SOURCES, "-o", lib + ".tmp"]
    if sanitize:
        cmd.insert(-2, "-shared-libsan")
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    os.replace(lib + ".tmp", lib)
    return lib
