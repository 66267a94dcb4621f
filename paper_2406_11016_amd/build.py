"""Build the HIP library ``libspec_verify.so`` for gfx950 in-tree with hipcc.

The kernel source is compiled in two passes so that each pass gets only the
flags meant for it: the device pass (``--cuda-device-only``) is built with
packed-fp32 instruction formation disabled, and its fat binary is embedded
into the host pass (``--cuda-host-only``).  Both passes and the host-only
decoding loop build with ``-Wall -Wextra -Werror``.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
CSRC = os.path.join(PKG_DIR, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_NAME = "libspec_verify.so"
LIB_PATH = os.path.join(PKG_DIR, LIB_NAME)
KERNEL_SOURCE = os.path.join(CSRC, "spec_verify.hip")
HOST_SOURCES = [os.path.join(CSRC, "decode_loop.hip")]
SOURCES = [KERNEL_SOURCE, *HOST_SOURCES]
ARCH = "gfx950"

COMMON_FLAGS = ["-O3", "-std=c++17", "-Wall", "-Wextra", "-Werror"]
# device code: no packed-fp32 instructions (the compiler would otherwise form
# them from scalar and float2 code)
DEVICE_FLAGS = [f"--offload-arch={ARCH}", "--cuda-device-only", "-munsafe-fp-atomics",
                "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
HOST_FLAGS = [f"--offload-arch={ARCH}", "--cuda-host-only", "-fPIC"]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; the HIP library cannot be built")
    return path


def _run(cmd, verbose: bool) -> None:
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed with status {res.returncode}")
    if res.stderr.strip():
        # -Werror turns every diagnostic into a failure; anything printed
        # here is a note from a tool, shown as is
        sys.stderr.write(res.stderr)


def build(verbose: bool = False, extra_flags=None) -> str:
    """Compile the library; returns its path.  Always recompiles."""
    inc = ["-I", INCLUDE, "-I", CSRC]
    extra = list(extra_flags or [])
    with tempfile.TemporaryDirectory(prefix="sv_build_") as tmpdir:
        fatbin = os.path.join(tmpdir, "spec_verify.hipfb")
        objs = [os.path.join(tmpdir, "spec_verify.o")]
        _run([hipcc(), *COMMON_FLAGS, *DEVICE_FLAGS, *extra, *inc, "-c", KERNEL_SOURCE, "-o", fatbin], verbose)
        _run([hipcc(), *COMMON_FLAGS, *HOST_FLAGS, *extra, *inc, "-Xclang", "-fcuda-include-gpubinary",
              "-Xclang", fatbin, "-c", KERNEL_SOURCE, "-o", objs[0]], verbose)
        for src in HOST_SOURCES:
            obj = os.path.join(tmpdir, os.path.splitext(os.path.basename(src))[0] + ".o")
            _run([hipcc(), *COMMON_FLAGS, *HOST_FLAGS, *extra, *inc, "-c", src, "-o", obj], verbose)
            objs.append(obj)
        tmp = LIB_PATH + ".tmp"
        _run([hipcc(), "-shared", "-fPIC", *objs, "-o", tmp], verbose)
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
