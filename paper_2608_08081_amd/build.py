"""Build libisoquant.so (HIP, gfx950) in-tree with hipcc.

Usage: ``python -m paper_2608_08081_amd.build`` or ``build()`` from Python.
Every call compiles from source; the result is written next to this file.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_NAME = "libisoquant.so"
SOURCES = ["iq_api.cpp", "iq_fit.cpp", "iq_compress.hip", "iq_decode.hip", "iq_decode_g8.hip",
           "iq_decode_multi.hip", "iq_dequant.hip", "iq_decode_f16.hip", "iq_measure.hip",
           "iq_noalloc.hip"]
ARCH = "gfx950"

COMMON_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # no packed-fp32 instructions (v_pk_*_f32) in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
]


def _hipcc() -> str:
    cand = os.environ.get("HIPCC") or shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(cand):
        raise RuntimeError(f"hipcc not found ({cand})")
    return cand


# Host-code sanitizers (AddressSanitizer and UndefinedBehaviorSanitizer on
# the CPU side only: argument validation, planning, codebook construction,
# the seeded parameter generator and the fitters; device code is built as
# usual).  Each -fsanitize goes to the host compilation alone.
HOST_SANITIZE_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host",
                       "-fsanitize=undefined", "-Xarch_host", "-fno-sanitize-recover=undefined",
                       "-Xarch_host", "-fno-omit-frame-pointer", "-g"]


def build(verbose: bool = False, extra_flags: list[str] | None = None,
          host_sanitize: bool = False) -> str:
    """Compile every source for gfx950 and link the shared library.
    Returns the path of the built library.  host_sanitize: a separate build
    with sanitized host code, written to _build/host_sanitize/ (load it with
    the AddressSanitizer runtime preloaded; IQ_LIB_PATH selects it)."""
    hipcc = _hipcc()
    bdir = os.path.join(ROOT, "_build", "host_sanitize") if host_sanitize else \
        os.path.join(ROOT, "_build")
    if host_sanitize:
        extra_flags = list(extra_flags or []) + HOST_SANITIZE_FLAGS
    os.makedirs(bdir, exist_ok=True)
    flags = COMMON_FLAGS + ["-I", INCLUDE, "-I", CSRC] + list(extra_flags or [])

    def compile_one(src: str) -> str:
        obj = os.path.join(bdir, src + ".o")
        cmd = [hipcc, "-x", "hip", *flags, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
        if verbose and r.stderr.strip():
            print(r.stderr, file=sys.stderr)
        return obj

    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    out = os.path.join(bdir, LIB_NAME) if host_sanitize else os.path.join(PKG, LIB_NAME)
    tmp = out + ".tmp"
    link_extra = ["-fsanitize=address,undefined", "-shared-libsan"] if host_sanitize else []
    cmd = [hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs, *link_extra]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, host_sanitize="--host-sanitize" in sys.argv))
