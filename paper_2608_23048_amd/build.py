"""Build of the gfx950 HIP library ``libroi.so`` (the C ABI in include/roi.h).

``python -m paper_2608_23048_amd.build`` (or ``__graft_entry__.build()``)
compiles it in-tree with hipcc.  The flags matter for the noise: the keys must
be one exact fp32 value per input, so floating-point contraction is off
(``-ffp-contract=off``) and fast-math is never enabled; fp32 division keeps
HIP's default IEEE (correctly rounded) lowering.  Packed-fp32 instructions are
disabled for the whole library.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_PATH = os.path.join(PKG, "libroi.so")
SOURCES = [os.path.join(CSRC, "roi.hip"), os.path.join(CSRC, "wide_fwd.hip"),
           os.path.join(CSRC, "wide_bwd.hip"),
           os.path.join(CSRC, "export.hip"), os.path.join(CSRC, "cat.hip"),
           os.path.join(CSRC, "stream_copy.hip"), os.path.join(CSRC, "checks.cpp")]
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-ffp-contract=off",
    "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
    "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; the ROCm toolchain is required to build libroi.so")
    return path


def build(verbose: bool = False, extra_flags: list[str] | None = None) -> str:
    """Compile libroi.so for gfx950 (always recompiles; the translation units
    compile in parallel, then link)."""
    import tempfile
    tmp = f"{LIB_PATH}.tmp{os.getpid()}"
    common = [*HIPCC_FLAGS, *(extra_flags or []), f"-I{INCLUDE}", f"-I{CSRC}"]
    with tempfile.TemporaryDirectory() as td:
        objs, procs = [], []
        for src in SOURCES:
            obj = os.path.join(td, os.path.basename(src) + ".o")
            cmd = [hipcc(), *[f for f in common if f != "-shared"], "-c", src, "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            procs.append((subprocess.Popen(cmd), cmd))
            objs.append(obj)
        for p, cmd in procs:
            if p.wait() != 0:
                raise subprocess.CalledProcessError(p.returncode, cmd)
        link = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
        if verbose:
            print(" ".join(link), flush=True)
        subprocess.run(link, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    build(verbose=True, extra_flags=sys.argv[1:])
