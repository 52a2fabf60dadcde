"""Build the HIP library libefq_attn.so for gfx950 (in-tree)."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "efq_attn.hip")
INC = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libefq_attn.so")
# diagnostic build of the same source with phase stamps (EFQ_PHASE_STAMPS=1);
# only paper_2609_09721_amd.phases loads it
STAMPS_LIB = os.path.join(PKG, "libefq_attn_stamps.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-shared", "-fPIC",
    # decisions are bit-exact fp32 sequences: no contraction, no denormal flush
    "-ffp-contract=off", "-fno-gpu-flush-denormals-to-zero",
    # never emit packed fp32 VALU ops
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False, extra=(), out: str = LIB) -> str:
    tmp = out + f".tmp{os.getpid()}"
    cmd = [hipcc()] + HIPCC_FLAGS + list(extra) + ["-I", INC, SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed building {os.path.basename(out)}")
    # every kernel's host stub must be defined, or dlopen fails later
    nm = subprocess.run(["nm", "-D", "--undefined-only", tmp], capture_output=True, text=True)
    missing = [ln for ln in nm.stdout.splitlines() if "__device_stub__" in ln]
    if missing:
        os.remove(tmp)
        raise RuntimeError("kernel host stubs missing from the build:\n" + "\n".join(missing[:5]))
    os.replace(tmp, out)
    return out


def build_stamps(verbose: bool = False) -> str:
    return build(verbose, extra=("-DEFQ_PHASE_STAMPS=1",), out=STAMPS_LIB)


if __name__ == "__main__":
    build(verbose=True)
