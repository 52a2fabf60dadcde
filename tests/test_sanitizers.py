"""CPU sanitizer runs (AddressSanitizer + UndefinedBehaviorSanitizer).

* The C oracle, built with gcc -fsanitize=address,undefined, runs every
  entry point (P-gen in all modes with partial blocks and masked keys, the
  fp64 reading, the V and Q/K quantisers, and the attention recurrence
  causal and non-causal, grouped-query, ragged, with dumps and margins, on
  the MXFP8 path too) in a child process with the sanitizer runtime
  preloaded.
* The HIP library, with its host code built under the same sanitizers
  (device code unchanged; each -fsanitize flag applies to the host pass
  only), runs the argument-validation tests of test_abi.py in a child
  process.  No GPU is used: validation rejects every call before any HIP
  call, and the calls that reach the device check fail cleanly without one.

Any sanitizer report aborts the child, which fails the test.
"""
import hashlib
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN_ENV = {
    "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1:halt_on_error=1",
    "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
}


def _run(script: str, preload: str):
    env = dict(os.environ, LD_PRELOAD=preload, PYTHONPATH=ROOT, **SAN_ENV)
    r = subprocess.run([sys.executable, "-c", script], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=900)
    report = r.stdout[-3000:] + r.stderr[-6000:]
    assert r.returncode == 0, report
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, report
    return r


ORACLE_SCRIPT = r'''
import sys
import numpy as np
import torch
import oracle
from paper_2609_09721_amd import inputs
oracle._lib = oracle.load(sys.argv[1] if len(sys.argv) > 1 else "LIB")
rng = np.random.default_rng(0)
x = -rng.exponential(2.0, size=(37, 75)).astype(np.float32)
x[rng.random(x.shape) < 0.2] = -np.inf
x[3, :32] = -np.inf
for mode in (oracle.EFQ, oracle.LUT_MODE, oracle.EXPQ, oracle.EXPQ6):
    oracle.pgen(x, mode)
oracle.pgen_real(x.astype(np.float64), False)
oracle.pgen_real(x.astype(np.float64), True)
for (Bt, Sq, Sk, Hq, Hkv, D, causal) in [(1, 70, 70, 4, 2, 64, True), (2, 33, 95, 2, 1, 128, False)]:
    w = inputs.Workload("s", Bt, Hq, Hkv, max(Sq, Sk), D, causal, "qwen", 3)
    q, k, v = inputs.make_qkv(w)
    q, k, v = q[:, :Sq].contiguous(), k[:, :Sk].contiguous(), v[:, :Sk].contiguous()
    qb, kb, vb = (oracle.bf16_bits(t) for t in (q, k, v))
    oracle.quant_v(vb)
    oracle.quant_mxfp8(qb)
    for mode in (oracle.EFQ, oracle.LUT_MODE, oracle.EXPQ, oracle.EXPQ6, oracle.EXACT):
        oracle.attn(qb, kb, vb, w.scale, causal, mode, bc=64, dump=True, margins=True)
        oracle.attn(qb, kb, vb, w.scale, causal, mode, bc=32, qk8=True)
print("oracle ok")
'''


def test_oracle_under_address_and_ub_sanitizers(tmp_path):
    import oracle
    lib = str(tmp_path / "liboracle_san.so")
    oracle.compile_c(oracle._SRC, lib, extra=["-g", "-fno-omit-frame-pointer",
                                              "-fsanitize=address,undefined",
                                              "-fno-sanitize-recover=all"])
    rt = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                        text=True).stdout.strip()
    r = _run(ORACLE_SCRIPT.replace('"LIB"', repr(lib)), rt)
    assert "oracle ok" in r.stdout


def _hip_san_build():
    """Full build of the HIP library with host-side sanitizers, cached by the
    hash of the sources it is built from."""
    from paper_2609_09721_amd import build
    srcs = [build.SRC, os.path.join(build.INC, "efq_attn.h")]
    h = hashlib.sha256(b"".join(open(p, "rb").read() for p in srcs)).hexdigest()[:16]
    out_dir = os.path.join(ROOT, "_build", "san")
    os.makedirs(out_dir, exist_ok=True)
    lib = os.path.join(out_dir, f"libefq_attn_{h}.so")
    if not os.path.exists(lib):
        flags = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                 "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-g",
                 "-Xarch_host", "-fno-omit-frame-pointer"]
        cmd = [build.hipcc()] + build.HIPCC_FLAGS + flags + ["-I", build.INC, build.SRC, "-o",
                                                             lib + ".tmp"]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        os.replace(lib + ".tmp", lib)
    return lib


ABI_SCRIPT = r'''
import sys
import pytest
from paper_2609_09721_amd import binding
binding.LIB_PATH = "LIB"
sys.exit(pytest.main(["-q", "-p", "no:cacheprovider", "tests/test_abi.py"]))
'''


@pytest.mark.slow
def test_host_library_validation_under_address_and_ub_sanitizers():
    lib = _hip_san_build()
    rt = subprocess.run(["/opt/rocm/llvm/bin/clang", "-print-file-name=libclang_rt.asan-x86_64.so"],
                        capture_output=True, text=True).stdout.strip()
    if not os.path.exists(rt):
        import glob
        rt = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))[-1]
    r = _run(ABI_SCRIPT.replace('"LIB"', repr(lib)), rt)
    assert " passed" in r.stdout and "failed" not in r.stdout, r.stdout[-2000:]
