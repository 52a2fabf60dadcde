"""EFQ-Softmax CPU oracle -- test infrastructure only.

Plain, slow implementations of what the GPU path computes, written from the
paper (Alg. 1 inside Alg. 2, Secs. II-III).  The C file ``efq_oracle.c``
holds the attention recurrence, P-gen and V quantiser; ``twin.py`` holds an
independent numpy rendering of the P-gen and V-quant rules and of the
Alg. 2 recurrence used to cross-check it.  Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU
baseline of ``bench.py`` may import this package.  Nothing here imports the
HIP package, and the HIP package never imports this.

Parity pins that constrain these functions live in ``tests/test_oracle_*.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "efq_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

# Operating points (tau, h) of Sec. IV-A "Parameter selection".
MEAN = (-3.06, 2.30)
MMLU = (-2.90, 2.00)
BALANCE = (-2.10, 2.70)
# EFQ-Softmax-LUT constants of Sec. II-D: tau16 = log(1/24), h16 = 14/log 24.
LUT = (float(np.log(1.0 / 24.0)), float(14.0 / np.log(24.0)))

EFQ, EXPQ, EXACT, LUT_MODE, EXPQ6 = 0, 1, 2, 3, 4

C8 = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])  # Sec. II-B
C16 = np.array([0, 1, 1, 1, 1, 1, 2, 2, 3, 3, 4, 5, 5, 6, 7, 7])  # Sec. II-D


GCC_FLAGS = ["-O2", "-std=gnu99", "-Wall", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
             "-shared", "-fPIC"]


def compile_c(src: str, out: str, extra=()) -> str:
    """gcc build of an oracle source file (no fast-math, no FMA contraction)."""
    tmp = out + f".tmp{os.getpid()}"
    subprocess.run(["gcc"] + GCC_FLAGS + list(extra) + [src, "-o", tmp, "-lm"], check=True)
    os.replace(tmp, out)
    return out


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no fast-math, no FMA contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        compile_c(_SRC, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        _lib = load(_LIB)
    return _lib


def load(path: str):
    """ctypes handle of an oracle build with the argument types set."""
    L = ctypes.CDLL(path)
    P = ctypes.c_void_p
    L.orc_pgen.argtypes = [P, ctypes.c_long, ctypes.c_int, ctypes.c_int, ctypes.c_float,
                           ctypes.c_float, P, P]
    L.orc_pgen_real.argtypes = [P, ctypes.c_long, ctypes.c_int, ctypes.c_int,
                                ctypes.c_double, ctypes.c_double, P, P, P]
    L.orc_quant_v.argtypes = [P, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, P, P]
    L.orc_attn.argtypes = [P, P, P] + [ctypes.c_int] * 6 + [
        ctypes.c_float, ctypes.c_int, ctypes.c_int, ctypes.c_float, ctypes.c_float,
        ctypes.c_int, P, ctypes.c_long, P, P, P, P, P, P, ctypes.c_int, ctypes.c_int]
    L.orc_quant_mxfp8.argtypes = [P, ctypes.c_long, ctypes.c_int, P, P]
    for f in (L.orc_pgen, L.orc_pgen_real, L.orc_quant_v, L.orc_attn, L.orc_quant_mxfp8):
        f.restype = ctypes.c_int
    return L


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _params(mode: int, tau: Optional[float], h: Optional[float]):
    if tau is None or h is None:
        tau, h = LUT if mode == LUT_MODE else MEAN
    return float(tau), float(h)


def pgen(x: np.ndarray, mode: int = EFQ, tau: float = None, h: float = None):
    """P-gen unit on shifted scores x (rows x cols fp32, -inf = masked).

    Returns (codes uint8 [rows, cols], e8m0 uint8 [rows, ceil(cols/32)])."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.ndim == 1:
        x = x[None, :]
    rows, cols = x.shape
    tau, h = _params(mode, tau, h)
    codes = np.zeros((rows, cols), np.uint8)
    e8 = np.zeros((rows, (cols + 31) // 32), np.uint8)
    rc = lib().orc_pgen(_ptr(x), rows, cols, mode, tau, h, _ptr(codes), _ptr(e8))
    assert rc == 0
    return codes, e8


def pgen_real(x: np.ndarray, lut: bool = False, tau: float = None, h: float = None):
    """Alg. 1 evaluated step by step in fp64 (the real-valued reading).

    Returns (codes, k_b int16, u = (z - tau) h in fp64)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    if x.ndim == 1:
        x = x[None, :]
    rows, cols = x.shape
    if tau is None or h is None:
        tau, h = LUT if lut else MEAN
    codes = np.zeros((rows, cols), np.uint8)
    k = np.zeros((rows, (cols + 31) // 32), np.int16)
    u = np.zeros((rows, cols), np.float64)
    rc = lib().orc_pgen_real(_ptr(x), rows, cols, int(lut), float(tau), float(h), _ptr(codes),
                             _ptr(k), _ptr(u))
    assert rc == 0
    return codes, k, u


def quant_v(v_bits: np.ndarray):
    """V [B, S, H, D] (bf16 bit patterns, uint16) -> MXFP4 along the key axis.

    Returns (codes uint8 [B, H, nblk*32, D] with bit 3 = sign,
             e8m0 uint8 [B, H, nblk, D])."""
    v_bits = np.ascontiguousarray(v_bits, dtype=np.uint16)
    B, S, H, D = v_bits.shape
    nblk = (S + 31) // 32
    codes = np.zeros((B, H, nblk * 32, D), np.uint8)
    e8 = np.zeros((B, H, nblk, D), np.uint8)
    rc = lib().orc_quant_v(_ptr(v_bits), B, S, H, D, _ptr(codes), _ptr(e8))
    assert rc == 0
    return codes, e8


def all_rows(B: int, Hq: int, Sq: int) -> np.ndarray:
    b, h, i = np.meshgrid(np.arange(B), np.arange(Hq), np.arange(Sq), indexing="ij")
    return np.stack([b.ravel(), h.ravel(), i.ravel()], axis=1).astype(np.int32)


def attn(q_bits, k_bits, v_bits, scale: float, causal: bool, mode: int = EFQ,
         tau: float = None, h: float = None, bc: int = 64, rows: np.ndarray = None,
         dump: bool = False, nthreads: int = 0, margins: bool = False, qk8: bool = False):
    """Attention forward for the listed query rows (Alg. 2 over tiles of bc keys).

    q_bits [B, Sq, Hq, D], k_bits/v_bits [B, Sk, Hkv, D]: bf16 bit patterns.
    rows: int32 [n, 3] of (b, hq, i); None = every row, ordered (b, hq, i).
    Returns out [n, D] fp32, plus (codes [n, nblk*32], e8m0 [n, nblk],
    m [n] fp32, l [n] fp64) when dump is set, plus the per-row smallest
    decision margin [n] fp64 (in dot-product units) when margins is set.
    qk8: Q K^T on the MXFP8 values of Q and K (low-bit Q K^T)."""
    q_bits = np.ascontiguousarray(q_bits, dtype=np.uint16)
    k_bits = np.ascontiguousarray(k_bits, dtype=np.uint16)
    v_bits = np.ascontiguousarray(v_bits, dtype=np.uint16)
    B, Sq, Hq, D = q_bits.shape
    _, Sk, Hkv, _ = k_bits.shape
    if rows is None:
        rows = all_rows(B, Hq, Sq)
    rows = np.ascontiguousarray(rows, dtype=np.int32)
    n = rows.shape[0]
    tau, h = _params(mode, tau, h)
    nblk = (Sk + 31) // 32
    out = np.zeros((n, D), np.float32)
    codes = e8 = mm = ll = None
    if dump:
        codes = np.zeros((n, nblk * 32), np.uint8)
        e8 = np.zeros((n, nblk), np.uint8)
        mm = np.zeros((n,), np.float32)
        ll = np.zeros((n,), np.float64)
    mg = np.full((n,), np.inf, np.float64) if margins else None
    rc = lib().orc_attn(_ptr(q_bits), _ptr(k_bits), _ptr(v_bits), B, Sq, Sk, Hq, Hkv, D,
                        float(scale), int(causal), int(mode), tau, h, int(bc), _ptr(rows), n,
                        _ptr(out), _ptr(codes), _ptr(e8), _ptr(mm), _ptr(ll), _ptr(mg),
                        int(bool(qk8)), int(nthreads))
    if rc != 0:
        raise ValueError(f"orc_attn failed with {rc}")
    res = (out,)
    if dump:
        res += (codes, e8, mm, ll)
    if margins:
        res += (mg,)
    return res if len(res) > 1 else out




def quant_mxfp8(x_bits: np.ndarray):
    """MXFP8 (E4M3) along the last axis (a multiple of 32) of bf16 bits x:
    returns (codes uint8 [..., D], e8m0 uint8 [..., D/32])."""
    x_bits = np.ascontiguousarray(x_bits, dtype=np.uint16)
    D = x_bits.shape[-1]
    rows = x_bits.size // D
    codes = np.zeros(x_bits.shape, np.uint8)
    e8 = np.zeros(x_bits.shape[:-1] + (D // 32,), np.uint8)
    rc = lib().orc_quant_mxfp8(_ptr(x_bits), rows, D, _ptr(codes), _ptr(e8))
    if rc != 0:
        raise ValueError(f"orc_quant_mxfp8 failed with {rc}")
    return codes, e8


def e4m3_values(codes: np.ndarray, e8m0: np.ndarray) -> np.ndarray:
    """fp64 values of MXFP8 codes with their per-32 E8M0 scales."""
    c = codes.astype(np.int64)
    e = (c >> 3) & 15
    m = c & 7
    mag = np.where(e == 0, m * 2.0 ** -9, (1 + m / 8.0) * 2.0 ** (e - 7.0))
    k = np.repeat(e8m0.astype(np.int64) - 127, 32, axis=-1)
    return np.where(c & 0x80, -1.0, 1.0) * mag * 2.0 ** k

def calibrate(q_bits, k_bits, v_bits, scale: float, causal: bool, o_ref: np.ndarray, taus, hs,
              bc: int = 64, nthreads: int = 0):
    """Algorithm 3 (offline selection of (tau, h), Sec. III-C): for every
    candidate pair, tau outer and h inner, run EFQ attention on all rows and
    compute rho = ||O~ - O_ref||_F / ||O_ref||_F in fp64; keep the first pair
    with a strictly smaller rho.  o_ref: [B*Hq*Sq, D] in all_rows order.
    Candidates are used as fp32 values.  Returns ((tau*, h*), rho [nt, nh])."""
    taus = [np.float32(t) for t in taus]
    hs = [np.float32(x) for x in hs]
    ref = np.asarray(o_ref, np.float64)
    ref_norm = np.sqrt(np.sum(ref * ref))
    rho = np.zeros((len(taus), len(hs)))
    best, best_rho = None, np.inf
    for i, tau in enumerate(taus):
        for j, h in enumerate(hs):
            o = attn(q_bits, k_bits, v_bits, scale, causal, EFQ, tau=float(tau), h=float(h), bc=bc,
                     nthreads=nthreads).astype(np.float64)
            d = o - ref
            r = np.sqrt(np.sum(d * d)) / ref_norm
            rho[i, j] = r
            if r < best_rho:
                best_rho, best = r, (float(tau), float(h))
    return best, rho

def bf16_bits(t) -> np.ndarray:
    """Bit patterns of a bf16 torch tensor as a uint16 numpy array (a view of
    the same values; no arithmetic)."""
    import torch
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def bits_to_f64(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
