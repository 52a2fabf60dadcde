"""Independent numpy rendering of the P-gen and V-quant rules (oracle twin).

Test infrastructure only.  It computes the same fp32 decision contract as
``efq_oracle.c`` but is written differently (vectorised, thresholds instead
of a nearest search, exponent bits instead of frexp), so that a slip in one
of the two shows up as a disagreement.  numpy float32 arithmetic is IEEE
round-to-nearest-even per operation; the one fused multiply-add is emulated
exactly (exact fp64 product, TwoSum for the addition, directed fix-up of
fp32 ties).
"""
from __future__ import annotations

import numpy as np

F32 = np.float32
LN2 = F32(np.log(2.0))
INVLN2 = F32(1.0 / np.log(2.0))
LOG2_9 = F32(np.log(2.0 / 9.0))
LN6 = F32(np.log(6.0))
C16 = np.array([0, 1, 1, 1, 1, 1, 2, 2, 3, 3, 4, 5, 5, 6, 7, 7], np.int64)  # Sec. II-D


def fma32(a, b, c):
    """Correctly rounded fp32 fma(a, b, c) for fp32 arrays."""
    a = np.asarray(a, F32).astype(np.float64)
    b = np.asarray(b, F32).astype(np.float64)
    c = np.asarray(c, F32).astype(np.float64)
    p = a * b                      # exact: 24 + 24 significant bits
    s = p + c
    bb = s - p
    err = (p - (s - bb)) + (c - bb)  # TwoSum: s + err == p + c exactly
    r = s.astype(F32)              # nearest fp32 of s (ties to even)
    # s is a tie between two fp32 neighbours only if it is representable in
    # fp64 exactly halfway; then the sign of err decides the direction.
    lo = np.nextafter(r, F32(-np.inf))
    hi = np.nextafter(r, F32(np.inf))
    with np.errstate(invalid="ignore", over="ignore"):
        mid_lo = (r.astype(np.float64) + lo.astype(np.float64)) / 2
        mid_hi = (r.astype(np.float64) + hi.astype(np.float64)) / 2
    fix_down = (s == mid_lo) & (err < 0)   # rounded up to r, truth below the tie
    fix_up = (s == mid_hi) & (err > 0)
    r = np.where(fix_down, lo, r)
    r = np.where(fix_up, hi, r)
    return r


def pgen_fp32(x: np.ndarray, tau: float, h: float, lut: bool = False,
              scale: float = 1.0, m: float = 0.0):
    """Alg. 1 on rows of scores given as raw dot products x (fp32, -inf = masked).

    x_t = fl(fl(x*scale) - m).  Returns (codes int64 [rows, cols], k int64 [rows, nblk])."""
    x = np.asarray(x, F32)
    if x.ndim == 1:
        x = x[None, :]
    rows, cols = x.shape
    nblk = (cols + 31) // 32
    pad = nblk * 32 - cols
    xp = np.concatenate([x, np.full((rows, pad), -np.inf, F32)], axis=1).reshape(rows, nblk, 32)
    scale, m, tau, h = F32(scale), F32(m), F32(tau), F32(h)
    masked = np.isneginf(xp)
    with np.errstate(invalid="ignore"):
        xs = (xp * scale) - m
    xs = np.where(masked, F32(-np.inf), xs)
    Mb = xs.max(axis=2)                           # block maximum
    fin = np.isfinite(Mb)
    q = (np.where(fin, Mb, F32(0)) + LOG2_9) * INVLN2
    k = np.floor(q.astype(np.float64))
    k = np.clip(k, -127, 127).astype(np.int64)
    k = np.where(fin, k, -127)
    off = (k.astype(F32) * LN2) + (LN6 + tau)
    bias = -((m + off) * h)
    acc = np.where(masked, F32(0), xp)
    if lut:
        # w ~ 16 (u + 1) - 1/2, nearest-even, saturate, multiple of 16:
        # clip(floor(u) + 1, 0, 15)
        bias16 = fma32(bias, F32(16.0), F32(15.5))
        w = fma32(acc, F32(16.0) * F32(scale * h), bias16[:, :, None])
        r = np.rint(w.astype(np.float64))
        j = (np.clip(r, 0, 255) // 16).astype(np.int64)
        c = C16[j]
    else:
        # w ~ 32 (u + 1) - 1/2; nearest-even to an integer, saturate to
        # [0, 255], keep the multiple of 32: clip(floor(u) + 1, 0, 7)
        bias32 = fma32(bias, F32(32.0), F32(31.5))
        w = fma32(acc, F32(32.0) * F32(scale * h), bias32[:, :, None])
        r = np.rint(w.astype(np.float64))
        c = (np.clip(r, 0, 255) // 32).astype(np.int64)
    c = np.where(masked, 0, c)
    return c.reshape(rows, nblk * 32)[:, :cols], k


# E2M1 magnitudes and the round-to-nearest-even decision points between
# consecutive codes: y < 0.25 -> 0, y == 0.25 -> 0 (even), (0.25, 0.75) -> 1,
# 0.75 -> 2 (even), ..., [5, inf) -> ties/saturation handled below.
_MID = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0])


def e2m1_rne(y: np.ndarray) -> np.ndarray:
    """Round y >= 0 to the E2M1 code with nearest value (ties to even code),
    saturating at code 7 (value 6)."""
    y = np.asarray(y, np.float64)
    c = np.searchsorted(_MID, y, side="left")   # number of midpoints < y
    at_mid = np.isin(y, _MID)
    # at a midpoint between codes j and j+1 choose the even one
    j = np.searchsorted(_MID, y, side="left")
    c = np.where(at_mid, np.where(j % 2 == 0, j, j + 1), c)
    return np.minimum(c, 7).astype(np.int64)


def quant_v_bits(v_bits: np.ndarray):
    """MXFP4 along keys for V [B, S, H, D] bf16 bits.  Returns codes
    [B, H, nblk*32, D] (bit 3 = sign) and e8m0 [B, H, nblk, D]."""
    v_bits = np.asarray(v_bits, np.uint16)
    B, S, H, D = v_bits.shape
    nblk = (S + 31) // 32
    pad = nblk * 32 - S
    vb = np.concatenate([v_bits, np.zeros((B, pad, H, D), np.uint16)], axis=1)
    vb = vb.transpose(0, 2, 1, 3).reshape(B, H, nblk, 32, D)
    mag_bits = (vb & 0x7FFF).astype(np.uint32)
    mag = (mag_bits << 16).view(np.float32).astype(np.float64)
    amax = mag.max(axis=3)                        # [B, H, nblk, D]
    # floor(log2 amax) from the bf16 exponent field (subnormals: leading bit)
    amax_bits = mag_bits.max(axis=3)
    expf = (amax_bits >> 7).astype(np.int64)
    mant = (amax_bits & 0x7F).astype(np.int64)
    lead = np.where(mant > 0, np.floor(np.log2(np.maximum(mant, 1))).astype(np.int64), 0)
    fl2 = np.where(expf > 0, expf - 127, -133 + lead)
    k = np.where(amax > 0, np.clip(fl2 - 2, -127, 127), -127)
    y = mag * np.exp2(-k.astype(np.float64))[:, :, :, None, :]
    c = e2m1_rne(y)
    c = c | np.where((vb & 0x8000) != 0, 8, 0)
    return (c.reshape(B, H, nblk * 32, D).astype(np.uint8),
            (k + 127).astype(np.uint8))
