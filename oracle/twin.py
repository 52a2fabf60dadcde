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
              scale: float = 1.0, m=0.0):
    """Alg. 1 on rows of scores given as raw dot products x (fp32, -inf = masked).

    x_t = fl(fl(x*scale) - m), with m a scalar or one running maximum per row.
    Returns (codes int64 [rows, cols], k int64 [rows, nblk])."""
    x = np.asarray(x, F32)
    if x.ndim == 1:
        x = x[None, :]
    rows, cols = x.shape
    nblk = (cols + 31) // 32
    pad = nblk * 32 - cols
    xp = np.concatenate([x, np.full((rows, pad), -np.inf, F32)], axis=1).reshape(rows, nblk, 32)
    m = np.broadcast_to(np.asarray(m, F32).reshape(-1), (rows,)).reshape(rows, 1)
    scale, tau, h = F32(scale), F32(tau), F32(h)
    masked = np.isneginf(xp)
    with np.errstate(invalid="ignore"):
        xs = (xp * scale) - m[:, :, None]
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


C8 = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])   # Sec. II-B


def pgen_expq_fp32(acc: np.ndarray, scale: float, m, scale6: bool = False):
    """Exp-then-quantize, Eq. (post-softmax-path), on raw dot products (fp32,
    -inf = masked) with one running maximum per row: p_t = fl32(e^{x_t}),
    x_t = fl(fl(acc*scale) - m); per 32-key block the OCP exponent
    floor(log2 max p) - 2 (or the scale6 exponent ceil(log2(max p / 6))),
    then p / 2^k rounded to the nearest E2M1 value.  Written with frexp and
    a threshold search instead of the C oracle's nearest-value loop.
    Returns (codes int64 [rows, cols], k int64 [rows, nblk])."""
    acc = np.asarray(acc, F32)
    rows, cols = acc.shape
    nblk = (cols + 31) // 32
    pad = nblk * 32 - cols
    a = np.concatenate([acc, np.full((rows, pad), -np.inf, F32)], axis=1).reshape(rows, nblk, 32)
    m = np.asarray(m, F32).reshape(rows, 1, 1)
    masked = np.isneginf(a)
    with np.errstate(invalid="ignore"):
        x = (a * F32(scale)) - m
    p = np.where(masked, 0.0, np.exp(np.where(masked, 0.0, x).astype(np.float64))).astype(F32)
    amax = p.max(axis=2).astype(np.float64)                     # [rows, nblk]
    mant, ex = np.frexp(np.where(amax > 0, amax, 1.0))          # amax = mant 2^ex, mant in [0.5, 1)
    if scale6:
        # smallest k with 6 2^k >= amax: with amax = f 2^(ex-1), f in [1, 2),
        # that is ex - 3 when f <= 1.5, else ex - 2
        k = np.where(mant * 2 <= 1.5, ex - 3, ex - 2)
    else:
        k = ex - 1 - 2
    k = np.where(amax > 0, np.clip(k, -127, 127), -127).astype(np.int64)
    y = p.astype(np.float64) * np.exp2(-k.astype(np.float64))[:, :, None]
    c = e2m1_rne(y)
    return c.reshape(rows, nblk * 32)[:, :cols], k


def attn_twin(q_bits, k_bits, v_bits, scale: float, causal: bool, mode: str = "efq",
              tau: float = -3.06, h: float = 2.30, bc: int = 64):
    """Algorithm 2 over key tiles of bc keys in ascending order, for every
    query row, written independently of the C oracle (vectorised over the
    rows of one (batch, query head)).

    mode: "efq" or "lut" (Alg. 1, same fp32 decision contract as
    pgen_fp32), "expq" / "expq6" (exp-then-quantize).  V is the MXFP4 V~ of
    quant_v_bits.  Grouped-query attention: query head hq reads key/value
    head hq // (Hq / Hkv).  Per tile: S = fl32(acc * scale) with acc the fp32
    rounding of the dot product accumulated in fp64 over head_dim in order;
    m_new = max(m, max S) (Eq. rowmax-update); alpha = exp(m - m_new)
    (Eq. alpha, 0 before the first tile); A = alpha A + P~ V~ and
    l = alpha l + P~ 1 in fp64 (Eqs. numerator-lowbit, denominator-basic);
    O = fl32(A / l).  A row skips every tile that starts past its last
    visible key.

    Returns (out fp32 [B*Hq*Sq, D], codes uint8 [rows, nblk*32],
    e8m0 uint8 [rows, nblk], m fp32 [rows], l fp64 [rows]), rows ordered
    (b, hq, i)."""
    q_bits = np.asarray(q_bits, np.uint16)
    k_bits = np.asarray(k_bits, np.uint16)
    B, Sq, Hq, D = q_bits.shape
    _, Sk, Hkv, _ = k_bits.shape
    grp = Hq // Hkv
    nblk = (Sk + 31) // 32
    as64 = lambda b: (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    qf, kf = as64(q_bits), as64(k_bits)
    vc, ve = quant_v_bits(v_bits)                     # [B, Hkv, nblk*32, D], [B, Hkv, nblk, D]
    mag = C8[vc & 7] * np.exp2(np.repeat(ve.astype(np.float64) - 127, 32, axis=2))
    vhat = np.where(vc & 8, -mag, mag)
    out = np.zeros((B, Hq, Sq, D), np.float32)
    codes = np.zeros((B, Hq, Sq, nblk * 32), np.uint8)
    e8 = np.zeros((B, Hq, Sq, nblk), np.uint8)
    mm = np.zeros((B, Hq, Sq), np.float32)
    ll = np.zeros((B, Hq, Sq), np.float64)
    rows = np.arange(Sq)
    kend = rows + 1 if causal else np.full(Sq, Sk)    # keys [0, kend) are visible
    for b in range(B):
        for hq in range(Hq):
            g = hq // grp
            dot = np.zeros((Sq, Sk))
            for d in range(D):                        # fp64, head_dim in order
                dot += qf[b, :, hq, d][:, None] * kf[b, :, g, d][None, :]
            acc_all = dot.astype(F32)
            m = np.full(Sq, -np.inf, F32)
            A = np.zeros((Sq, D))
            l = np.zeros(Sq)
            for j0 in range(0, Sk, bc):
                act = j0 < kend                       # rows that reach this tile
                if not act.any():
                    break
                t = np.arange(j0, j0 + bc)
                vis = (t[None, :] < Sk) & (t[None, :] < kend[:, None])
                acc = np.full((Sq, bc), -np.inf, F32)
                nt = min(bc, Sk - j0)
                acc[:, :nt] = acc_all[:, j0:j0 + nt]
                acc = np.where(vis, acc, F32(-np.inf))[act]
                S = np.where(np.isneginf(acc), F32(-np.inf), acc * F32(scale))
                mnew = np.maximum(m[act], S.max(axis=1))
                if mode in ("efq", "lut"):
                    c, kb = pgen_fp32(acc, tau, h, lut=(mode == "lut"), scale=scale, m=mnew)
                else:
                    c, kb = pgen_expq_fp32(acc, scale, mnew, scale6=(mode == "expq6"))
                p = C8[c] * np.exp2(np.repeat(kb, 32, axis=1)[:, :bc].astype(np.float64))
                mo = m[act].astype(np.float64)
                alpha = np.where(np.isneginf(mo), 0.0,
                                 np.exp(np.where(np.isneginf(mo), 0.0, mo - mnew.astype(np.float64))))
                vt = np.zeros((bc, D))
                vt[:nt] = vhat[b, g, j0:j0 + nt]
                A[act] = alpha[:, None] * A[act] + p @ vt
                l[act] = alpha * l[act] + p[:, :nt].sum(axis=1)
                m[act] = mnew
                blk0 = j0 // 32
                nb = min(bc // 32, nblk - blk0)
                ci = codes[b, hq]
                ci[act, j0:j0 + nb * 32] = c[:, :nb * 32]
                e8[b, hq][act, blk0:blk0 + nb] = (kb[:, :nb] + 127).astype(np.uint8)
            with np.errstate(invalid="ignore", divide="ignore"):
                o = np.where(l[:, None] > 0, A / l[:, None], 0.0)
            out[b, hq] = o.astype(np.float32)
            mm[b, hq], ll[b, hq] = m, l
    return (out.reshape(-1, D), codes.reshape(-1, nblk * 32), e8.reshape(-1, nblk),
            mm.reshape(-1), ll.reshape(-1))
