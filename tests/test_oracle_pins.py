"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: the
paper's printed constants, closed forms that follow from Eqs. (k-rule),
(k-interval), (z-def), (d8-index) and the threshold form of Sec. II-C, a
brute-force exp-then-quantize search, numpy's softmax, invariants of the
online recurrence (Alg. 2), and an independently written numpy twin.
"""
import math
import os

import numpy as np
import pytest
import torch

from paper_2609_09721_amd import inputs

HERE = os.path.dirname(os.path.abspath(__file__))
LN2, LN6 = math.log(2.0), math.log(6.0)
POINTS = {"mean": (-3.06, 2.30), "mmlu": (-2.90, 2.00), "balance": (-2.10, 2.70)}


def golden_constants():
    vals = {}
    with open(os.path.join(HERE, "golden", "operating_points.txt")) as f:
        for line in f:
            line = line.split("#")[0].split()
            if line:
                vals[line[0]] = [float(v) for v in line[1:]]
    return vals


def blocks_with_max(rng, M, n_other=31, spread=2.0):
    """Blocks of 32 shifted scores whose maximum is exactly M (fp32)."""
    M = np.asarray(M, np.float32).reshape(-1, 1)
    x = (M - rng.exponential(spread, size=(M.shape[0], n_other))).astype(np.float32)
    return np.concatenate([M, x], axis=1)


# --------------------------------------------------------------- constants
def test_constants_match_paper(orc):
    g = golden_constants()
    assert orc.MEAN == (g["mean_tau"][0], g["mean_h"][0])
    assert orc.MMLU == (g["mmlu_tau"][0], g["mmlu_h"][0])
    assert orc.BALANCE == (g["balance_tau"][0], g["balance_h"][0])
    assert orc.LUT[0] == pytest.approx(math.log(g["lut_tau_num"][0] / g["lut_tau_den"][0]), abs=1e-15)
    assert orc.LUT[1] == pytest.approx(g["lut_h_num"][0] / math.log(g["lut_h_logarg"][0]), abs=1e-15)
    assert list(orc.C16) == [int(v) for v in g["c16"]]
    assert list(orc.C8) == g["c8"]


# ------------------------------------------------------ scale rule (P1, P2)
def test_k_rule_interval(orc):
    """Eq. (k-interval): 2^k <= 2 e^M / 9 < 2^(k+1), for block maxima M <= 0."""
    rng = np.random.default_rng(1)
    M = np.concatenate([rng.uniform(-86, 0, 200000), -rng.exponential(1.0, 50000)]).astype(np.float32)
    x = blocks_with_max(rng, M)
    _, e8 = orc.pgen(x)
    k = e8[:, 0].astype(np.int64) - 127
    arg = (M.astype(np.float64) + math.log(2 / 9)) / LN2
    away = np.abs(arg - np.round(arg)) > 1e-6
    lhs = 2.0 ** k
    val = 2 * np.exp(M.astype(np.float64)) / 9
    assert away.mean() > 0.99
    assert np.all(lhs[away] <= val[away]) and np.all(val[away] < 2 * lhs[away])
    # equivalently e^M / s_b in [4.5, 9): the midpoint between codes 3 and 6
    ratio = np.exp(M.astype(np.float64)) / lhs
    assert np.all((ratio[away] >= 4.5) & (ratio[away] < 9.0))


def test_k_rule_special_values(orc):
    x = np.full((4, 32), -np.inf, np.float32)
    x[0, 0] = 0.0             # row maximum in the block: k = -3
    x[1, 0] = -87.0           # k would be -129: clamped to the E8M0 minimum
    x[2, 0] = -200.0
    # row 3 fully masked: no visible key
    _, e8 = orc.pgen(x)
    assert list(e8[:, 0].astype(int) - 127) == [-3, -127, -127, -127]
    # boundary values M = j log2 - log(2/9) sit at the k step; one ulp below
    # must give the smaller k
    for j in range(-20, -2):
        Mb = np.float32(j * LN2 - math.log(2 / 9))
        lo = np.nextafter(np.nextafter(Mb, np.float32(-np.inf)), np.float32(-np.inf))
        hi = np.nextafter(np.nextafter(Mb, np.float32(np.inf)), np.float32(np.inf))
        xs = np.full((2, 32), -np.inf, np.float32)
        xs[0, 0], xs[1, 0] = lo, hi
        _, e = orc.pgen(xs)
        assert int(e[0, 0]) - 127 == j - 1 and int(e[1, 0]) - 127 == j


def test_residual_range(orc):
    """z_max = M - k log2 - log6 lies in [log 3/4, log 3/2) (from Eq. k-interval)."""
    rng = np.random.default_rng(2)
    M = rng.uniform(-60, 0, 100000).astype(np.float32)
    _, e8 = orc.pgen(blocks_with_max(rng, M))
    k = e8[:, 0].astype(np.int64) - 127
    zmax = M.astype(np.float64) - k * LN2 - LN6
    assert zmax.min() >= math.log(0.75) - 1e-6
    assert zmax.max() < math.log(1.5) + 1e-6


# ------------------------------------------------------- code rule (P3-P7)
@pytest.mark.parametrize("point", ["mean", "mmlu", "balance"])
def test_code_matches_threshold_form(orc, point):
    """Sec. II-C: code c is selected when tau + (c-1)/h <= z < tau + c/h,
    c = 0 below the first threshold, c = 7 above the last one."""
    tau, h = POINTS[point]
    rng = np.random.default_rng(3)
    n = 4000
    x = np.zeros((n, 32), np.float32)           # block maximum 0: k = -3
    x[:, 1:] = -rng.uniform(0, 6, size=(n, 31)).astype(np.float32)
    codes, e8 = orc.pgen(x, tau=tau, h=h)
    assert np.all(e8 == 124)
    z = x.astype(np.float64) + 3 * LN2 - LN6
    thr = tau + np.arange(0, 7) / h              # tau + (c-1)/h for c = 1..7
    expect = (z[..., None] >= thr).sum(-1)
    near = np.min(np.abs(z[..., None] - thr), axis=-1) < 1e-5
    assert near.mean() < 1e-3
    assert np.array_equal(codes[~near], expect[~near])


def test_code_thresholds_mean_printed():
    """Threshold list tau + c/h of the Mean point (c = 0..6)."""
    tau, h = POINTS["mean"]
    thr = [tau + c / h for c in range(7)]
    want = [-3.06, -2.6252, -2.1904, -1.7557, -1.3209, -0.8861, -0.4513]
    assert np.allclose(thr, want, atol=6e-5)


def test_code_flips_at_threshold(orc):
    """Bisect the oracle's decision in x: the code steps at z = tau + c/h."""
    tau, h = POINTS["mean"]
    for c in range(7):
        zt = tau + c / h
        xt = zt - 3 * LN2 + LN6                  # k = -3 (block max 0)
        lo, hi = xt - 1e-3, xt + 1e-3
        for _ in range(40):
            mid = np.float32((lo + hi) / 2)
            x = np.full((1, 32), -np.inf, np.float32)
            x[0, 0], x[0, 1] = 0.0, mid
            codes, _ = orc.pgen(x, tau=tau, h=h)
            if codes[0, 1] > c:
                hi = float(mid)
            else:
                lo = float(mid)
        assert abs(hi - xt) < 2e-6, (c, hi, xt)


def test_lut_matches_index_threshold_form(orc):
    """Sec. II-D: the LUT index j16 counts the thresholds tau16 + (j-1)/h16
    (j = 1..15) at or below z, and the code is C16[j16] (the printed table)."""
    g = golden_constants()
    tau16 = math.log(g["lut_tau_num"][0] / g["lut_tau_den"][0])
    h16 = g["lut_h_num"][0] / math.log(g["lut_h_logarg"][0])
    c16 = np.array([int(v) for v in g["c16"]])
    rng = np.random.default_rng(31)
    n = 4000
    x = np.zeros((n, 32), np.float32)            # block maximum 0: k = -3
    x[:, 1:] = -rng.uniform(0, 6, size=(n, 31)).astype(np.float32)
    codes, e8 = orc.pgen(x, orc.LUT_MODE, *orc.LUT)
    assert np.all(e8 == 124)
    z = x.astype(np.float64) + 3 * LN2 - LN6
    thr = tau16 + np.arange(0, 15) / h16
    j16 = (z[..., None] >= thr).sum(-1)
    near = np.min(np.abs(z[..., None] - thr), axis=-1) < 1e-5
    assert near.mean() < 1e-3
    assert np.array_equal(codes[~near], c16[j16][~near])


def test_lut_index_steps_at_threshold(orc):
    """Bisect the oracle's LUT decision in x: the index (so the code, where
    C16 steps) changes at z = tau16 + j/h16."""
    tau16, h16 = orc.LUT
    c16 = list(orc.C16)
    for j in range(15):
        if c16[j] == c16[j + 1]:
            continue
        xt = tau16 + j / h16 - 3 * LN2 + LN6
        lo, hi = xt - 1e-3, xt + 1e-3
        for _ in range(40):
            mid = np.float32((lo + hi) / 2)
            x = np.full((1, 32), -np.inf, np.float32)
            x[0, 0], x[0, 1] = 0.0, mid
            codes, _ = orc.pgen(x, orc.LUT_MODE, tau16, h16)
            if codes[0, 1] > c16[j]:
                hi = float(mid)
            else:
                lo = float(mid)
        assert abs(hi - xt) < 2e-6, (j, hi, xt)


def test_format_and_nonnegativity(orc):
    """Codes are non-negative E2M1 patterns 0..7; E8M0 = k + 127 <= 124 for x <= 0."""
    rng = np.random.default_rng(4)
    x = -rng.exponential(3.0, size=(20000, 32)).astype(np.float32)
    x[rng.random(x.shape) < 0.05] = -np.inf
    for mode, (tau, h) in [(orc.EFQ, orc.MEAN), (orc.EFQ, orc.BALANCE), (orc.LUT_MODE, orc.LUT),
                           (orc.EXPQ, orc.MEAN)]:
        codes, e8 = orc.pgen(x, mode, tau, h)
        assert codes.max() <= 7 and e8.max() <= 124


@pytest.mark.parametrize("point", ["mean", "mmlu", "balance", "lut"])
def test_block_max_element(orc, point):
    """Weak form (all points): the block maximum gets the block's largest code.
    Strong form (Mean, tau + 6/h <= log 3/4): it always gets code 7."""
    rng = np.random.default_rng(5)
    M = rng.uniform(-40, 0, 50000).astype(np.float32)
    x = blocks_with_max(rng, M)
    mode, (tau, h) = (orc.LUT_MODE, orc.LUT) if point == "lut" else (orc.EFQ, POINTS[point])
    codes, _ = orc.pgen(x, mode, tau, h)
    assert np.all(codes[:, 0] == codes.max(axis=1))
    if point == "mean":
        assert tau + 6 / h <= math.log(0.75)
        assert np.all(codes[:, 0] == 7)


@pytest.mark.parametrize("point", ["mean", "mmlu", "balance", "lut"])
def test_row_max_element(orc, point):
    """x = 0 (the row maximum): k = -3, z = log(4/3), code 7, value 0.75."""
    mode, (tau, h) = (orc.LUT_MODE, orc.LUT) if point == "lut" else (orc.EFQ, POINTS[point])
    x = np.full((1, 32), -np.inf, np.float32)
    x[0, 0] = 0.0
    codes, e8 = orc.pgen(x, mode, tau, h)
    assert codes[0, 0] == 7 and e8[0, 0] == 124
    assert orc.C8[codes[0, 0]] * 2.0 ** (int(e8[0, 0]) - 127) == 0.75


@pytest.mark.parametrize("point,lo,hi", [("mean", -1, 2), ("mmlu", -1, 1), ("balance", -1, 0),
                                         ("lut", -1, 1)])
def test_vs_bruteforce_exp_then_quantize(orc, point, lo, hi):
    """Against exp-then-quantize with the same block scale: compute 6 e^z,
    search the nearest C8 value by brute force; EFQ's code stays within a
    fixed offset of it, and |s C8[c] - e^x| <= 3 s."""
    rng = np.random.default_rng(6)
    M = rng.uniform(-10, 0, 20000).astype(np.float32)
    x = blocks_with_max(rng, M)
    mode, (tau, h) = (orc.LUT_MODE, orc.LUT) if point == "lut" else (orc.EFQ, POINTS[point])
    codes, e8 = orc.pgen(x, mode, tau, h)
    s = 2.0 ** (e8[:, :1].astype(np.float64) - 127)
    p = np.exp(x.astype(np.float64))
    nearest = np.abs((p / s)[..., None] - orc.C8).argmin(-1)
    d = codes.astype(int) - nearest
    assert d.min() >= lo and d.max() <= hi
    assert d.min() == lo and d.max() == hi          # the bounds are attained
    assert np.max(np.abs(s * orc.C8[codes] - p) / s) <= 3.0


U32 = 2.0 ** -24            # unit roundoff of fp32


def _contract_vs_real(orc, x, mode, tau, h):
    """Compare the fp32 decision contract with the fp64 step-by-step reading
    of Alg. 1 (M_b, k_b = floor((M_b + log(2/9)) / log 2), z = x - k_b log 2 -
    log 6, c = clip(floor((z - tau) h) + 1, 0, 7), or the 16-level LUT index).
    Returns the per-code disagreement mask, the distances of the real u to
    the nearest integer there, their stated bounds, and the same for k."""
    lut = mode == orc.LUT_MODE
    c32, e32 = orc.pgen(x, mode, tau, h)
    c64, k64, u64 = orc.pgen_real(x.astype(np.float64), lut, tau, h)
    rows, cols = x.shape
    nb = k64.shape[1]
    xp = np.concatenate([x, np.full((rows, nb * 32 - cols), -np.inf, np.float32)], 1)
    Mb = xp.reshape(rows, nb, 32).max(axis=2).astype(np.float64)
    kbad = (e32.astype(np.int64) - 127) != k64
    fin = np.isfinite(Mb)
    q64 = np.where(fin, (np.where(fin, Mb, 0) + math.log(2 / 9)) / LN2, 0.0)
    kdist = np.abs(q64 - np.round(q64))
    # the fp32 k_b argument is three fp32 roundings of operands below |M_b| + 2
    kbound = 4 * U32 * (np.abs(np.where(fin, Mb, 0)) + 2) / LN2
    tau_r, h_r = (math.log(1 / 24), 14 / math.log(24)) if lut else (tau, h)
    kagree = np.repeat(~kbad, 32, axis=1)[:, :cols]
    bad = (c32 != c64) & kagree
    kk = np.repeat(k64, 32, axis=1)[:, :cols].astype(np.float64)
    with np.errstate(invalid="ignore"):
        mag = h_r * (np.abs(x.astype(np.float64)) + np.abs(kk) * LN2 + LN6 + abs(tau_r)) + \
            np.abs(u64) + 2
        udist = np.abs(u64 - np.round(u64))
    # the contract's argument w ~ 32 (u + 1) - 1/2 is about eight fp32
    # roundings of terms of size <= mag (in units of u)
    ubound = 4 * U32 * mag
    return bad, udist, ubound, kbad, kdist, kbound


@pytest.mark.parametrize("point", ["mean", "mmlu", "balance", "lut"])
def test_contract_vs_real_valued(orc, point):
    """The fp32 decision contract of the oracle (the fused argument of
    readings R-1 / R-2) against Alg. 1 evaluated step by step in fp64, at
    every operating point of Sec. IV-A and the LUT constants of Sec. II-D.

    Stated bound: a code differs only where the real u = (z - tau) h lies
    within 4 u32 (h (|x| + |k_b| log 2 + log 6 + |tau|) + |u| + 2) of an
    integer (a code threshold), and k_b differs only where
    (M_b + log(2/9)) / log 2 lies within 4 u32 (|M_b| + 2) / log 2 of an
    integer.  Checked on scores placed within +-2 ulps of every threshold and
    every k_b boundary (where disagreements are expected, and all must sit
    inside the bound) and on random scores (where they must be rare)."""
    from adversarial import adversarial_scores
    mode, (tau, h) = (orc.LUT_MODE, orc.LUT) if point == "lut" else (orc.EFQ, POINTS[point])
    rng = np.random.default_rng(7)
    adv = adversarial_scores(rng, 600, 256, tau, h)
    bad, udist, ubound, kbad, kdist, kbound = _contract_vs_real(orc, adv, mode, tau, h)
    assert bad.sum() > 0                       # the set does reach the thresholds
    assert np.all(udist[bad] <= ubound[bad]), np.max(udist[bad] / ubound[bad])
    assert np.all(kdist[kbad] <= kbound[kbad])
    x = -rng.exponential(2.5, size=(40000, 32)).astype(np.float32)
    x[:, 0] = -rng.exponential(0.5, size=40000).astype(np.float32)
    bad, udist, ubound, kbad, kdist, kbound = _contract_vs_real(orc, x, mode, tau, h)
    assert bad.mean() < 1e-5 and kbad.mean() < 1e-5
    assert np.all(udist[bad] <= ubound[bad]) and np.all(kdist[kbad] <= kbound[kbad])


def test_ln2_equivariance(orc):
    """Eq. (z-def): shifting a block by -j log2 lowers k by j and leaves the
    codes unchanged (fp64 reading; fp32 differs only next to thresholds)."""
    rng = np.random.default_rng(8)
    x = -rng.exponential(2.0, size=(5000, 32))
    x[:, 0] = -rng.uniform(0, 0.5, 5000)
    c0, k0, u0 = orc.pgen_real(x)
    for j in (1, 3, 17):
        c1, k1, u1 = orc.pgen_real(x - j * LN2)
        assert np.array_equal(k1, k0 - j)
        near = np.abs(u0 - np.round(u0)) < 1e-9
        assert np.array_equal(c1[~near], c0[~near])


def test_twin_agrees_pgen(orc):
    """C oracle and numpy twin: bit-identical codes and scales, including
    masked keys, partial blocks, tiny and huge magnitudes."""
    from oracle import twin
    rng = np.random.default_rng(9)
    x = -rng.exponential(3.0, size=(3000, 80)).astype(np.float32)   # 2.5 blocks per row
    x[rng.random(x.shape) < 0.1] = -np.inf
    x[::7, ::5] = 0.0
    x[5::11] *= np.float32(40.0)
    x[3::13, :3] = -np.float32(1e-40)                               # subnormal
    for mode, (tau, h) in [(orc.EFQ, orc.MEAN), (orc.EFQ, orc.MMLU), (orc.LUT_MODE, orc.LUT)]:
        c, e = orc.pgen(x, mode, tau, h)
        c2, k2 = twin.pgen_fp32(x, tau, h, lut=(mode == orc.LUT_MODE))
        assert np.array_equal(c, c2)
        assert np.array_equal(e.astype(int) - 127, k2)
    # the scale/offset form used inside attention (raw dot products, scale, m)
    acc = rng.normal(0, 8, size=(2000, 64)).astype(np.float32)
    scale = np.float32(1 / math.sqrt(128))
    m = np.float32((acc.max() * scale))
    c_tw, k_tw = twin.pgen_fp32(acc, *orc.MEAN, scale=scale, m=m)
    xs = (acc * scale) - m
    c_or, e_or = orc.pgen(xs)
    # not the same evaluation (fused vs shifted input), so only mostly equal
    assert np.mean(c_tw == c_or) > 0.999
    assert np.array_equal(e_or.astype(int) - 127, k_tw)


# ---------------------------------------------------------------- EXPQ pins
def test_expq_definition(orc):
    """Eq. (post-softmax-path) with the OCP MXFP4 rule: the row maximum
    (p = 1) is encoded exactly, the block max maps to 4 or 6 times 2^k, and
    each element is the nearest E2M1 value (error <= half a grid step)."""
    rng = np.random.default_rng(10)
    M = rng.uniform(-20, 0, 20000).astype(np.float32)
    x = blocks_with_max(rng, M)
    x[0, 0] = 0.0
    codes, e8 = orc.pgen(x, orc.EXPQ)
    k = e8[:, :1].astype(np.float64) - 127
    assert codes[0, 0] == 6 and e8[0, 0] == 125            # 4 * 2^-2 = 1
    assert set(np.unique(codes[:, 0])) <= {6, 7}
    p = np.exp(x.astype(np.float32).astype(np.float64)).astype(np.float32).astype(np.float64)
    y = p / 2.0 ** k
    assert np.all((y.max(axis=1) >= 4) & (y.max(axis=1) < 8))
    grid = np.array(orc.C8)
    err = np.abs(grid[codes] - y)
    step = np.where(y < 2, 0.25, np.where(y < 4, 0.5, np.where(y <= 6, 1.0, 2.0)))
    assert np.all(err <= step + 1e-12)


def test_expq_scale6_definition(orc):
    """The scale6 comparison rule: 2^k is the smallest power of two with
    6 * 2^k >= max p, so max p / 2^k lies in (3, 6] and no element
    saturates; the row maximum p = 1 gets k = -2 (1 / 2^-2 = 4, code 6);
    a block max just above 6 * 2^j moves k to j + 1; each element is the
    nearest E2M1 value."""
    rng = np.random.default_rng(12)
    M = rng.uniform(-20, 0, 20000).astype(np.float32)
    x = blocks_with_max(rng, M)
    x[0, 0] = 0.0
    codes, e8 = orc.pgen(x, orc.EXPQ6)
    k = e8[:, :1].astype(np.float64) - 127
    assert codes[0, 0] == 6 and e8[0, 0] == 125            # 1 = 4 * 2^-2
    p = np.exp(x.astype(np.float32).astype(np.float64)).astype(np.float32).astype(np.float64)
    y = p / 2.0 ** k
    ymax = y.max(axis=1)
    assert np.all((ymax > 3) & (ymax <= 6))
    # the scale is the smallest power of two that keeps the block max <= 6
    assert np.all(p.max(axis=1) / 2.0 ** (k[:, 0] - 1) > 6)
    grid = np.array(orc.C8)
    err = np.abs(grid[codes] - y)
    step = np.where(y < 2, 0.25, np.where(y < 4, 0.5, 1.0))
    assert np.all(err <= step + 1e-12)
    # boundary: p_max = 6 * 2^-3 = 0.75 exactly gives k = -3 (ratio 6, code 7);
    # the next fp32 value above it gives k = -2 (ratio just above 3, code 5)
    for pm, kk, c in [(0.75, -3, 7), (float(np.nextafter(np.float32(0.75), np.float32(1))), -2, 5)]:
        xb = np.full((1, 32), -np.inf, np.float32)
        # a score whose fp32 exp is pm: search the float32 neighbourhood of log(pm)
        s0 = np.float32(np.log(pm))
        cand = [s0]
        for _ in range(4):
            cand += [np.nextafter(cand[-1], np.float32(-np.inf))]
        cand += [np.nextafter(s0, np.float32(np.inf))]
        hit = [v for v in cand if np.float32(np.exp(np.float64(v))) == np.float32(pm)]
        assert hit, pm
        xb[0, 0] = hit[0]
        cb, eb = orc.pgen(xb, orc.EXPQ6)
        assert int(eb[0, 0]) - 127 == kk and int(cb[0, 0]) == c, (pm, eb, cb)


# ------------------------------------------------------------- V quantiser
def _bits(t):
    return t.view(torch.int16).numpy().view(np.uint16)


def test_vquant_twin_and_bounds(orc):
    from oracle import twin
    g = torch.Generator().manual_seed(11)
    v = torch.randn(2, 75, 3, 40, generator=g) * torch.exp2(torch.randint(-20, 20, (1, 1, 3, 40), generator=g).float())
    v[0, 5:9, 1, 3] = 0.0
    v[1, :, 2, 7] = 0.0                                    # all-zero column
    v[1, 40, 0, 0] = -1e-39                                # bf16 subnormal
    vb = _bits(v.to(torch.bfloat16))
    c, e = orc.quant_v(vb)
    c2, e2 = twin.quant_v_bits(vb)
    assert np.array_equal(c, c2) and np.array_equal(e, e2)
    vals = orc.bits_to_f64(vb)                              # [B, S, H, D]
    B, S, H, D = vb.shape
    nblk = (S + 31) // 32
    k = e.astype(np.float64) - 127                          # [B, H, nblk, D]
    kk = np.repeat(k, 32, axis=2)[:, :, :S]                 # per key
    vv = vals.transpose(0, 2, 1, 3)                         # [B, H, S, D]
    mag = orc.C8[c[:, :, :S] & 7] * 2.0 ** kk
    vhat = np.where(c[:, :, :S] & 8, -mag, mag)
    y = np.abs(vv) / 2.0 ** kk
    step = np.where(y < 2, 0.25, np.where(y < 4, 0.5, np.where(y <= 6, 1.0, 2.0)))
    assert np.all(np.abs(vhat - vv) <= step * 2.0 ** kk * (1 + 1e-12))
    # the block maximum maps to magnitude code 6 or 7 (values 4 or 6)
    blocks = (c & 7).reshape(B, H, nblk, 32, D).max(axis=3)
    assert np.all(np.isin(blocks[k > -127], [6, 7]))
    # all-zero column: scale 0x00 and zero codes
    assert np.all(e[1, 2, :, 7] == 0) and np.all(c[1, 2, :, 7] == 0)


def test_vquant_ties_to_even(orc):
    # block max 4 -> k = 0, so elements are quantised on the E2M1 grid itself
    ties = [0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 7.0, -0.75]
    want = [0, 2, 2, 4, 4, 6, 6, 7, 0x8 | 2]
    v = torch.zeros(1, 32, 1, 1)
    v[0, 0, 0, 0] = 4.0
    for i, t in enumerate(ties):
        v[0, 1 + i, 0, 0] = t
    c, e = orc.quant_v(_bits(v.to(torch.bfloat16)))
    assert e[0, 0, 0, 0] == 127 + 0
    assert list(c[0, 0, 1:1 + len(ties), 0]) == want


# ------------------------------------------------------ attention recurrence
def _tiny(seed=1, S=256, D=64, Hq=2, Hkv=1, dist="normal", causal=False):
    w = inputs.Workload("t", 1, Hq, Hkv, S, D, causal, dist, seed)
    q, k, v = inputs.make_qkv(w)
    return w, q, k, v


def test_exact_mode_matches_numpy_softmax(orc):
    """EXACT mode of the online recurrence (tiles of 32 keys, Eq. alpha
    rescaling) equals softmax(Q K^T / sqrt d) V computed directly."""
    for causal in (False, True):
        w, q, k, v = _tiny(S=200, causal=causal, Hq=4, Hkv=2)
        out = orc.attn(orc.bf16_bits(q), orc.bf16_bits(k), orc.bf16_bits(v), w.scale, causal,
                       orc.EXACT, bc=32)
        qf, kf, vf = (orc.bits_to_f64(orc.bf16_bits(t)) for t in (q, k, v))
        ref = []
        for h in range(4):
            s = qf[0, :, h] @ kf[0, :, h // 2].T * w.scale
            if causal:
                s = np.where(np.tri(200, dtype=bool), s, -np.inf)
            p = np.exp(s - s.max(1, keepdims=True))
            p /= p.sum(1, keepdims=True)
            ref.append(p @ vf[0, :, h // 2])
        ref = np.stack(ref)                                   # [H, S, D]
        got = out.reshape(1, 4, 200, 64)[0]
        assert np.max(np.abs(got - ref)) < 1e-6


def test_same_operand_numerator_denominator(orc):
    """Sec. III-A: with V = c 1 for c on the E2M1 x 2^j grid, O = c exactly
    up to rounding, because the same operand feeds P~V and P~1."""
    w, q, k, v = _tiny(S=256, causal=False, dist="qwen", D=128)
    for c in (1.0, -3.0, 0.375):
        vc = torch.full_like(v, c)
        for mode, bc in [(orc.EFQ, 64), (orc.EXPQ, 64), (orc.LUT_MODE, 128)]:
            out = orc.attn(orc.bf16_bits(q), orc.bf16_bits(k), orc.bf16_bits(vc), w.scale,
                           False, mode, bc=bc)
            assert np.max(np.abs(out - c)) <= 1e-6 * abs(c)


def test_single_visible_key(orc):
    """Causal row 0 sees key 0 only: O_0 equals the quantised v_0."""
    w, q, k, v = _tiny(S=96, causal=True, Hq=1, Hkv=1)
    rows = np.array([[0, 0, 0]], np.int32)
    out = orc.attn(orc.bf16_bits(q), orc.bf16_bits(k), orc.bf16_bits(v), w.scale, True, orc.EFQ,
                   rows=rows)
    c, e = orc.quant_v(orc.bf16_bits(v))
    kk = e[0, 0, 0].astype(np.float64) - 127
    vhat = orc.C8[c[0, 0, 0] & 7] * 2.0 ** kk * np.where(c[0, 0, 0] & 8, -1, 1)
    assert np.array_equal(out[0], vhat.astype(np.float32))


def test_decision_margin_single_key(orc):
    """Causal row 0: the only visible score is the row maximum, so M_b = 0
    and k_b = floor(log(2/9) / log 2) = -3 (Eq. k-rule).  The nearest
    decision change is that floor at the integer -2, at a distance
    |2 log 2 + log(2/9)| / scale in dot-product units; the code of the max
    (u ~ 7.70 for Mean, code 7) is farther from its thresholds."""
    w, q, k, v = _tiny(S=96, causal=True, Hq=1, Hkv=1)
    rows = np.array([[0, 0, 0]], np.int32)
    out, mg = orc.attn(orc.bf16_bits(q), orc.bf16_bits(k), orc.bf16_bits(v), w.scale, True,
                       orc.EFQ, rows=rows, margins=True)
    want = abs(2 * math.log(2) + math.log(2 / 9)) / w.scale
    assert abs(mg[0] - want) <= 1e-5 * want
    # more keys can only bring a decision closer to its threshold
    rows = np.array([[0, 0, i] for i in range(96)], np.int32)
    _, mg = orc.attn(orc.bf16_bits(q), orc.bf16_bits(k), orc.bf16_bits(v), w.scale, True,
                     orc.EFQ, rows=rows, margins=True)
    assert np.all(mg > 0) and np.all(mg <= want * (1 + 1e-5))


def _dominant_key0(D=64, S=256, seed=3):
    """Dyadic inputs where key 0 holds the maximum score of every row."""
    g = torch.Generator().manual_seed(seed)
    q = torch.randint(-1, 2, (1, S, 1, D), generator=g).float() * 0.5
    k = torch.randint(-1, 2, (1, S, 1, D), generator=g).float() * 0.5
    q[..., :16] = 2.0
    k[:, 1:, :, :16] = -2.0
    k[:, 0, :, :16] = 2.0
    v = torch.randn(1, S, 1, D, generator=g)
    return [orc_bits(t) for t in (q, k, v)]


def orc_bits(t):
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def test_online_equals_single_tile_when_max_is_first(orc):
    """If key 0 holds every row's maximum, m never changes after the first
    tile (alpha = 1), so tiles of 32 keys give the same codes, scales and
    output as one tile spanning all keys."""
    qb, kb, vb = _dominant_key0()
    scale = 1 / 8
    for mode in (orc.EFQ, orc.LUT_MODE, orc.EXPQ):
        o1, c1, e1, m1, l1 = orc.attn(qb, kb, vb, scale, False, mode, bc=32, dump=True)
        o2, c2, e2, m2, l2 = orc.attn(qb, kb, vb, scale, False, mode, bc=256, dump=True)
        assert np.array_equal(c1, c2) and np.array_equal(e1, e2) and np.array_equal(m1, m2)
        assert np.allclose(l1, l2, rtol=1e-14)
        assert np.max(np.abs(o1 - o2)) <= 1e-6


def test_attn_dump_matches_pgen_twin(orc):
    """The codes the recurrence feeds to P~V (single tile, dyadic scores,
    so acc is exact) are those of the twin's Alg. 1 on the same (acc, m)."""
    from oracle import twin
    w = inputs.Workload("d", 1, 1, 1, 192, 64, False, "dyadic", 12)
    q, k, v = inputs.dyadic_qkv(w)
    qb, kb, vb = (orc.bf16_bits(t) for t in (q, k, v))
    out, codes, e8, m, l = orc.attn(qb, kb, vb, w.scale, False, orc.EFQ, bc=256, dump=True)
    qf, kf = orc.bits_to_f64(qb), orc.bits_to_f64(kb)
    acc = (qf[0, :, 0] @ kf[0, :, 0].T).astype(np.float32)        # exact dyadic sums
    S = acc * np.float32(w.scale)
    mrow = S.max(axis=1)
    assert np.array_equal(m, mrow)
    for i in range(0, 192, 17):
        c2, k2 = twin.pgen_fp32(acc[i:i + 1], *orc.MEAN, scale=w.scale, m=mrow[i])
        assert np.array_equal(codes[i, :192], c2[0])
        assert np.array_equal(e8[i].astype(int) - 127, k2[0])


def test_shift_invariance_dyadic(orc):
    """Eq. (shifted-x): adding a constant to every score of a row leaves the
    codes unchanged (fp32: except within 1e-4 of a code threshold)."""
    w = inputs.Workload("d", 1, 1, 1, 128, 64, False, "dyadic", 13)
    q, k, v = inputs.dyadic_qkv(w)
    q[..., 0] = 0
    k[..., 0] = 1.0                       # constant channel
    q2 = q.clone()
    q2[0, :, 0, 0] = torch.randint(-2, 3, (128,)).float()   # per-row shift of S by q/8
    a = orc.attn(orc.bf16_bits(q), orc.bf16_bits(k), orc.bf16_bits(v), 1 / 8, False, orc.EFQ,
                 bc=64, dump=True)
    b = orc.attn(orc.bf16_bits(q2), orc.bf16_bits(k), orc.bf16_bits(v), 1 / 8, False, orc.EFQ,
                 bc=64, dump=True)
    assert np.mean(a[1] == b[1]) > 0.999
    assert np.array_equal(a[2], b[2])
    assert np.max(np.abs(a[0] - b[0])) < 0.2


def test_all_zero_codes_give_zero_output(orc):
    """With tau above the block-max residual range [log 3/4, log 3/2) (Eq.
    z-def: z_max = M_b - k_b log 2 - log 6 lies in that range), even the
    block maximum gets (z - tau) h < 0, so code 0 (Eq. d8-index): every code
    of the row is 0, l = 0, and the oracle defines O = 0."""
    w, q, k, v = _tiny(S=128, causal=False, Hq=2, Hkv=1)
    tau = 0.5
    assert tau > math.log(1.5)
    out, codes, e8, m, l = orc.attn(orc.bf16_bits(q), orc.bf16_bits(k), orc.bf16_bits(v), w.scale,
                                    False, orc.EFQ, tau=tau, h=2.3, dump=True)
    assert np.all(codes == 0) and np.all(l == 0.0) and np.all(out == 0.0)


def test_l_positive_and_bounded(orc):
    """Non-negative codes make l >= 0.75 (the row maximum's contribution)."""
    w, q, k, v = _tiny(S=300, causal=True, Hq=2, Hkv=1, dist="qwen", D=128)
    _, _, _, m, l = orc.attn(orc.bf16_bits(q), orc.bf16_bits(k), orc.bf16_bits(v), w.scale, True,
                             orc.EFQ, bc=64, dump=True)
    assert np.all(l >= 0.75)


@pytest.mark.parametrize("dist", ["normal", "qwen"])
def test_rescaling_keeps_tiles_consistent(orc, dist):
    """Eq. (alpha): with correct rescaling, the online result over tiles of
    64 keys stays close to the single-tile result (codes differ only through
    the running maximum), and exp-then-quantize stays close to exact
    softmax; a wrong or missing alpha moves both by several times more."""
    w = inputs.Workload("t", 1, 4, 2, 512, 128, True, dist, 7)
    q, k, v = inputs.make_qkv(w)
    qb, kb, vb = (orc.bf16_bits(t) for t in (q, k, v))
    ex = orc.attn(qb, kb, vb, w.scale, True, orc.EXACT, bc=64)
    rho = lambda a, b: np.linalg.norm(a - b) / np.linalg.norm(b)
    for mode in (orc.EFQ, orc.EXPQ, orc.LUT_MODE):
        o64 = orc.attn(qb, kb, vb, w.scale, True, mode, bc=64)
        o512 = orc.attn(qb, kb, vb, w.scale, True, mode, bc=512)
        assert rho(o64, o512) < 0.12
    assert rho(orc.attn(qb, kb, vb, w.scale, True, orc.EXPQ, bc=64), ex) < 0.25


# ------------------------------------------------ recurrence vs numpy twin
TWIN_CASES = [
    # (batch, seq_q, seq_k, heads_q, heads_kv, head_dim, causal, distribution)
    (1, 200, 200, 4, 2, 64, True, "qwen"),
    (2, 75, 75, 2, 1, 128, False, "normal"),
    (1, 300, 300, 8, 2, 128, True, "qwen"),
    (1, 100, 300, 4, 4, 64, False, "qwen_spread"),
]


@pytest.mark.parametrize("case", TWIN_CASES)
@pytest.mark.parametrize("mode", ["efq", "lut", "expq", "expq6"])
def test_recurrence_matches_numpy_twin(orc, case, mode):
    """Alg. 2 as the C oracle runs it, against the independently written
    numpy recurrence of oracle/twin.py (64-key tiles in ascending order,
    Eq. (alpha) rescaling, the grouped-query head map, V~ from the twin's own
    MXFP4 quantiser, codes from the twin's Alg. 1 or exp-then-quantize):
    codes, E8M0 and final row maxima bit for bit, row sums within 1e-12
    relative, outputs within one fp32 ulp.  Causal and non-causal,
    grouped-query ratios 2 and 4, seq_q < seq_k, ragged tails."""
    from oracle import twin
    Bt, Sq, Sk, Hq, Hkv, D, causal, dist = case
    w = inputs.Workload("tw", Bt, Hq, Hkv, max(Sq, Sk), D, causal, dist, 31 + Sq)
    q, k, v = inputs.make_qkv(w)
    q, k, v = q[:, :Sq].contiguous(), k[:, :Sk].contiguous(), v[:, :Sk].contiguous()
    qb, kb, vb = (orc.bf16_bits(t) for t in (q, k, v))
    om = {"efq": orc.EFQ, "lut": orc.LUT_MODE, "expq": orc.EXPQ, "expq6": orc.EXPQ6}[mode]
    tau, h = orc.LUT if mode == "lut" else orc.MEAN
    o1, c1, e1, m1, l1 = orc.attn(qb, kb, vb, w.scale, causal, om, tau=tau, h=h, bc=64, dump=True)
    o2, c2, e2, m2, l2 = twin.attn_twin(qb, kb, vb, w.scale, causal, mode, tau, h, bc=64)
    assert np.array_equal(c1, c2)
    assert np.array_equal(e1, e2)
    assert np.array_equal(m1, m2)
    assert np.max(np.abs(l1 - l2) / l2) <= 1e-12
    np.testing.assert_array_max_ulp(o1, o2, maxulp=1)


# ------------------------------------------------------------ calibration
def test_calibration_recovers_generating_point(orc):
    """Alg. 3 pinned on a case with a known answer: when the reference
    output is itself the EFQ output at one candidate pair, that pair has
    rho = 0, every other pair on this input has rho > 0, and the search
    returns it wherever it sits in the grid."""
    w, q, k, v = _tiny(S=128, causal=False, Hq=2, Hkv=1)
    qb, kb, vb = orc.bf16_bits(q), orc.bf16_bits(k), orc.bf16_bits(v)
    taus, hs = [-3.5, -3.06, -2.6], [1.9, 2.3, 2.8]
    for tau0, h0 in [(-3.06, 2.3), (-2.6, 1.9), (-3.5, 2.8)]:
        ref = orc.attn(qb, kb, vb, w.scale, False, orc.EFQ, tau=tau0, h=h0)
        best, rho = orc.calibrate(qb, kb, vb, w.scale, False, ref, taus, hs)
        i, j = taus.index(tau0), hs.index(h0)
        assert rho[i, j] == 0.0
        assert np.sum(rho == 0.0) == 1
        assert best == (float(np.float32(tau0)), float(np.float32(h0)))


def test_calibration_objective_and_order(orc):
    """rho is the relative Frobenius error of Sec. III-C and the selection
    keeps the first strict minimum in tau-major order."""
    w, q, k, v = _tiny(S=96, causal=True, Hq=1, Hkv=1)
    qb, kb, vb = orc.bf16_bits(q), orc.bf16_bits(k), orc.bf16_bits(v)
    ref = orc.attn(qb, kb, vb, w.scale, True, orc.EXACT)
    taus, hs = [-3.3, -3.06, -3.06], [2.3, 2.3]      # repeated pairs tie exactly
    best, rho = orc.calibrate(qb, kb, vb, w.scale, True, ref, taus, hs)
    o = orc.attn(qb, kb, vb, w.scale, True, orc.EFQ, tau=-3.06, h=2.3)
    want = np.linalg.norm(o.astype(np.float64) - ref) / np.linalg.norm(ref.astype(np.float64))
    assert abs(rho[1, 0] - want) <= 1e-12 * want
    assert rho[1, 0] == rho[1, 1] == rho[2, 0] == rho[2, 1]
    flat = rho.ravel()
    first = int(np.argmin(flat))                     # first occurrence of the minimum
    assert best == (float(np.float32(taus[first // 2])), float(np.float32(hs[first % 2])))
    assert np.all(rho > 0)


# ------------------------------------------------------- MXFP8 Q / K (low-bit Q K^T)
def _e4m3_bits_torch(y):
    """torch's own float32 -> float8_e4m3fn cast (round to nearest even)."""
    return torch.from_numpy(np.ascontiguousarray(y, np.float32)).to(torch.float8_e4m3fn) \
        .view(torch.uint8).numpy()


def _mxfp8_dequant_torch(codes, e8):
    """Values of MXFP8 codes decoded by torch's float8_e4m3fn type."""
    v = torch.from_numpy(np.ascontiguousarray(codes)).view(torch.float8_e4m3fn).double().numpy()
    return v * np.repeat(2.0 ** (e8.astype(np.float64) - 127), 32, axis=-1)


def test_mxfp8_scale_rule(orc):
    """OCP microscaling for E4M3: the shared exponent is floor(log2 amax)
    minus 8 (the largest E4M3 exponent), written as E8M0 (k + 127); an
    all-zero block takes the smallest scale."""
    rng = np.random.default_rng(20)
    x = (rng.standard_normal((4000, 64)) * 2.0 ** rng.integers(-30, 30, (4000, 1))).astype(np.float32)
    x[5, :32] = 0.0
    xb = orc_bits(torch.from_numpy(x))
    codes, e8 = orc.quant_mxfp8(xb)
    xv = orc.bits_to_f64(xb).reshape(4000, 2, 32)
    amax = np.abs(xv).max(axis=2)
    expo = np.array([[math.frexp(a)[1] - 1 if a > 0 else -119 for a in r] for r in amax])
    want = np.clip(expo - 8, -127, 127) + 127
    want[5, 0] = 0
    assert np.array_equal(e8.astype(np.int64), want)
    assert np.all(codes[5, :32] == 0)


def test_mxfp8_codes_match_torch_cast(orc):
    """Element codes are the round-to-nearest-even E4M3 of x / 2^k, which
    is torch's float8_e4m3fn cast wherever |x| / 2^k <= 464 (torch turns
    larger values into NaN); above that the MX rule saturates to 448
    (code 0x7E with the sign)."""
    rng = np.random.default_rng(21)
    w = inputs.Workload("t", 1, 4, 2, 512, 128, False, "qwen", 21)
    q, k, _ = inputs.make_qkv(w)
    for t in (q, k, torch.from_numpy(rng.standard_normal((300, 96)).astype(np.float32) * 3)):
        xb = orc_bits(t)
        D = xb.shape[-1]
        codes, e8 = orc.quant_mxfp8(xb)
        xv = orc.bits_to_f64(xb).reshape(-1, D)
        sc = np.repeat(2.0 ** (e8.reshape(-1, D // 32).astype(np.float64) - 127), 32, axis=1)
        y = xv / sc
        assert np.all(np.abs(y) < 512)                 # amax / 2^k < 2^9
        ref = _e4m3_bits_torch(y)
        big = np.abs(y) > 464
        got = codes.reshape(-1, D)
        assert np.array_equal(got[~big], ref[~big])
        assert np.all((got[big] & 0x7F) == 0x7E)
        assert np.array_equal(got[big] >> 7, (y[big] < 0).astype(np.uint8))


def test_mxfp8_grid_round_trip_ties_and_saturation(orc):
    """Every finite E4M3 value times a power of two comes back unchanged in
    a block whose maximum is 448 * 2^j; midpoints go to the even mantissa;
    460 saturates to 448 and 2^-10 (half the smallest subnormal) to zero."""
    mags = np.array([torch.tensor([c], dtype=torch.uint8).view(torch.float8_e4m3fn).double().item()
                     for c in range(0x7F)])
    vals = np.concatenate([mags, -mags[1:]])           # 253 codes
    rows = []
    for j in (-12, 0, 7):
        for s in range(0, len(vals), 31):
            blk = np.zeros(32)
            blk[0] = 448.0
            part = vals[s:s + 31]
            blk[1:1 + len(part)] = part
            rows.append(blk * 2.0 ** j)
    x = np.array(rows)
    codes, e8 = orc.quant_mxfp8(orc_bits(torch.from_numpy(x)))
    back = _mxfp8_dequant_torch(codes, e8)
    assert np.array_equal(back, x)
    # ties and saturation in a block with k = 0
    blk = np.zeros((1, 32))
    blk[0, :7] = [448.0, 1.0625, 1.1875, 460.0, -460.0, 2.0 ** -10, 3 * 2.0 ** -11]
    codes, e8 = orc.quant_mxfp8(orc_bits(torch.from_numpy(blk)))
    assert e8[0, 0] == 127
    assert list(codes[0, :7]) == [0x7E, 0x38, 0x3A, 0x7E, 0xFE, 0x00, 0x01]


def test_lowbit_attention_is_attention_on_mxfp8_values(orc):
    """With qk8 set, the recurrence runs on the MXFP8 values of Q and K:
    the same output as the plain path on those values (decoded by torch and
    exactly representable in bf16), for every P mode; and inputs already on
    the MXFP8 grid are left unchanged by it."""
    w, q, k, v = _tiny(S=160, D=64, Hq=4, Hkv=2, dist="qwen", causal=True)
    qb, kb, vb = orc.bf16_bits(q), orc.bf16_bits(k), orc.bf16_bits(v)
    deq = []
    for xb in (qb, kb):
        c, e = orc.quant_mxfp8(xb)
        d = _mxfp8_dequant_torch(c, e)
        db = orc_bits(torch.from_numpy(d))
        assert np.array_equal(orc.bits_to_f64(db), d)      # exact in bf16
        deq.append(db)
    for mode in (orc.EFQ, orc.EXPQ, orc.EXACT):
        a = orc.attn(qb, kb, vb, w.scale, True, mode, bc=64, qk8=True)
        b = orc.attn(deq[0], deq[1], vb, w.scale, True, mode, bc=64)
        c = orc.attn(deq[0], deq[1], vb, w.scale, True, mode, bc=64, qk8=True)
        assert np.array_equal(a, b) and np.array_equal(b, c)
    # and it is a different (lower precision) computation from the bf16 path
    assert not np.array_equal(orc.attn(qb, kb, vb, w.scale, True, orc.EXACT, bc=64),
                              orc.attn(qb, kb, vb, w.scale, True, orc.EXACT, bc=64, qk8=True))
