"""GPU path vs the CPU oracle (run on an MI355X; every call goes through the C ABI).

Bar: bit-exact E2M1 codes and E8M0 scales where the scores are bit-identical
(the P-gen unit, and the fused kernel on exact-score inputs), attention
output within 2e-3 max abs of the oracle's fp32 output.
"""
import ctypes
import math

import numpy as np
import pytest
import torch

from paper_2609_09721_amd import inputs

from adversarial import adversarial_scores

pytestmark = pytest.mark.gpu

TOL = 2e-3
LN2 = math.log(2.0)


@pytest.fixture(scope="module")
def B():
    from paper_2609_09721_amd import binding
    binding.lib()
    assert torch.cuda.is_available(), "no GPU"
    return binding


def unpack(codes_u8: np.ndarray) -> np.ndarray:
    c = codes_u8.astype(np.uint8)
    return np.stack([c & 0xF, c >> 4], axis=-1).reshape(*c.shape[:-1], -1)


@pytest.mark.parametrize("kind,params", [("efq", (-3.06, 2.30)), ("efq", (-2.90, 2.00)),
                                         ("efq", (-2.10, 2.70)), ("lut", None)])
def test_pgen_bitexact(B, orc, kind, params):
    rng = np.random.default_rng(1)
    mode = orc.LUT_MODE if kind == "lut" else orc.EFQ
    tau, h = orc.LUT if kind == "lut" else params
    for rows, cols in [(96, 200), (37, 64), (5, 1000), (64, 31)]:
        x = adversarial_scores(rng, rows, cols, tau, h)
        cg, eg = B.pgen(torch.from_numpy(x).cuda(), kind, (tau, h))
        cg = unpack(cg.cpu().numpy())[:, :cols]
        co, eo = orc.pgen(x, mode, tau, h)
        assert np.array_equal(eg.cpu().numpy(), eo), (rows, cols)
        assert np.array_equal(cg, co), (rows, cols, np.argwhere(cg != co)[:5])


def test_pgen_random_bitexact(B, orc):
    """1e8 random shifted scores in six chunks of 2^24 (block maxima from 0
    down to the E8M0 floor, zeros, masked keys), bit-exact."""
    rng = np.random.default_rng(2)
    for chunk, spread in enumerate([0.5, 1.0, 3.0, 8.0, 30.0, 120.0]):
        x = -rng.exponential(spread, size=(32768, 512)).astype(np.float32)
        x[:, ::97] = 0.0
        if chunk % 2:
            x[rng.random(x.shape) < 0.05] = -np.inf
        cg, eg = B.pgen(torch.from_numpy(x).cuda(), "efq")
        co, eo = orc.pgen(x)
        assert np.array_equal(eg.cpu().numpy(), eo), chunk
        assert np.array_equal(unpack(cg.cpu().numpy()), co), chunk


@pytest.mark.parametrize("kind", ["expq", "expq6"])
def test_pgen_expq_close(B, orc, kind):
    """Exp-then-quantize (OCP and scale6 rules): the GPU's exp is not
    correctly rounded, so codes and scales may differ at rounding
    midpoints and scale boundaries only."""
    rng = np.random.default_rng(3)
    x = -rng.exponential(3.0, size=(2048, 256)).astype(np.float32)
    x[:, ::32] = np.minimum(x[:, ::32], -1e-3)
    x[7, :32] = 0.0                       # row maximum p = 1 in a block
    cg, eg = B.pgen(torch.from_numpy(x).cuda(), kind)
    co, eo = orc.pgen(x, orc.EXPQ if kind == "expq" else orc.EXPQ6)
    cg = unpack(cg.cpu().numpy())
    assert np.mean(eg.cpu().numpy() == eo) > 0.9999
    assert np.mean(cg == co) > 0.9999


@pytest.mark.parametrize("S,H,D", [(75, 3, 128), (256, 1, 64), (200, 2, 128)])
def test_vquant_bitexact(B, orc, S, H, D):
    g = torch.Generator().manual_seed(S + D)
    v = torch.randn(2, S, H, D, generator=g) * torch.exp2(torch.randint(-30, 30, (1, 1, H, D), generator=g).float())
    v[0, :5, 0, :3] = 0.0
    v[1, :, H - 1, 5] = 0.0
    v[1, 7, 0, 0] = -1e-39
    v[0, 1, 0, 1] = -0.0
    vb = v.to(torch.bfloat16)
    vh = B.quant_v(vb.cuda())
    sh = B.Shape(2, 1, S, H, H, D)
    cg, eg = B.vhat_natural(vh, sh)
    co, eo = orc.quant_v(orc.bf16_bits(vb))
    nblk = (S + 31) // 32
    assert np.array_equal(eg[:, :, :nblk].cpu().numpy(), eo)
    assert np.array_equal(cg[:, :, :nblk * 32].cpu().numpy(), co)
    # padding blocks are zero
    assert int(cg[:, :, nblk * 32:].abs().sum()) == 0
    assert int(eg[:, :, nblk:].sum()) == 0


def _bf16_next(x: float, up: bool) -> float:
    """The bf16 neighbour of a bf16-representable positive x."""
    b = torch.tensor([x], dtype=torch.bfloat16).view(torch.int16)
    return float((b + (1 if up else -1)).view(torch.bfloat16).float())


def test_vquant_ties(B, orc):
    """Exact E2M1 midpoints of v 2^-k, their bf16 neighbours on both sides,
    the grid points and the saturation region, with both signs and block
    scales 2^-20 .. 2^20: the codes (ties to the even code) and scales equal
    the oracle's."""
    mids = [0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0]
    vals0 = []
    for m in mids:
        vals0 += [m, _bf16_next(m, True), _bf16_next(m, False)]
    vals0 += [0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 0.0, 0.125, 0.0625, 0.375]
    vals0 = vals0[:31] + [6.0]                       # block maximum 6: k = e
    vals1 = [5.0, 5.5, 5.75, 6.0, 6.5, 7.0, 4.0, 4.5, 3.0, 2.5, 0.25] * 3
    vals1 = vals1[:31] + [7.5]                       # maximum 7.5: k = e, codes saturate
    S, H, D = 64, 2, 64
    v = torch.zeros(1, S, H, D)
    for h in range(H):
        for d in range(D):
            e = (d + 29 * h) % 41 - 20
            sgn = torch.tensor([1.0 if ((t * 7 + d + h) % 3) else -1.0 for t in range(32)])
            v[0, :32, h, d] = torch.tensor(vals0) * sgn * 2.0 ** e
            v[0, 32:, h, d] = torch.tensor(vals1) * sgn.flip(0) * 2.0 ** e
    vb = v.to(torch.bfloat16)
    assert torch.equal(vb.float(), v)              # every value is exact in bf16
    vh = B.quant_v(vb.cuda())
    cg, eg = B.vhat_natural(vh, B.Shape(1, 1, S, H, H, D))
    co, eo = orc.quant_v(orc.bf16_bits(vb))
    assert np.array_equal(eg[:, :, :2].cpu().numpy(), eo)
    assert np.array_equal(cg[:, :, :64].cpu().numpy(), co)


CASES = [
    # (batch, seq_q, seq_k, heads_q, heads_kv, head_dim, causal)
    (1, 256, 256, 2, 1, 64, False),
    (1, 200, 200, 4, 2, 128, True),
    (2, 75, 75, 2, 1, 128, False),
    (1, 100, 300, 2, 2, 64, False),
    (1, 333, 333, 1, 1, 128, True),
]

# Degenerate and boundary shapes: one key, one query, a partial first MX
# block, exactly one tile and one key past it, one query past a 256-query
# workgroup, grouped-query ratio 8 with seq_q < seq_k, seq_k < 32.
EDGE = [
    (1, 1, 1, 1, 1, 64, True),
    (1, 1, 1, 2, 1, 128, False),
    (1, 33, 33, 2, 2, 64, True),
    (1, 64, 64, 1, 1, 128, True),
    (1, 65, 65, 1, 1, 128, True),
    (1, 257, 257, 1, 1, 64, True),
    (1, 7, 40, 8, 1, 64, False),
    (3, 40, 5, 2, 1, 128, False),
]


# Deep shapes: in the first three each wave streams 18-24 key tiles, so
# every slot of the K ring (6 tiles) and the V~ ring (7 tiles) is refilled
# several times under the four-tiles-ahead schedule: causal with
# grouped-query ratio 4, a ragged tail past 23 full tiles, and seq_q < seq_k
# over 21 tiles.  The last runs two batches causal with a ragged tail past
# 8 tiles under the XCD-grouped work order (24 work items, a multiple of
# the 8 XCDs).
DEEP = [
    (1, 1100, 1100, 8, 2, 128, True),
    (1, 64, 1500, 4, 1, 64, False),
    (1, 300, 1300, 2, 2, 128, False),
    (2, 520, 520, 4, 2, 128, True),
]


@pytest.mark.parametrize("case", CASES + EDGE + DEEP)
@pytest.mark.parametrize("kind", ["efq", "lut"])
def test_attn_dump_exact_scores(B, orc, case, kind):
    """Exact-score inputs: every Q.K partial sum is exact, so the fused
    kernel and the oracle see identical scores; codes and scales must match
    bit for bit, the output within tolerance."""
    Bt, Sq, Sk, Hq, Hkv, D, causal = case
    print(f"[parity] dump {case} {kind}", flush=True)
    w = inputs.Workload("d", Bt, Hq, Hkv, max(Sq, Sk), D, causal, "dyadic", 11 + Sq)
    q, k, v = inputs.dyadic_qkv(w)
    q, k, v = q[:, :Sq].contiguous(), k[:, :Sk].contiguous(), v[:, :Sk].contiguous()
    mode = orc.LUT_MODE if kind == "lut" else orc.EFQ
    vh = B.quant_v(v.cuda(), seq_q=Sq, heads_q=Hq)
    out, codes, e8, rm, rl = B.attn_fwd_dump(q.cuda(), k.cuda(), vh, w.scale, causal, kind)
    oo, co, eo, mo, lo = orc.attn(orc.bf16_bits(q), orc.bf16_bits(k), orc.bf16_bits(v), w.scale,
                                  causal, mode, bc=64, dump=True)
    nblk = (Sk + 31) // 32
    cg = unpack(codes.cpu().numpy()).reshape(-1, nblk * 32)
    assert np.array_equal(e8.cpu().numpy().reshape(-1, nblk), eo)
    assert np.array_equal(cg, co)
    assert np.array_equal(rm.cpu().numpy().ravel(), mo)
    assert np.allclose(rl.cpu().numpy().ravel(), lo, rtol=1e-5)
    og = out.cpu().numpy().transpose(0, 2, 1, 3).reshape(-1, D)
    assert np.max(np.abs(og - oo)) <= TOL


@pytest.mark.parametrize("case", CASES[:3])
@pytest.mark.parametrize("kind", ["expq", "expq6"])
def test_attn_expq_exact_scores(B, orc, case, kind):
    Bt, Sq, Sk, Hq, Hkv, D, causal = case
    w = inputs.Workload("d", Bt, Hq, Hkv, max(Sq, Sk), D, causal, "dyadic", 21 + Sq)
    q, k, v = inputs.dyadic_qkv(w)
    vh = B.quant_v(v.cuda(), seq_q=Sq, heads_q=Hq)
    out, codes, e8, rm, rl = B.attn_fwd_dump(q.cuda(), k.cuda(), vh, w.scale, causal, kind)
    mode = orc.EXPQ if kind == "expq" else orc.EXPQ6
    oo, co, eo, mo, lo = orc.attn(orc.bf16_bits(q), orc.bf16_bits(k), orc.bf16_bits(v), w.scale,
                                  causal, mode, bc=64, dump=True)
    nblk = (Sk + 31) // 32
    cg = unpack(codes.cpu().numpy()).reshape(-1, nblk * 32)
    assert np.mean(cg == co) > 1 - 1e-4
    og = out.cpu().numpy().transpose(0, 2, 1, 3).reshape(-1, D)
    assert np.max(np.abs(og - oo)) <= TOL


def test_single_key_returns_its_value(B):
    """Causal row 0 sees one key: p~ is the top code of the row maximum's
    block and O_0 is that key's quantised value row."""
    g = torch.Generator().manual_seed(5)
    for D in (64, 128):
        q = torch.randn(1, 1, 2, D, generator=g).to(torch.bfloat16)
        k = torch.randn(1, 1, 1, D, generator=g).to(torch.bfloat16)
        v = torch.randn(1, 1, 1, D, generator=g).to(torch.bfloat16)
        for kind in ("efq", "lut", "expq", "expq6"):
            out = B.attn_fwd(q.cuda(), k.cuda(), v.cuda(), D ** -0.5, True, kind)
            vh = B.quant_v(v.cuda(), seq_q=1, heads_q=2)
            cg, eg = B.vhat_natural(vh, B.Shape(1, 1, 1, 2, 1, D))
            # dequantise key 0 of every column: E2M1 magnitude times 2^(E8M0 - 127)
            mag = torch.tensor([0, 0.5, 1, 1.5, 2, 3, 4, 6], dtype=torch.float64)
            c = cg[0, 0, 0, :].cpu().long()
            sign = torch.where((c & 8) > 0, -1.0, 1.0).double()
            ref = (mag[c & 7] * sign * torch.exp2(eg[0, 0, 0, :].cpu().double() - 127)).float()
            for h in range(2):
                err = (out[0, 0, h].cpu() - ref).abs().max().item()
                assert err <= 1e-6 * max(1.0, ref.abs().max().item()), (D, kind, h, err)


def test_all_zero_codes_give_zero_output(B, orc):
    """tau above the block-max residual range [log 3/4, log 3/2) maps every
    score, the block maxima included, to code 0 (Eq. d8-index), so l = 0:
    the oracle defines O = 0 for such a row and the kernel must write 0, not
    0 * inf."""
    w = inputs.WORKLOADS["tiny"]
    q, k, v = inputs.make_qkv(w)
    out = B.attn_fwd(q.cuda(), k.cuda(), v.cuda(), w.scale, False, "efq", (0.5, 2.3))
    oo = orc.attn(orc.bf16_bits(q), orc.bf16_bits(k), orc.bf16_bits(v), w.scale, False, orc.EFQ,
                  tau=0.5, h=2.3)
    assert np.all(oo == 0.0)
    assert bool(torch.isfinite(out).all()) and float(out.abs().max()) == 0.0


def test_tiny_config_all_rows(B, orc):
    """The tiny workload (1 x 256 x 64, N(0,1)), every row."""
    w = inputs.WORKLOADS["tiny"]
    q, k, v = inputs.make_qkv(w)
    for kind, mode in [("efq", orc.EFQ), ("expq", orc.EXPQ), ("lut", orc.LUT_MODE),
                       ("expq6", orc.EXPQ6)]:
        out = B.attn_fwd(q.cuda(), k.cuda(), v.cuda(), w.scale, w.causal, kind)
        oo = orc.attn(orc.bf16_bits(q), orc.bf16_bits(k), orc.bf16_bits(v), w.scale, w.causal, mode)
        og = out.cpu().numpy().transpose(0, 2, 1, 3).reshape(-1, w.head_dim)
        err = np.abs(og - oo).max(axis=1)
        assert np.max(err) <= TOL, (kind, np.sort(err)[-5:])


def test_entry_points_match_ex(B):
    w = inputs.WORKLOADS["tiny"]
    q, k, v = (t.cuda() for t in inputs.make_qkv(w))
    a = B.efq_attn_fwd(q, k, v, w.scale, False)
    b = B.attn_fwd(q, k, v, w.scale, False, "efq")
    c = B.efq_attn_fwd_expq(q, k, v, w.scale, False)
    d = B.attn_fwd(q, k, v, w.scale, False, "expq")
    assert torch.equal(a, b) and torch.equal(c, d)


def test_same_operand_v_constant(B):
    """V = 1 makes O = 1: P~V and P~1 share one operand (Sec. III-A)."""
    w = inputs.Workload("c", 1, 4, 2, 1000, 128, True, "qwen", 5)
    q, k, v = inputs.make_qkv(w)
    for c in (1.0, -3.0):
        vc = torch.full_like(v, c)
        for kind in ("efq", "expq", "lut", "expq6"):
            out = B.attn_fwd(q.cuda(), k.cuda(), vc.cuda(), w.scale, True, kind)
            assert float((out - c).abs().max()) <= 1e-6 * abs(c) * 8


def _bshd(rows_out, Bt, Hq, S, D):
    """Oracle rows in (b, hq, i) order -> fp32 BSHD tensor."""
    return torch.from_numpy(rows_out.reshape(Bt, Hq, S, D).transpose(0, 2, 1, 3).copy())


def test_calibrate_matches_oracle(B, orc):
    """Alg. 3 on the GPU against the oracle's Alg. 3, on exact-score inputs
    with the exact-softmax reference: same objective grid (within fp32
    accumulation order), and the selected pair is a minimiser of the
    oracle's grid."""
    w = inputs.Workload("cal", 1, 2, 1, 256, 64, False, "dyadic", 77)
    q, k, v = inputs.dyadic_qkv(w)
    qb, kb, vb = orc.bf16_bits(q), orc.bf16_bits(k), orc.bf16_bits(v)
    ref = orc.attn(qb, kb, vb, w.scale, False, orc.EXACT)
    o_ref = _bshd(ref, 1, 2, 256, 64).cuda()
    taus, hs = [-3.5, -3.06, -2.6, -2.1], [1.9, 2.3, 2.8]
    (tg, hg), rho_g = B.calibrate(q.cuda(), k.cuda(), v.cuda(), o_ref, taus, hs, w.scale, False)
    (to, ho), rho_o = orc.calibrate(qb, kb, vb, w.scale, False, ref, taus, hs)
    assert np.allclose(rho_g, rho_o, rtol=1e-4, atol=0)
    i = [float(np.float32(t)) for t in taus].index(tg)
    j = [float(np.float32(x)) for x in hs].index(hg)
    assert rho_o[i, j] <= rho_o.min() * (1 + 1e-4)


def test_calibrate_recovers_generating_point(B):
    """With the GPU's own EFQ output at one candidate as the reference, that
    candidate has rho = 0 (the same kernel on the same inputs) and is
    selected."""
    w = inputs.WORKLOADS["tiny"]
    q, k, v = (t.cuda() for t in inputs.make_qkv(w))
    taus, hs = [-3.5, -3.06, -2.6], [1.9, 2.3, 2.8]
    o_ref = B.attn_fwd(q, k, v, w.scale, False, "efq", (-2.6, 1.9))
    (tg, hg), rho = B.calibrate(q, k, v, o_ref, taus, hs, w.scale, False)
    assert (tg, hg) == (float(np.float32(-2.6)), float(np.float32(1.9)))
    assert rho[2, 0] == 0.0 and np.sum(rho == 0.0) == 1



def test_clock_probe(B):
    """The diagnostic shader-clock probe: per workgroup the s_memtime ticks
    (shader clock) and the s_memrealtime ticks (100 MHz) of an MFMA stream.
    One workgroup of four waves per CU puts one wave on each SIMD, whose 16
    bf16 32x32x16 MFMAs per iteration take at least 32 shader cycles each;
    the real-time span lies inside the event-timed launch, and the clock the
    two give is a plausible MI355X shader clock."""
    blocks, iters = 64, 2000
    st = torch.cuda.current_stream()
    B.clock_probe(blocks, 10)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(st)
    t = B.clock_probe(blocks, iters)
    e1.record(st)
    torch.cuda.synchronize()
    a = t.cpu().numpy().astype(np.float64)
    assert (a > 0).all()
    assert (a[:, 0] >= iters * 16 * 31).all(), a[:, 0].min()
    assert a[:, 1].max() * 1e-5 <= e0.elapsed_time(e1) * 1.02 + 0.01
    ghz = 0.1 * a[:, 0] / a[:, 1]
    assert ((ghz > 0.5) & (ghz < 3.0)).all(), ghz


def test_stamped_build_matches_product(B):
    """The phase-stamp diagnostic build (the bench's in-kernel clock and the
    phase profile come from it) computes what the product build computes:
    outputs bit-identical on a causal GQA shape of many tiles and a ragged
    tail, for EFQ and the no-op stage; its clock pairs give a plausible
    shader clock, and every workgroup it stamps records its first phases."""
    from paper_2609_09721_amd import build as hip_build, phases
    if not __import__("os").path.exists(hip_build.STAMPS_LIB):
        pytest.skip("stamped build not built")
    w = inputs.Workload("stamp", 1, 8, 2, 1100, 128, True, "normal", 4242)
    q, k, v = inputs.make_qkv(w, device="cuda")
    vh = B.quant_v(v, seq_q=w.seq, heads_q=w.heads_q)
    ref = {kind: B.attn_fwd_vhat(q, k, vh, w.scale, True, kind) for kind in ("efq", "noop")}
    torch.cuda.synchronize()
    out = torch.empty_like(ref["efq"])
    clk = phases.kernel_sclk(w, q, k, vh, out, "efq", warm=1, reps=2)
    assert torch.equal(out, ref["efq"])
    assert 0.5 < clk < 3.0, clk
    saved = (B._lib, B.LIB_PATH)
    L = None
    try:
        L = phases._load()
        buf = torch.zeros(phases.NBLK * 2 * phases.SLOTS, dtype=torch.int64, device="cuda")
        assert L.efq_phase_stamps_set(ctypes.c_void_p(buf.data_ptr())) == 0
        B.attn_fwd_vhat(q, k, vh, w.scale, True, "noop", out=out)
        torch.cuda.synchronize()
        assert torch.equal(out, ref["noop"])
    finally:
        if L is not None:
            torch.cuda.synchronize()
            L.efq_phase_stamps_set(None)
        B._lib, B.LIB_PATH = saved
    B.lib()
    # 1100 queries of 8 heads: 40 workgroups of 256 queries (five per head).
    # Every stamping wave stamps its first phase and its clock pairs; the
    # stamps it takes only grow, the phases it does not reach read 0, and
    # workgroups past the grid leave their rows untouched.
    x = buf.cpu().numpy().reshape(phases.NBLK, 2, phases.SLOTS)
    nwg = 8 * ((w.seq + 255) // 256)
    assert (x[nwg:] == 0).all()
    t = x[:nwg, :, :2 * phases.NPH].reshape(nwg * 2, -1)
    assert (t[:, :2] > 0).all() and (x[:nwg, :, 2 * phases.NPH:] > 0).all()
    for row in t:
        n = int((row > 0).sum())
        assert (row[:n] > 0).all() and (row[n:] == 0).all() and (np.diff(row[:n]) >= 0).all()
