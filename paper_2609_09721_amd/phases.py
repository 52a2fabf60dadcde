"""Phase-stamp view of the fused attention kernel: in-kernel timer stamps
that time the probability stage inside the fused kernel.

usage: python3 -m paper_2609_09721_amd.phases [--workload qwen3_8b_32k] [--out FILE]

Loads the diagnostic build libefq_attn_stamps.so (the same kernel source
with EFQ_PHASE_STAMPS=1; build it beforehand with
paper_2609_09721_amd.build.build_stamps) and runs the fused kernel on one
workload for the EFQ, exp-then-quantize, EFQ-LUT and no-op stages.  The two
waves of SIMD 0 in each of the first 256 workgroups stamp the end of every
phase (work done, then wait and barrier done), which gives per phase:

  work  from the previous phase's end to this phase's work end
  wait  this phase's wait on its loads and, every fourth phase, the barrier

A matrix phase M(j) holds the Q K^T MFMAs of tile j and the code step of
tile j-1; a VALU phase V(j) the mask, maxima, parameters and rescale of
tile j (the P~V MFMAs may sit in either, where the compiler put them).  Per
tile a wave runs one of each, so the stage's own time per tile is
(M + V)(stage) - (M + V)(no-op), medians over the steady-state phases, and
the speedup 1 - t_EFQ / t_EXPQ (the paper's Table VIII definition).

Reading the counter makes a wave wait for its outstanding LDS and scalar
memory operations, so the stamped kernel is slower than the product build;
the summary records both kernel times.  Ticks are s_memtime units (shader
clock cycles); each wave also records s_memrealtime (100 MHz) beside its
first and last stamps, which gives the shader clock during the kernel.
"""
from __future__ import annotations

import argparse
import ctypes
import os
import sys

import numpy as np
import torch

from . import binding, build, inputs

NBLK, NPH = 256, 512          # workgroups and phases stamped (kStampBlocks, kStampPhases)
SLOTS = 2 * NPH + 4           # per wave: two stamps per phase, then the two clock pairs
SKIP = 8                      # leading phases left out (prologue)
KINDS = ("efq", "expq", "lut", "noop")


def _load():
    if not os.path.exists(build.STAMPS_LIB):
        raise RuntimeError(f"{build.STAMPS_LIB} is missing: run build.build_stamps() first")
    binding._lib = None
    binding.LIB_PATH = build.STAMPS_LIB
    L = binding.lib()
    L.efq_phase_stamps_set.argtypes = [ctypes.c_void_p]
    L.efq_phase_stamps_set.restype = ctypes.c_int
    return L


def _time(fn, n=5):
    for _ in range(2):
        fn()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    st = torch.cuda.current_stream()
    for a, b in ev:
        a.record(st)
        fn()
        b.record(st)
    torch.cuda.synchronize()
    return float(np.median([a.elapsed_time(b) for a, b in ev]))


def phase_stats(t: np.ndarray) -> dict:
    """t: [blocks, 2 groups, phases, 2] stamps.  Group g runs M(j) in phase
    2j + g and V(j) in phase 2j + 1 + g."""
    work = {"M": [], "V": []}
    wait = {"M": [], "V": []}
    for g in (0, 1):
        x = t[:, g]
        for p in range(SKIP, NPH - 2):
            ok = (x[:, p - 1, 1] > 0) & (x[:, p, 0] > 0) & (x[:, p, 1] > 0)
            kind = "M" if (p - g) % 2 == 0 else "V"
            work[kind].append((x[ok, p, 0] - x[ok, p - 1, 1]))
            wait[kind].append((x[ok, p, 1] - x[ok, p, 0]))
    out = {}
    for k in ("M", "V"):
        w = np.concatenate(work[k]).astype(np.float64)
        z = np.concatenate(wait[k]).astype(np.float64)
        out[k] = {"n": int(w.size), "median": float(np.median(w)), "mean": float(w.mean()),
                  "p90": float(np.percentile(w, 90)), "wait_median": float(np.median(z)),
                  "wait_mean": float(z.mean())}
    return out


def overlap(t: np.ndarray, grid: int = 4) -> tuple:
    """Fraction of the stamped time in which at least one of the SIMD's two
    waves, and in which both, are doing matrix-phase work (steady state of
    each workgroup, sampled every `grid` ticks)."""
    one = both = total = 0
    for blk in range(t.shape[0]):
        x = t[blk]
        if (x[:, SKIP - 1:NPH - 1] == 0).any():
            continue
        lo = max(x[0, SKIP, 1], x[1, SKIP, 1])
        hi = min(x[0, NPH - 2, 0], x[1, NPH - 2, 0])
        if hi <= lo:
            continue
        g = np.arange(lo, hi, grid)
        in_m = np.zeros((2, g.size), bool)
        for grp in (0, 1):
            for p in range(1, NPH - 1):
                if (p - grp) % 2 == 0:
                    i0, i1 = np.searchsorted(g, x[grp, p - 1, 1]), np.searchsorted(g, x[grp, p, 0])
                    in_m[grp, i0:i1] = True
        one += int((in_m[0] | in_m[1]).sum())
        both += int((in_m[0] & in_m[1]).sum())
        total += g.size
    return (one / total, both / total) if total else (0.0, 0.0)


def sclk_ghz(clk: np.ndarray) -> float:
    """clk: [blocks, 2 groups, 4] = (s_memtime, s_memrealtime) at the end of
    a wave's first and of its last stamped phase; the median over waves of
    the shader clock in GHz (s_memrealtime counts at 100 MHz)."""
    c = clk.reshape(-1, 4).astype(np.float64)
    dt, dr = c[:, 2] - c[:, 0], c[:, 3] - c[:, 1]
    ok = (dr > 0) & (dt > 0)
    return float(np.median(0.1 * dt[ok] / dr[ok])) if ok.any() else 0.0


def kernel_sclk(w, q, k, vhat, out, kind: str = "efq", warm: int = 3, reps: int = 5) -> float:
    """Shader clock (GHz) during the stamped build of the fused kernel on the
    given inputs (a V~ from efq_quant_v_mxfp4 and an output buffer): `warm`
    launches, then `reps` stamped ones back to back; the median of their
    clocks.  The library binding.lib() returned before is restored after."""
    saved = (binding._lib, binding.LIB_PATH)
    L = None
    try:
        L = _load()
        # no stamp buffer from an earlier call may still be set
        assert L.efq_phase_stamps_set(None) == 0
        bufs = [torch.zeros(NBLK * 2 * SLOTS, dtype=torch.int64, device=q.device)
                for _ in range(reps)]
        for _ in range(warm):
            binding.attn_fwd_vhat(q, k, vhat, w.scale, w.causal, kind, out=out)
        for buf in bufs:
            # the pointer is set by a blocking copy, after the launches before it
            assert L.efq_phase_stamps_set(ctypes.c_void_p(buf.data_ptr())) == 0
            binding.attn_fwd_vhat(q, k, vhat, w.scale, w.causal, kind, out=out)
        torch.cuda.synchronize()
        assert L.efq_phase_stamps_set(None) == 0
        clk = [sclk_ghz(b.cpu().numpy().reshape(NBLK, 2, SLOTS)[:, :, 2 * NPH:]) for b in bufs]
        return float(np.median(clk))
    finally:
        if L is not None:
            torch.cuda.synchronize()
            L.efq_phase_stamps_set(None)
        binding._lib, binding.LIB_PATH = saved


def measure(workload: str):
    L = _load()
    try:
        return _measure(L, workload)
    finally:
        torch.cuda.synchronize()
        L.efq_phase_stamps_set(None)


def _measure(L, workload: str):
    w = inputs.WORKLOADS[workload]
    dev = torch.device("cuda:0")
    q, k, v = inputs.make_qkv(w, device=dev)
    vh = binding.quant_v(v, seq_q=w.seq, heads_q=w.heads_q)
    out = torch.empty(q.shape, dtype=torch.float32, device=dev)
    buf = torch.zeros(NBLK * 2 * SLOTS, dtype=torch.int64, device=dev)
    res = {}
    for kind in KINDS:
        print(f"[phases] {workload} {kind}", flush=True)
        assert L.efq_phase_stamps_set(None) == 0
        fn = lambda: binding.attn_fwd_vhat(q, k, vh, w.scale, w.causal, kind, out=out)
        ms = _time(fn)
        buf.zero_()
        assert L.efq_phase_stamps_set(ctypes.c_void_p(buf.data_ptr())) == 0
        fn()
        torch.cuda.synchronize()
        assert L.efq_phase_stamps_set(None) == 0
        x = buf.cpu().numpy().reshape(NBLK, 2, SLOTS)
        t = x[:, :, :2 * NPH].reshape(NBLK, 2, NPH, 2)
        res[kind] = {"ms": ms, **phase_stats(t)}
        res[kind]["m_any"], res[kind]["m_both"] = overlap(t)
        res[kind]["sclk"] = sclk_ghz(x[:, :, 2 * NPH:])
    return res


def summarize(res: dict, workload: str, command: str, kernel_hash: str) -> str:
    lines = [
        "# phase stamps of the fused attention kernel (diagnostic build with EFQ_PHASE_STAMPS=1), "
        f"{workload}, bf16 Q K^T",
        "# command (from the repository root, after paper_2609_09721_amd.build.build_stamps()):",
        f"#   {command}",
        "# two waves of SIMD 0 in each of the first 256 workgroups, phases "
        f"{SKIP}..{NPH - 3} of each wave; ticks = s_memtime units",
        "# work: previous phase end -> this phase's work end; wait: load wait and barrier",
        "# stage per tile = median(M work) + median(V work) - the same for the no-op stage; "
        "speedup = 1 - stage(EFQ) / stage(exp-then-quantize)",
        "# M any / M both: share of the stamped time in which at least one / both of a SIMD's two "
        "waves do matrix-phase work",
        "# SCLK: shader clock during the stamped kernel, s_memtime ticks over s_memrealtime "
        "(100 MHz) between a wave's first and last stamped phase ends, median over waves",
        "# stage | stamped kernel ms | M work median | M work mean | M work p90 | M wait median | "
        "V work median | V work mean | V work p90 | V wait median | stage ticks per tile | "
        "M any | M both | SCLK GHz",
    ]
    base = res["noop"]["M"]["median"] + res["noop"]["V"]["median"]
    stage = {}
    for kind in KINDS:
        r = res[kind]
        stage[kind] = r["M"]["median"] + r["V"]["median"] - base
        lines.append(
            f"{kind} | {r['ms']:.3f} | {r['M']['median']:.0f} | {r['M']['mean']:.0f} | "
            f"{r['M']['p90']:.0f} | {r['M']['wait_median']:.0f} | {r['V']['median']:.0f} | "
            f"{r['V']['mean']:.0f} | {r['V']['p90']:.0f} | {r['V']['wait_median']:.0f} | "
            f"{stage[kind]:.0f} | {r.get('m_any', 0.0):.3f} | {r.get('m_both', 0.0):.3f} | "
            f"{r.get('sclk', 0.0):.3f}")
    for kind in ("efq", "expq", "lut"):
        lines.append(f"stamps_stage_ticks_{kind} = {stage[kind]:.0f}")
    if stage["expq"] > 0:
        lines.append(f"stamps_speedup = {1.0 - stage['efq'] / stage['expq']:.4f}")
    if res["efq"].get("sclk", 0.0) > 0:
        lines.append(f"stamps_sclk_ghz = {res['efq']['sclk']:.3f}")
    lines.append(f"kernel_hash = {kernel_hash}")
    return "\n".join(lines) + "\n"


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="qwen3_8b_32k")
    ap.add_argument("--out", default=None)
    a = ap.parse_args(argv)
    assert torch.cuda.is_available(), "the phase stamps need a GPU"
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    sys.path.insert(0, root)
    import bench
    res = measure(a.workload)
    cmd = f"python3 -m paper_2609_09721_amd.phases --workload {a.workload} --out <FILE>"
    text = summarize(res, a.workload, cmd, bench.kernel_hash())
    if a.out:
        with open(a.out, "w") as f:
            f.write(text)
    print(text, end="")


if __name__ == "__main__":
    main()
