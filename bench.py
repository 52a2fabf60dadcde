"""Benchmark: EFQ-Softmax attention forward on one MI355X.

One step = the whole hot path on one batch of synthetic input already in
HBM: V -> MXFP4 pre-pass, then the fused attention forward (bf16 Q K^T on
MFMA, EFQ probability stage, FP4 P~V and P~1, online rescaling, final
division).  The headline workload is the 32K-token Qwen3-8B-shaped causal
prefill (32 query / 8 key-value heads, head_dim 128).  Prints one JSON line.

Besides the headline TFLOP/s it reports
  * roofline: the fused attention kernel's algorithmic flops over its
    average launch time (HIP events on the launch stream), against the
    MI355X dense bf16 / MXFP4 peaks weighted by the flop split, with the
    kernel-trace average and the HBM traffic of the committed rocprofv3
    summaries when they were taken on the current kernel source;
  * pgen: the probability stage alone (register-resident probe), EFQ vs
    exp-then-quantize, in microseconds per 128x128 score tile on one CU;
    the exposed stage cost inside the fused kernel (policy minus a no-op
    probability stage); and the stage's VALU-active cycles from the
    committed counter summary;
  * lowbit: the low-bit variant (MXFP8 Q and K, Q K^T on the FP8 matrix
    core) on the same workload, per probability stage;
  * workloads: the fused kernel on the other benchmark shapes (Qwen3-8B 16K
    and 128K, Qwen3-VL 32K, WAN2.2 75600);
  * cpu_baseline: the CPU oracle on a bounded sample of the same workload,
    on all host threads and on one, plus the output quality
    rho = ||O - O_exact||_F / ||O_exact||_F of the GPU's EFQ, LUT and
    exp-then-quantize outputs on those rows against exact softmax.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16 = 2500.0     # TFLOP/s, MI355X dense bf16 MFMA
PEAK_FP4 = 10100.0     # TFLOP/s, MI355X dense MXFP4 MFMA
PEAK_FP8 = 5000.0      # TFLOP/s, MI355X dense FP8 MFMA
PEAK_CLOCK_GHZ = 2.4   # the clock the peaks are quoted at
PEAK_HBM = 8.0         # TB/s, MI355X HBM3E
N_CU = 256
COPY_BYTES = 1 << 30   # plain copy used to scale the HBM counters


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_hash(src_path: str = None) -> str:
    """Hash of the kernel source's code: comments and blank lines are left
    out, so an edit of the comments keeps a counter summary valid."""
    import re
    if src_path is None:
        src_path = os.path.join(ROOT, "paper_2609_09721_amd", "csrc", "efq_attn.hip")
    with open(src_path) as f:
        src = f.read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    lines = [re.sub(r"//.*$", "", ln).strip() for ln in src.splitlines()]
    code = "\n".join(ln for ln in lines if ln.strip())
    return hashlib.sha256(code.encode()).hexdigest()[:16]


def read_profile(path: str):
    """key = value lines of a committed rocprofv3 summary, or None if the
    summary is missing or was taken on another kernel source."""
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if "=" in line and not line.startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_hash") != kernel_hash():
        return None
    return kv


def _profiles(profiles_dir):
    return profiles_dir or os.path.join(ROOT, "profiles")


def read_traffic(workload: str, profiles_dir: str = None):
    """HBM bytes per launch of the attention kernel from the committed
    rocprofv3 counter summary, if it was taken on the current kernel source."""
    kv = read_profile(os.path.join(_profiles(profiles_dir), f"attn_fwd_{workload}_traffic.txt"))
    try:
        return float(kv["traffic_bytes_per_launch"]) if kv else None
    except (KeyError, ValueError):
        return None


def read_trace_avg_ms(workload: str, profiles_dir: str = None):
    """Average and median duration (ms) of the bench-configuration EFQ
    attention launches in the committed kernel-trace summary of this
    workload, if it was taken on the current kernel source."""
    kv = read_profile(os.path.join(_profiles(profiles_dir),
                                   f"attn_pp_kernel_{workload}_stats.txt"))
    try:
        return (float(kv["efq_avg_us"]) / 1e3, float(kv["efq_median_us"]) / 1e3) if kv else None
    except (KeyError, ValueError):
        return None


def read_stage_counters(workload: str, profiles_dir: str = None):
    """Probability-stage VALU-active cycles per SIMD from the committed
    counter summary (fused kernel with the EFQ, exp-then-quantize and no-op
    stages, bf16 Q K^T): the stage's own cycles are those above the no-op
    stage.  Returns the cycles and the saving 1 - t_EFQ / t_EXPQ, or None."""
    kv = read_profile(os.path.join(_profiles(profiles_dir),
                                   f"attn_pp_kernel_{workload}_counters.txt"))
    try:
        efq, expq, noop = (float(kv[f"valu_active_cycles_{k}"]) for k in ("efq", "expq", "noop"))
    except (TypeError, KeyError, ValueError):
        return None
    se, sx = efq - noop, expq - noop
    return {"unit": "VALU-active cycles per SIMD above the no-op stage (rocprofv3 "
                    "SQ_ACTIVE_INST_VALU)",
            "efq": round(se), "expq": round(sx),
            "speedup": round(1.0 - se / sx, 4) if sx > 0 else None}


def read_stage_stamps(workload: str, profiles_dir: str = None):
    """Probability-stage ticks per tile from the committed phase-stamp
    summary (diagnostic build of the same kernel source): the matrix- plus
    VALU-phase time above the no-op stage, and 1 - t_EFQ / t_EXPQ, or None."""
    kv = read_profile(os.path.join(_profiles(profiles_dir),
                                   f"attn_pp_kernel_{workload}_phases.txt"))
    try:
        efq, expq = (float(kv[f"stamps_stage_ticks_{k}"]) for k in ("efq", "expq"))
        speedup = float(kv["stamps_speedup"])
    except (TypeError, KeyError, ValueError):
        return None
    out = {"unit": "s_memtime ticks (shader-clock cycles) per tile and wave above the no-op "
                   "stage (phase stamps, diagnostic build)",
           "efq": round(efq), "expq": round(expq), "speedup": round(speedup, 4)}
    try:
        out["sclk_ghz"] = float(kv["stamps_sclk_ghz"])
    except (KeyError, ValueError):
        pass
    return out


def measure_sclk(binding, stream, blocks: int = None, iters: int = 12000, launches: int = 10):
    """Shader clock in GHz that a pure matrix-core load holds: `launches`
    back-to-back runs of efq_clock_probe (bf16 MFMAs with changing operands
    on every CU, a few milliseconds each; s_memtime over the 100 MHz
    s_memrealtime), the median over workgroups of the last run, by which
    time the power limit has set the clock."""
    import numpy as np
    import torch
    blocks = blocks or N_CU
    t = torch.empty((launches, blocks, 2), dtype=torch.int64, device="cuda")
    for i in range(launches):
        binding.clock_probe(blocks, iters, out=t[i], stream=stream)
    torch.cuda.synchronize()
    a = t[-1].cpu().numpy().astype(np.float64)
    ok = a[:, 1] > 0
    return float(np.median(0.1 * a[ok, 0] / a[ok, 1])) if ok.any() else 0.0


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="qwen3_8b_32k")
    ap.add_argument("--kind", default="efq", choices=["efq", "expq", "expq6", "lut"])
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-extra", action="store_true", help="skip the P-gen and policy comparisons")
    ap.add_argument("--cpu-seconds", type=float, default=8.0,
                    help="target time of one all-thread CPU oracle call")
    ap.add_argument("--sweep", action="store_true",
                    help="sequence sweep of the Qwen3-8B heads (16K..128K, causal): fused-kernel "
                         "time per probability stage, one JSON line per length")
    ap.add_argument("--pmc-run", action="store_true",
                    help="counter-collection run: the attention kernel 3 times, then a plain "
                         "device copy of COPY_BYTES bytes 3 times (the HBM-counter scale)")
    ap.add_argument("--pmc-variants", action="store_true",
                    help="counter-collection run: one launch of the fused kernel per probability "
                         "stage (EFQ, no-op, exp-then-quantize), bf16 and MXFP8 Q K^T")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path "
              "(the kernel would shard by (batch, head) with no communication)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_09721_amd import binding, inputs

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    binding.lib()
    dev = torch.device("cuda:0")
    if args.sweep:
        sweep(args, binding, inputs, dev)
        return
    w = inputs.WORKLOADS[args.workload]
    log(f"[bench] workload {w}")
    t0 = time.time()
    q, k, v = inputs.make_qkv(w, device=dev)
    torch.cuda.synchronize()
    log(f"[bench] inputs generated in {time.time() - t0:.1f}s")
    sh = binding.shape_of(q, k)
    vhat = torch.empty(binding.vhat_bytes(sh), dtype=torch.uint8, device=dev)
    out = torch.empty(q.shape, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    params = binding.PARAMS_LUT if args.kind == "lut" else binding.PARAMS_MEAN

    def prm(kind):
        return binding.PARAMS_LUT if kind == "lut" else binding.PARAMS_MEAN

    def step(kind=args.kind, ev=None):
        if ev is not None:
            ev[0].record(stream)
        binding.quant_v(v, seq_q=w.seq, heads_q=w.heads_q, out=vhat, stream=stream)
        if ev is not None:
            ev[1].record(stream)
        binding.attn_fwd_vhat(q, k, vhat, w.scale, w.causal, kind, prm(kind), out=out,
                              stream=stream)
        if ev is not None:
            ev[2].record(stream)

    def timed(kind, steps, warmup):
        for _ in range(warmup):
            step(kind)
        torch.cuda.synchronize()
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        wall0 = time.perf_counter()
        start.record(stream)
        for i in range(steps):
            step(kind, evs[i])
        end.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        total_ms = start.elapsed_time(end)
        attn_ms = [e[1].elapsed_time(e[2]) for e in evs]
        vq_ms = [e[0].elapsed_time(e[1]) for e in evs]
        return total_ms / steps, sum(attn_ms) / steps, sum(vq_ms) / steps, wall

    if args.pmc_variants:
        qh, kh = binding.quant_qk(q, k, stream=stream)
        binding.quant_v(v, seq_q=w.seq, heads_q=w.heads_q, out=vhat, stream=stream)
        for kind in ("efq", "noop", "expq"):
            binding.attn_fwd_vhat(q, k, vhat, w.scale, w.causal, kind, binding.PARAMS_MEAN,
                                  out=out, stream=stream)
            binding.attn_fwd_qk8(qh, kh, vhat, sh, w.scale, w.causal, kind, binding.PARAMS_MEAN,
                                 out=out, stream=stream)
        torch.cuda.synchronize()
        log(f"[bench] pmc variants done ({w.name})")
        return

    if args.pmc_run:
        binding.quant_v(v, seq_q=w.seq, heads_q=w.heads_q, out=vhat, stream=stream)
        for _ in range(3):
            binding.attn_fwd_vhat(q, k, vhat, w.scale, w.causal, args.kind, params, out=out,
                                  stream=stream)
        torch.cuda.synchronize()
        src = torch.ones(COPY_BYTES, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] pmc run done: 3 x attention ({w.name}), 3 x copy of {COPY_BYTES} bytes")
        return

    ms_step, attn_ms, vq_ms, wall = timed(args.kind, args.steps, args.warmup)
    kclk = None
    if args.kind == "efq":
        # the clock during the fused kernel on this machine: launches of the
        # kernel's stamped diagnostic build (built beside the product
        # library) right after the timed steps, before anything else runs
        from paper_2609_09721_amd import build as hip_build, phases
        if os.path.exists(hip_build.STAMPS_LIB):
            kclk = round(phases.kernel_sclk(w, q, k, vhat, out), 3) or None
            binding.lib()
    sclk = measure_sclk(binding, stream)
    # the V quantiser alone, 20 launches back to back (its HBM roofline)
    def vq():
        binding.quant_v(v, seq_q=w.seq, heads_q=w.heads_q, out=vhat, stream=stream)
    vq()
    torch.cuda.synchronize()
    vq_loop_ms = _time_calls(vq, 20, stream)
    vq_bytes = v.numel() * 2 + vhat.numel()
    flops = w.flops()
    value = flops / (ms_step * 1e-3) / 1e12
    achieved = flops / (attn_ms * 1e-3) / 1e12
    peak = 1.0 / (0.5 / PEAK_BF16 + 0.5 / PEAK_FP4)
    log(f"[bench] {args.kind}: {ms_step:.3f} ms/step (attn {attn_ms:.3f} ms, vquant {vq_ms:.3f} ms), "
        f"{value:.1f} TFLOP/s, wall {wall:.2f}s")
    trace_ms = read_trace_avg_ms(w.name) if args.kind == "efq" else None

    result = {
        "metric": "attention fwd TFLOPS (EFQ-Softmax P-gen) + P-gen stage us/tile vs exp-then-quant",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 QK^T + mxfp4 PV (fp32 accumulate)",
        "data": "synthetic (seeded Qwen3-8B-shaped attention inputs, no weights)",
        "config": {
            "workload": w.name, "batch": w.batch, "heads_q": w.heads_q, "heads_kv": w.heads_kv,
            "seq": w.seq, "head_dim": w.head_dim, "causal": w.causal, "pgen": args.kind,
            "tau": params[0], "h": params[1], "block": 32, "tile": "256x64",
            "parallelism": "single GPU",
        },
        "roofline": {
            "kernel": "attn_pp_kernel",
            "bound": "mfma",
            "achieved": round(achieved, 2),
            "peak": round(peak, 1),
            "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4),
            "traffic": read_traffic(w.name),
            "flops_per_launch": flops,
            "avg_launch_ms": round(attn_ms, 4),
            "trace_avg_ms": trace_ms[0] if trace_ms else None,
            "trace_median_ms": trace_ms[1] if trace_ms else None,
            "trace_frac": (round(flops / (trace_ms[0] * 1e-3) / 1e12 / peak, 4)
                           if trace_ms else None),
            # the peaks are quoted at the 2.4 GHz peak clock.  Shader clock
            # during the kernel's stamped build right after the timed steps
            # (median of 5 launches) and the fraction of the peak scaled to
            # it; the clock a sustained pure-MFMA load holds (the power
            # limit) and the fraction of the peak scaled to that
            "sclk_ghz_in_kernel": kclk,
            "frac_at_kernel_sclk": (round(achieved / (peak * kclk / PEAK_CLOCK_GHZ), 4)
                                    if kclk else None),
            "sclk_ghz_mfma_sustained": round(sclk, 3),
            "frac_at_mfma_sustained_sclk": (round(achieved / (peak * sclk / PEAK_CLOCK_GHZ), 4)
                                            if sclk > 0 else None),
        },
        "vquant_ms": round(vq_ms, 4),
        "vquant": {"bound": "hbm", "us_per_launch": round(vq_loop_ms * 1e3, 2),
                   "bytes": vq_bytes,
                   "achieved_tbps": round(vq_bytes / (vq_loop_ms * 1e-3) / 1e12, 3),
                   "peak_tbps": PEAK_HBM,
                   "frac": round(vq_bytes / (vq_loop_ms * 1e-3) / 1e12 / PEAK_HBM, 4)},
    }

    if not args.no_extra:
        extra = {}
        # other probability stages in the same fused kernel
        for kind in ("expq", "expq6", "noop", "lut"):
            if kind == args.kind:
                continue
            _, attn_k, _, _ = timed(kind, max(5, args.steps // 2), 2)
            extra[kind] = {"attn_ms": round(attn_k, 4),
                           "tflops": round(flops / (attn_k * 1e-3) / 1e12, 2)}
        extra[args.kind] = {"attn_ms": round(attn_ms, 4), "tflops": round(achieved, 2)}
        tiles = w.pairs() / 16384.0            # 128 x 128 score tiles (visible pairs)
        noop = extra["noop"]["attn_ms"]
        exposed = {}
        for kind in ("efq", "expq", "expq6", "lut"):
            if kind in extra:
                exposed[kind] = round((extra[kind]["attn_ms"] - noop) * 1e3 * N_CU / tiles, 4)
        # register-resident probe of the probability stage alone
        waves, iters = 8192, 400
        probe = {}
        for kind in ("efq", "expq", "expq6", "lut"):
            cs = torch.empty(waves, dtype=torch.int32, device=dev)
            binding.pgen_bench(kind, None, waves, 8, cs)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            binding.pgen_bench(kind, None, waves, iters, cs)
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1)
            scores = waves * iters * 32 * 64
            probe[kind] = round(ms * 1e3 * N_CU / (scores / 16384.0), 4)
        result["pgen"] = {
            "unit": "us per 128x128 score tile per CU",
            "probe_efq": probe["efq"], "probe_expq": probe["expq"], "probe_expq6": probe["expq6"],
            "probe_lut": probe["lut"],
            "probe_speedup": round(1.0 - probe["efq"] / probe["expq"], 4),
            "probe_speedup_vs_scale6": round(1.0 - probe["efq"] / probe["expq6"], 4),
            "exposed_in_kernel": exposed,
            "exposed_speedup": (round(1.0 - exposed["efq"] / exposed["expq"], 4)
                                if exposed.get("expq", 0) > 0 else None),
            "stage_valu_counters": read_stage_counters(w.name),
            "stage_stamps": read_stage_stamps(w.name),
            "paper_context": "Ascend 950PR vector-stage latency reduction 40.33% (16K-128K)",
        }
        result["policies"] = extra
        result["lowbit"] = lowbit_run(w, binding, q, k, v, vhat, out, stream, args.steps)
        result["workloads"] = workloads_run(binding, inputs, dev, stream, skip=w.name)

    if not args.no_cpu:
        # GPU outputs of the sampled rows for the quality figure, then the
        # CPU oracle leg on the same rows
        rows = inputs.sample_rows(w, 1024, seed=1)
        gpu_rows = {}
        binding.quant_v(v, seq_q=w.seq, heads_q=w.heads_q, out=vhat, stream=stream)
        for kind in ("efq", "lut", "expq"):
            binding.attn_fwd_vhat(q, k, vhat, w.scale, w.causal, kind, prm(kind), out=out,
                                  stream=stream)
            gpu_rows[kind] = out[rows[:, 0].long(), rows[:, 2].long(),
                                 rows[:, 1].long()].cpu().numpy()
        del vhat, out
        torch.cuda.empty_cache()
        result["cpu_baseline"] = cpu_baseline(w, q, k, v, args.cpu_seconds, rows.numpy(),
                                              gpu_rows)

    print(json.dumps(result), flush=True)


def sweep(args, binding, inputs, dev):
    """Fused-kernel time on the Qwen3-8B heads (32 q / 8 kv, D 128, causal)
    over the sequence lengths of the paper's kernel table (16K..128K), for
    each probability stage; the exposed stage cost is t(policy) - t(no-op).
    One JSON line per length."""
    import torch
    base = inputs.WORKLOADS["qwen3_8b_32k"]
    stream = torch.cuda.current_stream()
    peak = 1.0 / (0.5 / PEAK_BF16 + 0.5 / PEAK_FP4)
    for seq in (16384, 24576, 32768, 49152, 65536, 131072):
        w = base.with_seq(seq)
        q, k, v = inputs.make_qkv(w, device=dev)
        vh = binding.quant_v(v, seq_q=w.seq, heads_q=w.heads_q, stream=stream)
        out = torch.empty(q.shape, dtype=torch.float32, device=dev)
        n = 10 if seq <= 32768 else 4
        if seq == 16384:   # bring the clocks up before the first timed length
            for _ in range(30):
                binding.attn_fwd_vhat(q, k, vh, w.scale, True, "efq", binding.PARAMS_MEAN, out=out,
                                      stream=stream)
            torch.cuda.synchronize()
        res = {"seq": seq, "causal": True, "pairs": w.pairs(), "flops": w.flops()}
        for kind in ("efq", "expq", "expq6", "lut", "noop"):
            prm = binding.PARAMS_LUT if kind == "lut" else binding.PARAMS_MEAN
            for _ in range(3):   # warm-up
                binding.attn_fwd_vhat(q, k, vh, w.scale, True, kind, prm, out=out, stream=stream)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(n):
                binding.attn_fwd_vhat(q, k, vh, w.scale, True, kind, prm, out=out, stream=stream)
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / n
            tf = w.flops() / (ms * 1e-3) / 1e12
            res[kind] = {"attn_ms": round(ms, 4), "tflops": round(tf, 1), "frac": round(tf / peak, 4)}
        noop = res["noop"]["attn_ms"]
        ex = {kd: res[kd]["attn_ms"] - noop for kd in ("efq", "expq", "expq6", "lut")}
        res["exposed_ms"] = {kd: round(x, 4) for kd, x in ex.items()}
        res["exposed_speedup_vs_expq"] = round(1 - ex["efq"] / ex["expq"], 4) if ex["expq"] > 0 else None
        # low-bit Q K^T (MXFP8 Q and K)
        sh = binding.shape_of(q, k)
        qh, kh = binding.quant_qk(q, k, stream=stream)
        peak8 = 1.0 / (0.5 / PEAK_FP8 + 0.5 / PEAK_FP4)
        lb = {}
        for kind in ("efq", "expq", "noop"):
            def call(kind=kind):
                binding.attn_fwd_qk8(qh, kh, vh, sh, w.scale, True, kind, binding.PARAMS_MEAN,
                                     out=out, stream=stream)
            for _ in range(3):
                call()
            torch.cuda.synchronize()
            ms = _time_calls(call, n, stream)
            tf = w.flops() / (ms * 1e-3) / 1e12
            lb[kind] = {"attn_ms": round(ms, 4), "tflops": round(tf, 1), "frac": round(tf / peak8, 4)}
        exl = {kd: lb[kd]["attn_ms"] - lb["noop"]["attn_ms"] for kd in ("efq", "expq")}
        lb["exposed_speedup_vs_expq"] = round(1 - exl["efq"] / exl["expq"], 4) if exl["expq"] > 0 else None
        res["lowbit"] = lb
        print(json.dumps(res), flush=True)
        del q, k, v, vh, out, qh, kh
        torch.cuda.empty_cache()


def _time_calls(fn, n, stream):
    """Mean time per call (ms) of n back-to-back calls on stream."""
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(n):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / n


def _median_call(fn, n, stream):
    """Median time (ms) of n calls, each bracketed by its own events."""
    import torch
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(n)]
    for a, b in ev:
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    ts = sorted(a.elapsed_time(b) for a, b in ev)
    return ts[n // 2]


def lowbit_run(w, binding, q, k, v, vhat, out, stream, steps):
    """Low-bit Q K^T on the same inputs: the MXFP8 pre-pass of Q and K, the
    MXFP4 pre-pass of V, then the fused kernel with the FP8 Q K^T.  Fused
    kernel time per probability stage (and the exposed stage cost against
    the no-op stage), the pre-pass time, and the whole step."""
    import torch
    sh = binding.shape_of(q, k)
    qh, kh = binding.quant_qk(q, k, stream=stream)
    binding.quant_v(v, seq_q=w.seq, heads_q=w.heads_q, out=vhat, stream=stream)
    peak = 1.0 / (0.5 / PEAK_FP8 + 0.5 / PEAK_FP4)
    n = max(5, steps // 2)
    res = {"qk": "mxfp8 (e4m3, e8m0 per 32)", "peak": round(peak, 1), "unit": "TFLOP/s"}
    for kind in ("efq", "expq", "expq6", "noop"):
        def call(kind=kind):
            binding.attn_fwd_qk8(qh, kh, vhat, sh, w.scale, w.causal, kind, binding.PARAMS_MEAN,
                                 out=out, stream=stream)
        for _ in range(2):
            call()
        torch.cuda.synchronize()
        ms = _time_calls(call, n, stream)
        tf = w.flops() / (ms * 1e-3) / 1e12
        res[kind] = {"attn_ms": round(ms, 4), "tflops": round(tf, 2), "frac": round(tf / peak, 4)}
    ex = {kd: res[kd]["attn_ms"] - res["noop"]["attn_ms"] for kd in ("efq", "expq", "expq6")}
    res["exposed_ms"] = {kd: round(x, 4) for kd, x in ex.items()}
    res["exposed_speedup_vs_expq"] = round(1 - ex["efq"] / ex["expq"], 4) if ex["expq"] > 0 else None

    def prepass():
        binding.quant_qk(q, k, stream=stream)
    prepass()   # its output buffers come from the allocator's cache from here on
    torch.cuda.synchronize()
    pms = _time_calls(prepass, n, stream)
    pbytes = (q.numel() + k.numel()) * 2 + qh.numel() + kh.numel()
    res["qk_prepass_ms"] = round(pms, 4)
    res["qk_prepass_tbps"] = round(pbytes / (pms * 1e-3) / 1e12, 3)
    res["qk_prepass_frac_hbm"] = round(pbytes / (pms * 1e-3) / 1e12 / PEAK_HBM, 4)
    ws = torch.empty(binding.lowbit_workspace_bytes(sh) + 256, dtype=torch.uint8, device=q.device)
    off = (-ws.data_ptr()) % 256
    wsv = ws[off: off + binding.lowbit_workspace_bytes(sh)]

    def whole():
        binding.attn_fwd_lowbit(q, k, v, w.scale, w.causal, "efq", out=out, workspace=wsv,
                                stream=stream)
    whole()
    torch.cuda.synchronize()
    ms = _time_calls(whole, n, stream)
    res["step_ms"] = round(ms, 4)
    res["step_tflops"] = round(w.flops() / (ms * 1e-3) / 1e12, 2)
    del qh, kh, ws
    return res


def workloads_run(binding, inputs, dev, stream, skip=None):
    """The other benchmark shapes (Qwen3-8B 16K and 128K causal, Qwen3-VL 32K
    and WAN2.2 75600 non-causal): fused-kernel time (median of 3 launches)
    per probability stage, bf16 and MXFP8 Q K^T, and the fraction of each
    path's MFMA roofline."""
    import torch
    peak = 1.0 / (0.5 / PEAK_BF16 + 0.5 / PEAK_FP4)
    peak8 = 1.0 / (0.5 / PEAK_FP8 + 0.5 / PEAK_FP4)
    res = {"timing": "median of 3 launches after one warm-up"}
    for name in ("qwen3_8b_16k", "qwen3_8b_128k", "qwen3_vl_32k", "wan22_75600"):
        if name == skip:
            continue
        w = inputs.WORKLOADS[name]
        q, k, v = inputs.make_qkv(w, device=dev)
        vh = binding.quant_v(v, seq_q=w.seq, heads_q=w.heads_q, stream=stream)
        qh, kh = binding.quant_qk(q, k, stream=stream)
        sh = binding.shape_of(q, k)
        out = torch.empty(q.shape, dtype=torch.float32, device=dev)
        r = {"batch": w.batch, "heads_q": w.heads_q, "heads_kv": w.heads_kv, "seq": w.seq,
             "causal": w.causal, "flops": w.flops()}
        for kind in ("efq", "expq"):
            def call(kind=kind):
                binding.attn_fwd_vhat(q, k, vh, w.scale, w.causal, kind, binding.PARAMS_MEAN,
                                      out=out, stream=stream)

            def call8(kind=kind):
                binding.attn_fwd_qk8(qh, kh, vh, sh, w.scale, w.causal, kind, binding.PARAMS_MEAN,
                                     out=out, stream=stream)
            for fn, key, pk in ((call, kind, peak), (call8, "lowbit_" + kind, peak8)):
                fn()
                torch.cuda.synchronize()
                ms = _median_call(fn, 3, stream)
                tf = w.flops() / (ms * 1e-3) / 1e12
                r[key] = {"attn_ms": round(ms, 3), "tflops": round(tf, 1), "frac": round(tf / pk, 4)}
        res[name] = r
        log(f"[bench] {name}: efq {r['efq']['attn_ms']} ms, low-bit efq {r['lowbit_efq']['attn_ms']} ms")
        del q, k, v, vh, qh, kh, out
        torch.cuda.empty_cache()
    return res


def cpu_baseline(w, q, k, v, target_s: float, rows, gpu_rows):
    """The CPU oracle (unchanged) on a stratified sample of query rows: the
    rate is algorithmic flops of the sampled rows over the wall time of one
    call, on all the host threads this job may use (at most 16) and on one
    thread.  Each call also quantises all of V.  The sample grows (at most
    16x per round) until the all-thread call takes at least half the time
    target; the one-thread call gets a subsample sized to take about as
    long.  Also the output quality on the first 1024-row sample:
    rho = ||O - O_exact||_F / ||O_exact||_F (Sec. III-C's objective) of the
    GPU outputs of EFQ, EFQ-Softmax-LUT and exp-then-quantize against the
    oracle's exact fp64 softmax with unquantised V."""
    import numpy as np
    import oracle
    from paper_2609_09721_amd import inputs

    oracle.lib()
    qb = oracle.bf16_bits(q)
    kb = oracle.bf16_bits(k)
    vb = oracle.bf16_bits(v)
    host = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    threads = max(1, min(host, 16))
    total_rows = w.batch * w.heads_q * w.seq

    def row_flops(rs):
        keys = (rs[:, 2].astype(np.int64) + 1) if w.causal else np.full(len(rs), w.seq)
        return float(4 * w.head_dim * keys.sum())

    def call(rs, nth):
        t = time.perf_counter()
        oracle.attn(qb, kb, vb, w.scale, w.causal, oracle.EFQ, bc=64, rows=rs, nthreads=nth)
        dt = time.perf_counter() - t
        log(f"[bench] cpu oracle: {len(rs)} rows in {dt:.2f}s on {nth} threads")
        return dt

    # quality against exact softmax on the given rows
    exact = oracle.attn(qb, kb, vb, w.scale, w.causal, oracle.EXACT, bc=64, rows=rows,
                        nthreads=threads).astype(np.float64)
    norm = np.sqrt(np.sum(exact * exact))
    rho = {kind: round(float(np.sqrt(np.sum((o.astype(np.float64) - exact) ** 2)) / norm), 6)
           for kind, o in gpu_rows.items()}

    n, seed, spent = 64, 2, 0.0
    while True:
        rs = inputs.sample_rows(w, n, seed=seed).numpy()
        dt = call(rs, threads)
        spent += dt
        if dt >= 0.5 * target_s or n >= total_rows or spent >= 3 * target_s:
            break
        n = int(min(total_rows, n * min(16.0, max(2.0, target_s / max(dt, 1e-3)))))
        seed += 1
    rate = row_flops(rs) / dt
    # one thread: a subsample expected to take about as long as the call above
    sub = rs[:: max(1, threads)]
    dt1 = call(sub, 1)
    rate1 = row_flops(sub) / dt1
    return {"value": round(rate / 1e12, 8), "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"{len(rs)} of {total_rows} query rows of the same workload, stratified "
                      f"over heads and positions; one call of {dt:.1f}s on {threads} threads "
                      f"(includes quantising all of V)",
            "seconds": round(dt, 2),
            "host_cores": host,
            "single_thread": {"value": round(rate1 / 1e12, 8), "unit": "TFLOP/s", "cores": 1,
                              "rows": len(sub), "seconds": round(dt1, 2)},
            "rho_vs_exact": dict(rho, rows=len(rows),
                                 definition="||O - O_exact||_F / ||O_exact||_F over the sampled "
                                            "rows; O_exact = fp64 softmax attention with "
                                            "unquantised V (oracle EXACT mode)")}


if __name__ == "__main__":
    main()
