"""Text summaries of rocprofv3 output for the profiles/ folder.

traffic FETCH_DIR WRITE_DIR WORKLOAD [OUT_FILE]
    HBM traffic per launch of the attention kernel from two counter runs of
    `bench.py --pmc-run` (one with FETCH_SIZE, one with WRITE_SIZE).  Both
    counters are scaled by what they read for the plain device copy of
    known size in the same run (the runtime's copyBuffer kernel; bytes read
    and written = COPY_BYTES each).  Writes
    profiles/attn_fwd_<workload>_traffic.txt, which bench.py reports as
    roofline.traffic while the kernel source is unchanged.

stats TRACE_DIR OUT_FILE WORKLOAD COMMAND...
    Kernel-time summary of a `rocprofv3 --kernel-trace --stats` run: the
    per-kernel statistics, and per launch configuration (grid size) the
    calls and average duration of the attention kernels.  Records the
    average of the bf16 EFQ attention kernel at WORKLOAD's launch
    configuration (efq_avg_us) with the kernel-source hash, which bench.py
    reports beside its own HIP-event average.

sweep JSONL OUT_FILE COMMAND...
    Table of a `bench.py --sweep` run (one JSON line per sequence length).

counters OUT_FILE WORKLOAD COMMAND... -- PMC_DIR [PMC_DIR ...]
    Per attention-kernel variant of `bench.py --pmc-variants` runs (one
    directory per counter pass, merged by dispatch order): matrix-core busy,
    VALU-active and co-execution cycles per SIMD as fractions of the
    kernel's cycles, VALU / MFMA / SALU / LDS instructions per SIMD and VALU
    instructions per score, LDS bank conflicts, and, where the passes hold
    them, the wave wait counters.  Records the VALU-active cycles per SIMD
    of the bf16 EFQ, exp-then-quantize and no-op kernels with the
    kernel-source hash, which bench.py reads as the probability stage's
    counter view.
"""
from __future__ import annotations

import csv
import glob
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def per_dispatch(d: str, counter: str):
    """[(kernel name, value)] per dispatch, in dispatch order."""
    rows = []
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        rows += list(csv.DictReader(open(f)))
    acc = {}
    for r in rows:
        if r["Counter_Name"] != counter:
            continue
        key = int(r["Dispatch_Id"])
        name, val = acc.get(key, (r["Kernel_Name"], 0.0))
        acc[key] = (name, val + float(r["Counter_Value"]))
    return [acc[k] for k in sorted(acc)]


def mean_of(disp, pred):
    vals = [v for n, v in disp if pred(n)]
    if not vals:
        raise SystemExit("no matching dispatch in the counter output")
    return sum(vals) / len(vals), len(vals)


def _grid_items(workload: str) -> int:
    """Work-items of the attention launch of a workload (256 queries and 512
    threads per workgroup)."""
    from paper_2609_09721_amd import inputs
    w = inputs.WORKLOADS[workload]
    return w.batch * w.heads_q * ((w.seq + 255) // 256) * 512


def stats(trace_dir: str, out: str, workload: str, command: str):
    rows = []
    for f in glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True):
        rows += list(csv.DictReader(open(f)))
    trace = []
    for f in glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True):
        trace += list(csv.DictReader(open(f)))
    def short(n: str) -> str:
        n = n.replace("(anonymous namespace)::", "").replace("void ", "")
        return n.split("(")[0][:110]
    with open(out, "w") as fh:
        fh.write("# rocprofv3 kernel-time summary\n")
        fh.write(f"# command (from the repository root, TMPDIR=/tmp):\n#   {command}\n")
        fh.write("# kernel | calls | average us | min us | max us | share of kernel time %\n")
        for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
            fh.write(f"{short(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                     f"{float(r['Percentage']):.2f}\n")
        fh.write("# attention kernels per launch configuration (grid size in work-items)\n")
        fh.write("# kernel | grid | calls | average us | median us | min us | max us\n")
        groups = {}
        for r in trace:
            n = r["Kernel_Name"]
            if "attn_" not in n:
                continue
            g = r.get("Grid_Size") or r.get("Grid_Size_X") or "?"
            d = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
            groups.setdefault((short(n), g), []).append(d)
        for (n, g), ds in sorted(groups.items()):
            med = sorted(ds)[len(ds) // 2]
            fh.write(f"{n} | {g} | {len(ds)} | {sum(ds) / len(ds):.1f} | {med:.1f} | "
                     f"{min(ds):.1f} | {max(ds):.1f}\n")
        import bench
        grid = str(_grid_items(workload))
        efq = [ds for (n, g), ds in groups.items()
               if n == "attn_pp_kernel<128, 0, true, false, false>" and g == grid]
        if efq:
            ds = efq[0]
            fh.write(f"# bf16 EFQ attention kernel at the {workload} launch configuration "
                     f"(grid {grid})\n")
            fh.write(f"efq_calls = {len(ds)}\nefq_avg_us = {sum(ds) / len(ds):.1f}\n")
            fh.write(f"efq_median_us = {sorted(ds)[len(ds) // 2]:.1f}\n")
            fh.write(f"kernel_hash = {bench.kernel_hash()}\n")
    print(open(out).read())


def sweep(jsonl: str, out: str, command: str):
    import json
    rows = [json.loads(l) for l in open(jsonl) if l.strip().startswith("{")]
    with open(out, "w") as fh:
        fh.write("# fused attention kernel time per sequence length, Qwen3-8B heads "
                 "(32 q / 8 kv, D 128, causal), HIP events on the launch stream\n")
        fh.write(f"# command (from the repository root):\n#   {command}\n")
        fh.write("# exposed = t(policy) - t(no-op probability stage); speedup = 1 - exposed(EFQ) / "
                 "exposed(exp-then-quantize)\n")
        fh.write("# seq | efq ms | expq ms | expq6 ms | lut ms | noop ms | efq TFLOP/s | frac | "
                 "exposed speedup | low-bit efq ms | low-bit expq ms | low-bit noop ms | "
                 "low-bit frac | low-bit exposed speedup\n")
        for r in rows:
            lb = r.get("lowbit", {})
            g = lambda d, k: d.get(k, {}).get("attn_ms", float("nan"))
            fh.write(f"{r['seq']} | {g(r, 'efq'):.3f} | {g(r, 'expq'):.3f} | {g(r, 'expq6'):.3f} | "
                     f"{g(r, 'lut'):.3f} | {g(r, 'noop'):.3f} | {r['efq']['tflops']} | "
                     f"{r['efq']['frac']} | {r['exposed_speedup_vs_expq']} | {g(lb, 'efq'):.3f} | "
                     f"{g(lb, 'expq'):.3f} | {g(lb, 'noop'):.3f} | "
                     f"{lb.get('efq', {}).get('frac')} | {lb.get('exposed_speedup_vs_expq')}\n")
    print(open(out).read())


def counters(dirs, out: str, workload: str, command: str):
    import collections
    acc = collections.defaultdict(lambda: collections.defaultdict(float))
    names = {}
    for d in dirs:
        rows = []
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            rows += list(csv.DictReader(open(f)))
        order = sorted({int(r["Dispatch_Id"]) for r in rows if "attn_pp_kernel" in r["Kernel_Name"]})
        pos = {dsp: i for i, dsp in enumerate(order)}
        for r in rows:
            n = r["Kernel_Name"]
            if "attn_pp_kernel" not in n:
                continue
            key = pos[int(r["Dispatch_Id"])]
            names[key] = n.replace("(anonymous namespace)::", "").replace("void ", "").split("(")[0]
            acc[key][r["Counter_Name"]] += float(r["Counter_Value"])
    simds, xcds = 1024, 8
    from paper_2609_09721_amd import inputs
    pairs = inputs.WORKLOADS[workload].pairs()
    kinds = {"attn_pp_kernel<128, 0, true, false, false>": "efq",
             "attn_pp_kernel<128, 1, true, false, false>": "expq",
             "attn_pp_kernel<128, 3, true, false, false>": "noop"}
    with open(out, "w") as fh:
        fh.write(f"# matrix-core and VALU activity of the fused attention kernel, {workload}\n")
        fh.write(f"# command (from the repository root, TMPDIR=/tmp), one run per counter pass:\n")
        for c in command.split(" ;; "):
            fh.write(f"#   {c}\n")
        fh.write("# kernel template: <head_dim, pgen kind (0 EFQ, 1 EXPQ, 3 no-op), causal, dump, "
                 "MXFP8 Q K^T>\n")
        fh.write("# cycles per XCD = GRBM_GUI_ACTIVE / 8; MFMA busy and VALU active are per SIMD "
                 "(SQ_ACTIVE_INST_VALU is in quad-cycles, summed over the SIMD's waves)\n")
        fh.write("# VALU per score: wave instructions (MFMA included) x 64 lanes / visible "
                 "(query, key) pairs\n")
        fh.write("# co-exec: cycles in which the matrix core was busy and a VALU instruction "
                 "issued (SQ_VALU_MFMA_COEXEC_CYCLES), per SIMD\n")
        fh.write("# wait / wait-issue: wave cycles waiting on a dependency or counter "
                 "(SQ_WAIT_ANY) and with an instruction ready but not issued "
                 "(SQ_WAIT_INST_ANY), per SIMD cycle, summed over the SIMD's waves\n")
        fh.write("# LDS busy: SQ_LDS_IDX_ACTIVE per CU cycle (4 per 1 KB ds_read_b128, i.e. "
                 "cycles at 256 B/clk); TA coalesced: TA_BUFFER_COALESCED_READ_CYCLES / "
                 "TA_BUFFER_TOTAL_CYCLES; TA busy: TA_BUFFER_TOTAL_CYCLES per TA cycle\n")
        fh.write("# kernel | cycles | MFMA busy | VALU active | co-exec | wait | wait-issue | "
                 "VALU instr per SIMD | MFMA instr per SIMD | SALU instr per SIMD | "
                 "VALU per score | LDS instr per SIMD | bank-conflict cycles per LDS instr | "
                 "LDS busy | TA coalesced | TA busy\n")
        per_kind = {}
        for key in sorted(acc):
            c = acc[key]
            cyc = c["GRBM_GUI_ACTIVE"] / xcds / max(1, len(dirs))
            g = lambda n, scale=1.0: (c[n] * scale / simds / cyc) if n in c else float("nan")
            va = 4 * c.get("SQ_ACTIVE_INST_VALU", float("nan")) / simds
            fh.write(f"{names[key]} | {cyc:.0f} | {g('SQ_VALU_MFMA_BUSY_CYCLES'):.3f} | "
                     f"{va / cyc:.3f} | {g('SQ_VALU_MFMA_COEXEC_CYCLES'):.3f} | "
                     f"{g('SQ_WAIT_ANY', 4):.3f} | {g('SQ_WAIT_INST_ANY', 4):.3f} | "
                     f"{c.get('SQ_INSTS_VALU', float('nan')) / simds:.0f} | "
                     f"{c.get('SQ_INSTS_MFMA', float('nan')) / simds:.0f} | "
                     f"{c.get('SQ_INSTS_SALU', float('nan')) / simds:.0f} | "
                     f"{c.get('SQ_INSTS_VALU', float('nan')) * 64 / pairs:.2f} | "
                     f"{c.get('SQ_INSTS_LDS', float('nan')) / simds:.0f} | "
                     f"{c.get('SQ_LDS_BANK_CONFLICT', 0) / max(c.get('SQ_INSTS_LDS', 0), 1):.4f} | "
                     f"{c.get('SQ_LDS_IDX_ACTIVE', float('nan')) / (simds / 4) / cyc:.3f} | "
                     f"{c.get('TA_BUFFER_COALESCED_READ_CYCLES', float('nan')) / max(c.get('TA_BUFFER_TOTAL_CYCLES', 0), 1):.3f} | "
                     f"{c.get('TA_BUFFER_TOTAL_CYCLES', float('nan')) / (simds / 4) / cyc:.3f}\n")
            if names[key] in kinds:
                per_kind[kinds[names[key]]] = (va, g("SQ_VALU_MFMA_BUSY_CYCLES"))
        for kind, (va, mf) in sorted(per_kind.items()):
            fh.write(f"valu_active_cycles_{kind} = {va:.0f}\nmfma_busy_{kind} = {mf:.4f}\n")
        import bench
        fh.write(f"kernel_hash = {bench.kernel_hash()}\n")
    print(open(out).read())


def main():
    if sys.argv[1] == "counters":
        rest = sys.argv[4:]
        cut = rest.index("--")
        counters(rest[cut + 1:], sys.argv[2], sys.argv[3], " ".join(rest[:cut]))
        return
    if sys.argv[1] == "stats":
        stats(sys.argv[2], sys.argv[3], sys.argv[4], " ".join(sys.argv[5:]))
        return
    if sys.argv[1] == "sweep":
        sweep(sys.argv[2], sys.argv[3], " ".join(sys.argv[4:]))
        return
    import bench
    from paper_2609_09721_amd import inputs
    args = sys.argv[2:]
    l2_dir = None
    if "--l2" in args:
        i = args.index("--l2")
        l2_dir = args[i + 1]
        del args[i:i + 2]
    fetch_dir, write_dir, wl = args[0], args[1], args[2]
    out = args[3] if len(args) > 3 else os.path.join(ROOT, "profiles",
                                                     f"attn_fwd_{wl}_traffic.txt")
    is_attn = lambda n: "attn_pp_kernel" in n or "attn_fwd_kernel" in n
    is_copy = lambda n: "copyBuffer" in n
    f = per_dispatch(fetch_dir, "FETCH_SIZE")
    wr = per_dispatch(write_dir, "WRITE_SIZE")
    fa, na = mean_of(f, is_attn)
    fc, nc = mean_of(f, is_copy)
    wa, _ = mean_of(wr, is_attn)
    wc, _ = mean_of(wr, is_copy)
    kf = bench.COPY_BYTES / fc          # bytes per counter unit, reads
    kw = bench.COPY_BYTES / wc          # bytes per counter unit, writes
    rd, wb = fa * kf, wa * kw
    w = inputs.WORKLOADS[wl]
    algo = (w.batch * w.seq * w.heads_q * w.head_dim * 2               # Q bf16
            + w.batch * w.seq * w.heads_kv * w.head_dim * 2            # K bf16
            + w.batch * w.heads_kv * 2 * ((w.seq + 63) // 64) * w.head_dim * 17  # V~
            + w.batch * w.seq * w.heads_q * w.head_dim * 4)            # O fp32
    algo_rd = algo - w.batch * w.seq * w.heads_q * w.head_dim * 4
    with open(out, "w") as fh:
        fh.write(f"# HBM traffic of one attention launch, {wl} (EFQ), from rocprofv3 counters\n")
        fh.write("# commands (from the repository root, TMPDIR=/tmp):\n")
        fh.write("#   rocprofv3 --pmc FETCH_SIZE -d <FETCH_DIR> -o p --output-format csv -- "
                 f"python3 bench.py --pmc-run --workload {wl}\n")
        fh.write("#   rocprofv3 --pmc WRITE_SIZE -d <WRITE_DIR> -o p --output-format csv -- "
                 f"python3 bench.py --pmc-run --workload {wl}\n")
        if l2_dir:
            fh.write("#   rocprofv3 --pmc TCC_HIT_sum TCC_MISS_sum TCC_EA0_RDREQ_sum TCC_EA0_RDREQ_DRAM_sum "
                     f"-d <L2_DIR> -o p --output-format csv -- python3 bench.py --pmc-run --workload {wl}\n")
        fh.write(f"#   python3 -m paper_2609_09721_amd.profsum traffic <FETCH_DIR> <WRITE_DIR> {wl}"
                 + (" --l2 <L2_DIR>" if l2_dir else "") + "\n")
        fh.write(f"# attention dispatches {na}, copy dispatches {nc}; copy size {bench.COPY_BYTES} B\n")
        fh.write(f"fetch_counter_attn = {fa:.1f}\nfetch_counter_copy = {fc:.1f}\n")
        fh.write(f"write_counter_attn = {wa:.1f}\nwrite_counter_copy = {wc:.1f}\n")
        fh.write(f"fetch_scale_bytes_per_unit = {kf:.4f}\nwrite_scale_bytes_per_unit = {kw:.4f}\n")
        fh.write(f"read_bytes_per_launch = {rd:.0f}\nwrite_bytes_per_launch = {wb:.0f}\n")
        fh.write(f"algorithmic_bytes_per_launch = {algo}\n")
        fh.write(f"traffic_bytes_per_launch = {rd + wb:.0f}\n")
        fh.write(f"algorithmic_read_bytes_per_launch = {algo_rd}\n")
        fh.write(f"read_over_algorithmic = {rd / algo_rd:.3f}\n")
        if l2_dir:
            hit, _ = mean_of(per_dispatch(l2_dir, "TCC_HIT_sum"), is_attn)
            miss, _ = mean_of(per_dispatch(l2_dir, "TCC_MISS_sum"), is_attn)
            ea, _ = mean_of(per_dispatch(l2_dir, "TCC_EA0_RDREQ_sum"), is_attn)
            dram, _ = mean_of(per_dispatch(l2_dir, "TCC_EA0_RDREQ_DRAM_sum"), is_attn)
            fh.write(f"l2_hit_rate = {hit / max(hit + miss, 1):.4f}\n")
            fh.write(f"l2_read_requests_to_memory = {ea:.0f}\n")
            fh.write(f"of_them_to_dram = {dram:.0f}\n")
        fh.write(f"kernel_hash = {bench.kernel_hash()}\n")
    print(open(out).read())


if __name__ == "__main__":
    main()
