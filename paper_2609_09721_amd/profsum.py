"""Text summaries of rocprofv3 output for the profiles/ folder.

traffic FETCH_DIR WRITE_DIR WORKLOAD [OUT_FILE]
    HBM traffic per launch of the attention kernel from two counter runs of
    `bench.py --pmc-run` (one with FETCH_SIZE, one with WRITE_SIZE).  Both
    counters are scaled by what they read for the plain device copy of
    known size in the same run (the runtime's copyBuffer kernel; bytes read
    and written = COPY_BYTES each).  Writes
    profiles/attn_fwd_<workload>_traffic.txt, which bench.py reports as
    roofline.traffic while the kernel source is unchanged.

stats TRACE_DIR OUT_FILE COMMAND...
    Kernel-time summary of a `rocprofv3 --kernel-trace --stats` run: the
    per-kernel statistics, and per launch configuration (grid size) the
    calls and average duration of the attention kernels.

sweep JSONL OUT_FILE COMMAND...
    Table of a `bench.py --sweep` run (one JSON line per sequence length).

counters PMC_DIR OUT_FILE COMMAND...
    Per attention-kernel variant of a `bench.py --pmc-variants` run with
    SQ_VALU_MFMA_BUSY_CYCLES, SQ_ACTIVE_INST_VALU, SQ_INSTS_VALU,
    SQ_INSTS_MFMA, SQ_INSTS_LDS, SQ_LDS_BANK_CONFLICT and GRBM_GUI_ACTIVE:
    matrix-core busy and VALU-active cycles per SIMD as fractions of the
    kernel's cycles, VALU instructions per SIMD and per score, and LDS
    bank-conflict stall cycles per LDS instruction.
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


def stats(trace_dir: str, out: str, command: str):
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


def counters(d: str, out: str, command: str):
    import collections
    rows = []
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        rows += list(csv.DictReader(open(f)))
    acc = collections.defaultdict(lambda: collections.defaultdict(float))
    names = {}
    for r in rows:
        n = r["Kernel_Name"]
        if "attn_pp_kernel" not in n:
            continue
        key = int(r["Dispatch_Id"])
        names[key] = n.replace("(anonymous namespace)::", "").replace("void ", "").split("(")[0]
        acc[key][r["Counter_Name"]] += float(r["Counter_Value"])
    simds, xcds = 1024, 8
    from paper_2609_09721_amd import inputs
    pairs = inputs.WORKLOADS["qwen3_8b_16k"].pairs()
    with open(out, "w") as fh:
        fh.write("# matrix-core and VALU activity of the fused attention kernel, qwen3_8b_16k\n")
        fh.write(f"# command (from the repository root, TMPDIR=/tmp):\n#   {command}\n")
        fh.write("# kernel template: <head_dim, pgen kind (0 EFQ, 1 EXPQ, 3 no-op), causal, dump, "
                 "MXFP8 Q K^T>\n")
        fh.write("# cycles per XCD = GRBM_GUI_ACTIVE / 8; MFMA busy and VALU active are per SIMD "
                 "(SQ_ACTIVE_INST_VALU is in quad-cycles, summed over the SIMD's waves)\n")
        fh.write("# VALU per score: wave instructions x 64 lanes / visible (query, key) pairs\n")
        fh.write("# co-exec: cycles in which the matrix core was busy and a VALU instruction "
                 "issued (SQ_VALU_MFMA_COEXEC_CYCLES), per SIMD\n")
        fh.write("# kernel | cycles | MFMA busy / cycles | VALU active / cycles | "
                 "(MFMA + VALU) / cycles | co-exec / cycles | VALU instr per SIMD | "
                 "MFMA instr per SIMD | VALU per score | LDS instr per SIMD | "
                 "bank-conflict cycles per LDS instr\n")
        for key in sorted(acc):
            c = acc[key]
            cyc = c["GRBM_GUI_ACTIVE"] / xcds
            mf = c["SQ_VALU_MFMA_BUSY_CYCLES"] / simds
            va = 4 * c["SQ_ACTIVE_INST_VALU"] / simds
            co = c.get("SQ_VALU_MFMA_COEXEC_CYCLES", float("nan")) / simds
            fh.write(f"{names[key]} | {cyc:.0f} | {mf / cyc:.3f} | {va / cyc:.3f} | "
                     f"{(mf + va) / cyc:.3f} | {co / cyc:.3f} | {c['SQ_INSTS_VALU'] / simds:.0f} | "
                     f"{c['SQ_INSTS_MFMA'] / simds:.0f} | {c['SQ_INSTS_VALU'] * 64 / pairs:.2f} | "
                     f"{c.get('SQ_INSTS_LDS', 0) / simds:.0f} | "
                     f"{c.get('SQ_LDS_BANK_CONFLICT', 0) / max(c.get('SQ_INSTS_LDS', 0), 1):.4f}\n")
    print(open(out).read())


def main():
    if sys.argv[1] == "counters":
        counters(sys.argv[2], sys.argv[3], " ".join(sys.argv[4:]))
        return
    if sys.argv[1] == "stats":
        stats(sys.argv[2], sys.argv[3], " ".join(sys.argv[4:]))
        return
    if sys.argv[1] == "sweep":
        sweep(sys.argv[2], sys.argv[3], " ".join(sys.argv[4:]))
        return
    import bench
    from paper_2609_09721_amd import inputs
    fetch_dir, write_dir, wl = sys.argv[2], sys.argv[3], sys.argv[4]
    out = sys.argv[5] if len(sys.argv) > 5 else os.path.join(ROOT, "profiles",
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
    with open(out, "w") as fh:
        fh.write(f"# HBM traffic of one attention launch, {wl} (EFQ), from rocprofv3 counters\n")
        fh.write("# commands (from the repository root, TMPDIR=/tmp):\n")
        fh.write("#   rocprofv3 --pmc FETCH_SIZE -d <FETCH_DIR> -o p --output-format csv -- "
                 "python3 bench.py --pmc-run\n")
        fh.write("#   rocprofv3 --pmc WRITE_SIZE -d <WRITE_DIR> -o p --output-format csv -- "
                 "python3 bench.py --pmc-run\n")
        fh.write(f"#   python3 -m paper_2609_09721_amd.profsum traffic <FETCH_DIR> <WRITE_DIR> {wl}\n")
        fh.write(f"# attention dispatches {na}, copy dispatches {nc}; copy size {bench.COPY_BYTES} B\n")
        fh.write(f"fetch_counter_attn = {fa:.1f}\nfetch_counter_copy = {fc:.1f}\n")
        fh.write(f"write_counter_attn = {wa:.1f}\nwrite_counter_copy = {wc:.1f}\n")
        fh.write(f"fetch_scale_bytes_per_unit = {kf:.4f}\nwrite_scale_bytes_per_unit = {kw:.4f}\n")
        fh.write(f"read_bytes_per_launch = {rd:.0f}\nwrite_bytes_per_launch = {wb:.0f}\n")
        fh.write(f"algorithmic_bytes_per_launch = {algo}\n")
        fh.write(f"traffic_bytes_per_launch = {rd + wb:.0f}\n")
        fh.write(f"kernel_hash = {bench.kernel_hash()}\n")
    print(open(out).read())


if __name__ == "__main__":
    main()
