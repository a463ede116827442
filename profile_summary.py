#!/usr/bin/env python3
"""Summarise rocprofv3 output of bench.py into profiles/.

Inputs (directories written by the commands below, CSV output format):
  TRACE   rocprofv3 --kernel-trace --stats --output-format csv -d TRACE -o run --
              python3 bench.py DECODE_ONLY --steps K --warmup W
  FETCH   rocprofv3 --pmc FETCH_SIZE --output-format csv -d FETCH -o run --
              python3 bench.py DECODE_ONLY --steps K --warmup W --calibrate-copy 1024
  WRITE   the same with --pmc WRITE_SIZE
  with DECODE_ONLY = the flags in DECODE_ONLY below (the EAT decode alone)

Writes profiles/<name>.md (kernel table, the dominant kernel's per-launch
duration and HBM traffic) and profiles/<name>.traffic.txt (key: value lines
that bench.py reads for roofline.traffic, with the SHA-1 of the expert
kernel source they were measured on).

    python profile_summary.py --trace T --fetch F --write W --bench-json B.json --name NAME

The traffic file records the batch, timed steps and warm-up steps of the
run; bench.py reports the figure only for a run with the same three.

Prefill (MFMA-bound) summary of the wide tile kernels, from a trace of

  TRACE   rocprofv3 --kernel-trace --stats --output-format csv -d TRACE -o run --
              python3 bench.py --only-prefill LAYER --modes topk

    python profile_summary.py --prefill --trace T --bench-json B.json --name NAME

One more decode layer (per-step kernel breakdown of bench's decode_layers
workload, e.g. the fine-grained layer's 256-token EAT decode), from a trace of

  TRACE   rocprofv3 --kernel-trace --stats --output-format csv -d TRACE -o run --
              python3 bench.py --only-decode-layer LAYER --modes eat

    python profile_summary.py --layer-decode --trace T --bench-json B.json --name NAME

Stacked-layer decode (per-layer kernel breakdown), from a trace of

  TRACE   rocprofv3 --kernel-trace --stats --output-format csv -d TRACE -o run --
              python3 bench.py --only-stack --modes eat --stack-steps 128

    python profile_summary.py --stack --trace T --bench-json B.json --name NAME
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import statistics

ROOT = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCE = os.path.join(ROOT, "paper_2609_33614_amd", "csrc", "expert.hip")
DOMINANT = "stream_kernel<true"
DECODE_ONLY = ("--no-sweep --no-cpu-baseline --no-prefill --no-stack --no-wide-experts --no-decode-layers "
               "--no-share --no-trajectory --modes eat")
COPY = "__amd_rocclr_copyBuffer"


def source_sha1() -> str:
    return hashlib.sha1(open(KERNEL_SOURCE, "rb").read()).hexdigest()


def counter_rows(d):
    return list(csv.DictReader(open(os.path.join(d, "run_counter_collection.csv"))))


def copy_factor(rows, mib: int, expect_bytes: float) -> float:
    """Bytes a known-size copy really moves / what the counter reports for it."""
    vals = [float(r["Counter_Value"]) * 1024 for r in rows
            if COPY in r["Kernel_Name"] and int(r["Grid_Size"]) >= 65536]
    assert vals, "no calibration copy dispatch found"
    return expect_bytes / statistics.mean(vals)


BF16_PEAK_TFLOPS = 2500.0


def prefill_summary(args) -> int:
    """Per-launch duration and achieved bf16 TFLOP/s of the wide tile kernels
    (gated up/gate and plain down) of one traced prefill configuration."""
    bench = json.loads(open(args.bench_json).read().strip().splitlines()[-1])
    pf = bench["prefill"][0]
    modes = [m for m in ("eat", "topk", "topp") if m in pf]
    assert len(modes) == 1, "trace one routing mode at a time"
    r = pf[modes[0]]
    T, d, F = pf["tokens"], pf["d_model"], pf["d_ffn"]
    sk = r["mean_activated_experts"] * T
    stats = list(csv.DictReader(open(os.path.join(args.trace, "run_kernel_stats.csv"))))
    trace = list(csv.DictReader(open(os.path.join(args.trace, "run_kernel_trace.csv"))))
    trace.sort(key=lambda x: int(x["Start_Timestamp"]))

    def launches(key):
        return [(int(x["End_Timestamp"]) - int(x["Start_Timestamp"])) / 1e3 for x in trace if key in x["Kernel_Name"]]

    rows = []
    shared = pf.get("d_shared", 0)
    per_fwd = 2 if shared else 1          # routed (+ always-on) launches per forward
    # the kernel name carries <gated, packed-weights>
    for key, label, fl, ev_us in (("wide_kernel<true,", "up/gate (gated)", 4.0 * d * F * sk, r["up_gate"]["us"]),
                                  ("wide_kernel<false,", "down (plain)", 2.0 * d * F * sk, r["down"]["us"])):
        durs = launches(key)
        routed = durs[0::per_fwd][-args.reps:]
        us = statistics.mean(routed)
        rows.append((key, label, len(durs), us, fl, ev_us))
    md = os.path.join(ROOT, "profiles", args.name + ".md")
    with open(md, "w") as f:
        f.write(f"# {args.name}\n\n")
        f.write(f"Workload: {pf['workload']}, {T} tokens, d_model {d}, {pf['experts']} experts of width {F}"
                f"{', always-on expert of width ' + str(shared) if shared else ''}, K={pf['top_k']}, "
                f"{modes[0]} routing from zero accounts (mean {r['mean_activated_experts']} experts per token), "
                f"MI355X.\n\n")
        f.write("Commands (from the repository root):\n\n```\n")
        f.write(f"rocprofv3 --kernel-trace --stats --output-format csv -d TRACE -o run -- "
                f"python3 bench.py --only-prefill {pf['workload'].split()[0]} --modes {modes[0]}\n")
        f.write(f"python3 profile_summary.py --prefill --trace TRACE --bench-json TRACED_BENCH.json --name {args.name}\n```\n\n")
        f.write("## Kernel time (rocprofv3 --stats, whole traced run incl. warm-up)\n\n")
        f.write("| kernel | calls | avg us | % time |\n|---|---|---|---|\n")
        for x in stats[:10]:
            name = x["Name"].replace("(anonymous namespace)::", "").split("(")[0]
            f.write(f"| `{name}` | {x['Calls']} | {float(x['AverageNs']) / 1e3:.2f} | {float(x['Percentage']):.1f} |\n")
        f.write(f"\n## Routed expert GEMMs (last {args.reps} launches of each)\n\n")
        f.write("| kernel | stage | avg us (trace) | us (bench events) | algorithmic GFLOP | TFLOP/s | % of 2.5 PF bf16 |\n")
        f.write("|---|---|---|---|---|---|---|\n")
        for key, label, n, us, fl, ev_us in rows:
            f.write(f"| `{key}` | {label} | {us:.1f} | {ev_us:.1f} | {fl / 1e9:.1f} | {fl / us / 1e6:.1f} | "
                    f"{fl / us / 1e6 / BF16_PEAK_TFLOPS * 100:.1f} |\n")
        f.write("\nAlgorithmic flops: up/gate 4 d F sum(k), down 2 d F sum(k), sum(k) = the call's "
                "(token, expert) assignments; padding rows of partly filled tiles are not counted.\n")
    print(open(md).read())
    return 0


def per_kernel(trace_dir):
    """Durations (us) of every eat:: kernel launch of a trace, in launch order."""
    trace = list(csv.DictReader(open(os.path.join(trace_dir, "run_kernel_trace.csv"))))
    trace.sort(key=lambda x: int(x["Start_Timestamp"]))
    per = {}
    for x in trace:
        name = x["Kernel_Name"].replace("(anonymous namespace)::", "").split("(")[0].replace("void ", "")
        if name.startswith("eat::") and "pack_kernel" not in name and "reset_accounts" not in name:
            per.setdefault(name, []).append((int(x["End_Timestamp"]) - int(x["Start_Timestamp"])) / 1e3)
    return per


def layer_decode_summary(args) -> int:
    """Per-step kernel breakdown of one traced decode_layers workload (one
    routing mode), with the gated expert kernel's achieved MFMA rate and
    weight bandwidth on its algorithmic flops and bytes."""
    bench = json.loads(open(args.bench_json).read().strip().splitlines()[-1])
    dl = bench["decode_layers"][0]
    modes = [m for m in ("eat", "topk", "topp") if m in dl]
    assert len(modes) == 1, "trace one routing mode at a time"
    r = dl[modes[0]]
    B, steps, d, F = dl["batch"], dl["steps"], dl["d_model"], dl["d_ffn"]
    warm = args.warmup
    per = per_kernel(args.trace)
    md = os.path.join(ROOT, "profiles", args.name + ".md")
    rows = []
    for name, durs in per.items():
        n_per = len(durs) / (steps + warm)
        timed = durs[-int(round(n_per * steps)):] if n_per > 0 else durs
        avg = statistics.mean(timed)
        rows.append((avg * n_per, name, n_per, avg))
    up = [x for x in rows if x[1].startswith("eat::stream_kernel<true") or x[1].startswith("eat::wide_kernel<true")]
    sk = r["mean_activated_experts"] * B
    with open(md, "w") as f:
        f.write(f"# {args.name}\n\n")
        f.write(f"Workload: {dl['workload']}, batch {B}, d_model {d}, {dl['experts']} experts of width {F}"
                f"{', always-on expert of width ' + str(dl['d_shared']) if dl.get('d_shared') else ''}, "
                f"K={dl['top_k']}, {modes[0]} routing, {steps} timed steps after {warm} warm-up steps from zero "
                f"accounts; {r['mean_activated_experts']} experts per token, "
                f"{r['mean_experts_touched_per_step']} touched per step, MI355X.\n\n")
        f.write("Commands (from the repository root):\n\n```\n")
        f.write(f"rocprofv3 --kernel-trace --stats --output-format csv -d TRACE -o run -- "
                f"python3 bench.py --only-decode-layer {dl['workload'].split()[0]} --modes {modes[0]}\n")
        f.write(f"python3 profile_summary.py --layer-decode --trace TRACE --bench-json TRACED_BENCH.json "
                f"--name {args.name}\n```\n\n")
        f.write(f"Step time in the traced run (HIP events): {r['ms_per_step'] * 1e3:.1f} us; "
                f"{r['tokens_per_s']:.0f} tokens/s.\n\n")
        f.write("| kernel | launches per step | avg us per launch | us per step |\n|---|---|---|---|\n")
        for tot, name, n_per, avg in sorted(rows, reverse=True):
            f.write(f"| `{name}` | {n_per:.2f} | {avg:.2f} | {tot:.2f} |\n")
        f.write(f"| **sum** | | | **{sum(x[0] for x in rows):.1f}** |\n")
        if up:
            us = sum(x[0] for x in up)
            fl = 4.0 * d * F * sk
            wb = r["mean_experts_touched_per_step"] * 4.0 * d * F
            f.write(f"\nRouted up/gate per step: {us:.1f} us for {fl / 1e9:.2f} GFLOP (4 d F sum(k), "
                    f"sum(k) = {sk:.0f}) = {fl / us / 1e6:.0f} TFLOP/s = "
                    f"{fl / us / 1e6 / BF16_PEAK_TFLOPS * 100:.1f}% of the 2.5 PF bf16 peak; weights of the "
                    f"experts touched {wb / 1e6:.1f} MB = {wb / us / 1e6:.2f} TB/s.\n")
    print(open(md).read())
    return 0


def stack_summary(args) -> int:
    """Average duration of every kernel of the traced stacked-layer decode
    per launch and per layer of a timed step (16 warm-up steps, then the
    timed steps; one traced routing mode)."""
    bench = json.loads(open(args.bench_json).read().strip().splitlines()[-1])
    st = bench["stack"]
    modes = [m for m in ("eat", "topk", "topp", "eat_layerwise") if m in st]
    assert len(modes) == 1, "trace one routing mode at a time"
    r = st[modes[0]]
    layers, steps = st["layers"], st["steps"]
    # the timed steps' launches are the last ones of the kernels a step runs
    per = per_kernel(args.trace)
    total_steps = steps + 16
    md = os.path.join(ROOT, "profiles", args.name + ".md")
    with open(md, "w") as f:
        f.write(f"# {args.name}\n\n")
        f.write(f"Workload: {st['workload']}, {layers} layers, batch {st['batch']}, d_model {st['d_model']}, "
                f"{st['experts']} experts of width {st['d_ffn']}, K={st['top_k']}, {modes[0]} routing, "
                f"{steps} timed steps after 16 warm-up steps, MI355X.\n\n")
        f.write("Commands (from the repository root):\n\n```\n")
        f.write(f"rocprofv3 --kernel-trace --stats --output-format csv -d TRACE -o run -- "
                f"python3 bench.py --only-stack --modes {modes[0]} --stack-steps {steps}\n")
        f.write(f"python3 profile_summary.py --stack --trace TRACE --bench-json TRACED_BENCH.json --name {args.name}\n```\n\n")
        f.write(f"Step time in the traced run (HIP events): {r['ms_per_step'] * 1e3:.0f} us = "
                f"{r['ms_per_step'] * 1e3 / layers:.1f} us per layer; {r['tokens_per_s']:.0f} tokens/s.\n\n")
        f.write("| kernel | launches per layer and step | avg us per launch | us per layer and step |\n")
        f.write("|---|---|---|---|\n")
        rows = []
        for name, durs in per.items():
            n_per = len(durs) / (total_steps * layers)
            timed = durs[-int(round(n_per * steps * layers)):] if n_per > 0 else durs
            avg = statistics.mean(timed)
            rows.append((avg * n_per, name, n_per, avg))
        for tot, name, n_per, avg in sorted(rows, reverse=True):
            f.write(f"| `{name}` | {n_per:.2f} | {avg:.2f} | {tot:.2f} |\n")
        f.write(f"| **sum** | | | **{sum(x[0] for x in rows):.1f}** |\n")
    print(open(md).read())
    return 0


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace", required=True)
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--bench-json", required=True, help="JSON line printed by the traced bench run")
    ap.add_argument("--name", required=True)
    ap.add_argument("--copy-mib", type=int, default=1024)
    ap.add_argument("--steps", type=int, default=256, help="timed steps of the traced decode run")
    ap.add_argument("--prefill", action="store_true", help="summarise a prefill trace (wide tile kernels)")
    ap.add_argument("--reps", type=int, default=10, help="timed prefill calls in the traced run")
    ap.add_argument("--stack", action="store_true", help="summarise a stacked-layer decode trace")
    ap.add_argument("--layer-decode", action="store_true", help="summarise a decode_layers trace")
    ap.add_argument("--warmup", type=int, default=16, help="warm-up steps of the traced decode_layers run")
    args = ap.parse_args(argv)
    if args.prefill:
        return prefill_summary(args)
    if args.stack:
        return stack_summary(args)
    if args.layer_decode:
        return layer_decode_summary(args)
    assert args.fetch and args.write, "--fetch and --write are needed for the decode summary"

    bench = json.loads(open(args.bench_json).read().strip().splitlines()[-1])
    stats = list(csv.DictReader(open(os.path.join(args.trace, "run_kernel_stats.csv"))))
    trace = list(csv.DictReader(open(os.path.join(args.trace, "run_kernel_trace.csv"))))
    dom = [r for r in trace if DOMINANT in r["Kernel_Name"]]
    dom.sort(key=lambda r: int(r["Start_Timestamp"]))
    timed = dom[-args.steps:]
    dur_us = statistics.mean((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in timed)

    # counters: the copy kernel is a (split) 1 GiB read + 1 GiB write in 512 MiB dispatches
    fetch, write = counter_rows(args.fetch), counter_rows(args.write)
    copy_disp = [r for r in fetch if COPY in r["Kernel_Name"] and int(r["Grid_Size"]) >= 65536]
    per_copy = args.copy_mib * (1 << 20) * 4 / len(copy_disp)       # bytes each dispatch moves
    f_fac = copy_factor(fetch, args.copy_mib, per_copy)
    w_fac = copy_factor(write, args.copy_mib, per_copy)
    fd = [float(r["Counter_Value"]) * 1024 * f_fac for r in fetch if DOMINANT in r["Kernel_Name"]][-args.steps:]
    wd = [float(r["Counter_Value"]) * 1024 * w_fac for r in write if DOMINANT in r["Kernel_Name"]][-args.steps:]
    fetch_b, write_b = statistics.mean(fd), statistics.mean(wd)
    alg = bench["roofline"]["bytes_per_launch"]
    ev_us = bench["roofline"]["us_per_launch"]

    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    md = os.path.join(ROOT, "profiles", args.name + ".md")
    with open(md, "w") as f:
        f.write(f"# {args.name}\n\n")
        f.write(f"Workload: {bench['config']['workload']}, batch {bench['config']['batch']}, "
                f"{bench['steps']} timed steps (+{bench['warmup']} warm-up), MI355X.\n\n")
        f.write("Commands (from the repository root):\n\n```\n")
        run = (f"python3 bench.py {DECODE_ONLY} --batch {bench['config']['batch']} --steps {bench['steps']} "
               f"--warmup {bench['warmup']}")
        f.write(f"rocprofv3 --kernel-trace --stats --output-format csv -d TRACE -o run -- {run}\n")
        f.write(f"rocprofv3 --pmc FETCH_SIZE --output-format csv -d FETCH -o run -- {run} --calibrate-copy 1024\n")
        f.write(f"rocprofv3 --pmc WRITE_SIZE --output-format csv -d WRITE -o run -- {run} --calibrate-copy 1024\n")
        f.write(f"python3 profile_summary.py --trace TRACE --fetch FETCH --write WRITE "
                f"--bench-json TRACED_BENCH.json --name {args.name}\n```\n\n")
        f.write("## Kernel time (rocprofv3 --stats, whole traced run incl. warm-up)\n\n")
        f.write("| kernel | calls | avg us | % time |\n|---|---|---|---|\n")
        for r in stats[:10]:
            name = r["Name"].replace("(anonymous namespace)::", "").split("(")[0]
            f.write(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | {float(r['Percentage']):.1f} |\n")
        f.write("\n## Dominant kernel: expert up/gate (`stream_kernel<true, ...>`)\n\n")
        f.write(f"- average duration over the {len(timed)} timed launches (trace): **{dur_us:.2f} us**\n")
        f.write(f"- average duration measured in bench.py with HIP events (same run): {ev_us:.2f} us\n")
        f.write(f"- algorithmic bytes per launch (weights of the experts touched + token rows + H): "
                f"{alg / 1e6:.1f} MB -> {alg / dur_us / 1e3:.1f} GB/s = "
                f"{alg / dur_us / 1e3 / 8000 * 100:.1f}% of 8 TB/s\n")
        f.write(f"- HBM traffic per launch (FETCH_SIZE x {f_fac:.3f} + WRITE_SIZE x {w_fac:.3f}, the factors "
                f"that make a {args.copy_mib} MiB device copy read and write its size): "
                f"{fetch_b / 1e6:.1f} MB read + {write_b / 1e6:.1f} MB written = "
                f"{(fetch_b + write_b) / alg:.3f} x algorithmic\n")
    txt = os.path.join(ROOT, "profiles", args.name + ".traffic.txt")
    with open(txt, "w") as f:
        f.write(f"kernel: {DOMINANT}\n")
        f.write(f"source_sha1: {source_sha1()}\n")
        f.write(f"batch: {bench['config']['batch']}\n")
        f.write(f"steps: {len(timed)}\n")
        f.write(f"warmup: {bench['warmup']}\n")
        f.write(f"fetch_factor: {f_fac:.6f}\n")
        f.write(f"write_factor: {w_fac:.6f}\n")
        f.write(f"fetch_bytes_per_launch: {fetch_b:.0f}\n")
        f.write(f"write_bytes_per_launch: {write_b:.0f}\n")
        f.write(f"traffic_bytes_per_launch: {fetch_b + write_b:.0f}\n")
        f.write(f"algorithmic_bytes_per_launch: {alg:.0f}\n")
        f.write(f"trace_us_per_launch: {dur_us:.3f}\n")
    print(open(md).read())
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
