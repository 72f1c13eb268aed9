"""rocprofv3 runs and summaries for the elastic-ViT forward (ViT-B/16, bf16,
batch 256, one DN mode, mode 0 by default).

    PYTHONPATH=<repo> python -m paper_2609_10018_amd.pmc --out <dir> [--mode K]

runs four profiled passes of ``bench.py`` (each a child process under its own
time limit) and writes ``summary.md`` and ``traffic.json`` into ``--out``:

1. ``--kernel-trace --stats``: per-dispatch durations; ``bench.py`` also
   writes the library's algorithmic work per kernel class (``work.json``).
2. ``--pmc FETCH_SIZE``  3. ``--pmc WRITE_SIZE``: L2-to-fabric kilobytes per
   dispatch.  Both counters are scaled by what they read for a plain copy of
   known size (``bench.py --copy-probe``: out = in * 1 over 1 GiB of fp32),
   so the figures are bytes.
4. ``--pmc SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE``: matrix-core busy
   fraction per kernel class.

Dispatches are assigned to the library's kernel classes (patch, ln, qkv,
attn, proj, fc1, fc2, head) from their kernel names and order in the forward;
one class launch may be two dispatches (the GEMM's whole-rounds launch and
its tail launch), so per-launch figures sum over a class's consecutive
dispatches.
"""
from __future__ import annotations

import argparse
import csv
import glob
import json
import os
import re
import subprocess
import sys
from collections import defaultdict

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")
COPY_PROBE_BYTES = 1 << 30          # bench.py --copy-probe: reads and writes this many bytes
EPI_CLASS = {"0": "qkv", "1": "fc1", "3": "head", "4": "patch"}  # Epi 2 (residual): proj or fc2
CLASSES = ["patch", "ln", "qkv", "attn", "proj", "fc1", "fc2", "head"]

TRACE_ARGS = ["--steps", "20", "--warmup", "3", "--copy-probe"]
PMC_ARGS = ["--steps", "2", "--warmup", "1", "--copy-probe"]
# Published MI355X peaks the roofline column prices against: dense bf16 MFMA
# and HBM3E bandwidth.
PEAK_BF16_FLOPS = 2.5e15
PEAK_HBM_BYTES = 8.0e12
PASSES = {
    "fetch": ["FETCH_SIZE"],
    "write": ["WRITE_SIZE"],
    "mfma": ["SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE"],
}


def log(msg: str) -> None:
    print(f"[pmc] {msg}", flush=True)


def classify(names):
    """Kernel class of each dispatch, given the kernel names in dispatch order."""
    out, last = [], None
    for n in names:
        if "gemm_bf16_kernel" in n or "gemm_f32_kernel" in n or "gemm_bf16_persistent" in n:
            m = re.search(r"\(elasto::Epi\)(\d)", n)
            e = m.group(1) if m else "?"
            if e == "2":
                # The residual GEMM after attention is the projection, after fc1 it is fc2.
                c = last if last in ("proj", "fc2") else ("proj" if last == "attn" else "fc2")
            else:
                c = EPI_CLASS.get(e, "other")
        elif "attention" in n:
            c = "attn"
        elif "layernorm" in n:
            c = "ln"
        elif "FillFunctor" in n:
            c = "mark"
        elif "MulFunctor" in n:
            c = "copy"
        elif "reduce_kernel" in n:
            c = "read"
        else:
            c = "other"
        out.append(c)
        last = c
    return out


def after_mark(names, values):
    """The dispatches after the last marker (bench.py --profile-mode launches
    one before its forwards, so the handle's create-time tuning forwards are
    left out); all of them when there is none."""
    cls = classify(names)
    marks = [i for i, c in enumerate(cls) if c == "mark"]
    i0 = marks[-1] + 1 if marks else 0
    return names[i0:], values[i0:]


def launches(classes):
    """Maximal runs of one class: (class, [dispatch indices])."""
    runs = []
    for i, c in enumerate(classes):
        if runs and runs[-1][0] == c:
            runs[-1][1].append(i)
        else:
            runs.append((c, [i]))
    return runs


def read_trace(d):
    f = glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True)[0]
    rows = sorted(csv.DictReader(open(f)), key=lambda r: int(r["Dispatch_Id"]))
    names = [r["Kernel_Name"] for r in rows]
    dur = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3 for r in rows]  # us
    return names, dur


def read_counters(d):
    """Per dispatch (in dispatch order): name and {counter: value}."""
    f = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0]
    disp = {}
    for r in csv.DictReader(open(f)):
        key = (r["Process_Id"], int(r["Dispatch_Id"]))
        e = disp.setdefault(key, {"name": r["Kernel_Name"], "c": defaultdict(float)})
        e["c"][r["Counter_Name"]] += float(r["Counter_Value"])
    keys = sorted(disp)
    return [disp[k]["name"] for k in keys], [disp[k]["c"] for k in keys]


def simd_count(d):
    for f in glob.glob(os.path.join(d, "**", "*agent_info.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if r.get("Agent_Type") == "GPU":
                return int(r["Simd_Count"])
    return 1024


def per_launch(classes, values):
    """Per class: (number of launches, mean per launch of the summed values)."""
    acc = defaultdict(lambda: [0, 0.0])
    for c, idx in launches(classes):
        acc[c][0] += 1
        acc[c][1] += sum(values[i] for i in idx)
    return {c: (n, s / n) for c, (n, s) in acc.items()}


def run_pass(out, tag, rocprof_args, bench_args, limit):
    d = os.path.join(out, tag)
    cmd = ["timeout", "-s", "KILL", str(limit), "rocprofv3", *rocprof_args, "-f", "csv",
           "-d", d, "-o", "run", "--", sys.executable, BENCH, *bench_args]
    log(f"pass {tag}: {' '.join(cmd)}")
    env = dict(os.environ, TMPDIR="/tmp")
    with open(os.path.join(out, f"{tag}.log"), "w") as lf:
        r = subprocess.run(cmd, cwd="/tmp", env=env, stdout=lf, stderr=subprocess.STDOUT)
    log(f"pass {tag}: exit {r.returncode}")
    if r.returncode != 0:
        raise SystemExit(f"rocprofv3 pass {tag} failed with exit code {r.returncode}")
    return d, cmd


def _portable(cmd, extra_roots=()):
    """A command as text, with the checkout's absolute paths shown as <repo>
    (the checkout the command ran in: the directory of its bench.py)."""
    roots = {ROOT} | set(extra_roots) | {os.path.dirname(a) for a in cmd if a.endswith("/bench.py")}
    text = " ".join(cmd)
    for r in sorted(roots, key=len, reverse=True):
        text = text.replace(r, "<repo>")
    return text


def summarize(out, cmds, mode):
    work = json.load(open(os.path.join(out, "work.json")))
    names, dur = after_mark(*read_trace(os.path.join(out, "trace")))
    cls = classify(names)
    t_launch = per_launch(cls, dur)

    fetch_n, fetch_c = after_mark(*read_counters(os.path.join(out, "fetch")))
    write_n, write_c = after_mark(*read_counters(os.path.join(out, "write")))
    mfma_n, mfma_c = after_mark(*read_counters(os.path.join(out, "mfma")))
    simds = simd_count(os.path.join(out, "mfma"))

    def calibrated(names_, cvals, counter):
        c_ = classify(names_)
        vals = [v[counter] * 1024.0 for v in cvals]          # KiB -> bytes
        copies = [vals[i] for i, c in enumerate(c_) if c == "copy"]
        if not copies:
            raise SystemExit("no copy-probe dispatch found for calibration")
        scale = COPY_PROBE_BYTES / (sum(copies) / len(copies))
        return per_launch(c_, [v * scale for v in vals]), scale, sum(copies) / len(copies)

    rd, rd_scale, rd_copy = calibrated(fetch_n, fetch_c, "FETCH_SIZE")
    wr, wr_scale, wr_copy = calibrated(write_n, write_c, "WRITE_SIZE")
    # Second calibration of the fetch counter: a read-only probe (a sum over
    # the same 1 GiB), whose fetch is all it moves.
    fc_ = classify(fetch_n)
    reads = [sum(fetch_c[i]["FETCH_SIZE"] * 1024.0 for i in idx)
             for c_, idx in launches(fc_) if c_ == "read"]
    rd_read_scale = COPY_PROBE_BYTES / (sum(reads) / len(reads)) if reads else None
    mc = classify(mfma_n)
    busy = per_launch(mc, [v["SQ_VALU_MFMA_BUSY_CYCLES"] for v in mfma_c])
    # GRBM_GUI_ACTIVE comes summed over the 8 XCDs; each XCD counts the same cycles.
    active = per_launch(mc, [v["GRBM_GUI_ACTIVE"] / 8.0 for v in mfma_c])

    rows, table = [], {}
    for c in CLASSES:
        if c not in t_launch:
            continue
        n, us = t_launch[c]
        wk = work["classes"][c]
        flops, algo_b = wk["flops_per_launch"], wk["bytes_per_launch"]
        hbm = rd[c][1] + wr[c][1] if c in rd and c in wr else None
        util = busy[c][1] / (active[c][1] * simds) if c in busy and active[c][1] > 0 else None
        e = {"launches": n, "avg_us": us, "flops": flops, "algo_bytes": algo_b,
             "tflops": flops / us * 1e-6 if flops else None, "gbs": algo_b / us * 1e-3,
             "fetch_bytes": rd.get(c, (0, None))[1], "write_bytes": wr.get(c, (0, None))[1],
             "hbm_bytes": hbm, "mfma_util": util,
             # Roofline time: the larger of the FLOPs at the bf16 peak and the
             # algorithmic bytes at the HBM peak; frac = that / measured time.
             "roofline_frac": max(flops / PEAK_BF16_FLOPS, algo_b / PEAK_HBM_BYTES) / (us * 1e-6),
             "roofline_bound": "mfma" if flops / PEAK_BF16_FLOPS >= algo_b / PEAK_HBM_BYTES
             else "hbm"}
        table[c] = e
        rows.append(
            f"| {c} | {n} | {us:.1f} | "
            + (f"{e['tflops']:.0f} TF/s" if flops else "-") + f" | {e['gbs']:.0f} GB/s | "
            + (f"{100 * util:.1f}%" if util is not None else "-") + " | "
            + f"{e['roofline_frac']:.2f} ({e['roofline_bound']}) | "
            + f"{algo_b / 1e6:.1f} | "
            + (f"{e['fetch_bytes'] / 1e6:.1f} | {e['write_bytes'] / 1e6:.1f} | {hbm / algo_b:.2f}"
               if hbm is not None else "- | - | -") + " |")

    dom = work["dominant"]
    traffic = {
        "workload": f"elastic ViT-B/16 forward, DN mode {mode}, batch 256, bf16",
        "kernel_class": dom,
        "source_hash": work["source_hash"],
        "hbm_bytes_per_launch": table[dom]["hbm_bytes"],
        "fetch_bytes_per_launch": table[dom]["fetch_bytes"],
        "write_bytes_per_launch": table[dom]["write_bytes"],
        "algorithmic_bytes_per_launch": table[dom]["algo_bytes"],
        "calibration": {"copy_bytes": COPY_PROBE_BYTES, "fetch_scale": rd_scale,
                        "write_scale": wr_scale, "fetch_copy_bytes_raw": rd_copy,
                        "write_copy_bytes_raw": wr_copy,
                        "fetch_scale_read_probe": rd_read_scale},
        "classes": table,
        "commands": {k: _portable(v) for k, v in cmds.items()},
    }
    json.dump(traffic, open(os.path.join(out, "traffic.json"), "w"), indent=1)

    md = [
        f"# Kernel classes of the elastic ViT-B/16 forward — bf16, batch 256, DN mode {mode}",
        "",
        "Commands (GPU box, run from `/tmp` with `TMPDIR=/tmp`; committed files only):",
        "",
        "    PYTHONPATH=<repo> " + _portable(
            ["python", "-m", "paper_2609_10018_amd.pmc", "--out", out, "--mode", str(mode)],
            {os.path.dirname(a) for c in cmds.values() for a in c if a.endswith("/bench.py")}),
        "",
        "which runs:",
        "",
    ]
    md += [f"    {_portable(v)}" for v in cmds.values()]
    md += [
        "",
        f"Per launch of each kernel class (a GEMM class launch can be two dispatches: whole "
        f"rounds of 256x256 tiles, then the tail rows). Durations from the kernel trace "
        f"({sum(n for n, _ in t_launch.values())} class launches). MFMA util = "
        f"SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE x {simds} SIMDs). Fetch / write = "
        f"FETCH_SIZE / WRITE_SIZE scaled by the copy probe (1 GiB read + 1 GiB written; "
        f"raw counters read {rd_copy / 2**30:.3f} GiB and {wr_copy / 2**30:.3f} GiB, "
        f"scales {rd_scale:.3f} and {wr_scale:.3f}; a read-only probe, a sum over the same "
        f"1 GiB, gives a fetch scale of "
        + (f"{rd_read_scale:.3f}" if rd_read_scale else "n/a") +
        "). Ratio = (fetch + write) / algorithmic bytes. Roofline frac = max(FLOPs / "
        "2.5 PFLOP/s, algorithmic bytes / 8 TB/s) / time, with the bound that sets it.",
        "",
        "| class | launches | avg µs | achieved (algorithmic FLOP) | algorithmic bytes / time "
        "| MFMA util | roofline frac | algorithmic MB | fetch MB | write MB | ratio |",
        "|---|---|---|---|---|---|---|---|---|---|---|",
        *rows,
        "",
        f"Dominant class: **{dom}**, {table[dom]['avg_us']:.1f} µs per launch in the trace; "
        f"bench.py's HIP-event timing in the traced run: {work['dominant_avg_us']:.1f} µs.",
        f"Source hash of the kernels profiled: `{work['source_hash']}`.",
        "",
    ]
    stats = glob.glob(os.path.join(out, "trace", "**", "*kernel_stats.csv"), recursive=True)
    if stats:
        md += ["rocprofv3 `--stats` per kernel name (trace pass, every dispatch of the run):", "",
               "| kernel | calls | avg µs | min µs | max µs | share |", "|---|---|---|---|---|---|"]
        for r in csv.DictReader(open(stats[0])):
            name = re.sub(r"\(elasto::\(anonymous namespace\)::\w+\)$", "", r["Name"])
            name = name.replace("elasto::(anonymous namespace)::", "").replace("void ", "")
            md.append(f"| `{name[:110]}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                      f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                      f"{float(r['Percentage']):.1f}% |")
        md.append("")
    open(os.path.join(out, "summary.md"), "w").write("\n".join(md))
    log(f"wrote {out}/summary.md and traffic.json")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=os.path.join(ROOT, "pmc_out"))
    ap.add_argument("--summarize-only", action="store_true")
    ap.add_argument("--mode", type=int, default=0, help="DN mode to profile")
    args = ap.parse_args()
    out = os.path.abspath(args.out)
    os.makedirs(out, exist_ok=True)
    cmds = {}
    if not args.summarize_only:
        _, cmds["trace"] = run_pass(out, "trace", ["--kernel-trace", "--stats"],
                                    TRACE_ARGS + ["--profile-mode", str(args.mode),
                                                  "--work-out", os.path.join(out, "work.json")],
                                    300)
        for tag, counters in PASSES.items():
            _, cmds[tag] = run_pass(out, tag, ["--pmc", *counters],
                                    PMC_ARGS + ["--profile-mode", str(args.mode)], 180)
        json.dump(cmds, open(os.path.join(out, "commands.json"), "w"))
    else:
        cmds = json.load(open(os.path.join(out, "commands.json")))
    summarize(out, cmds, args.mode)


if __name__ == "__main__":
    main()
