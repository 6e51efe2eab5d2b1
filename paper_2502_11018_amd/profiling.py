"""Measurement helpers for rocprofv3 runs of the verify path.

    python -m paper_2502_11018_amd.profiling copy --mib 1024 --reps 5
        Device-to-device copies of a known size: the reference kernel whose
        FETCH_SIZE / WRITE_SIZE readings give the scale factors of those
        counters (bytes the counter reports per byte actually moved).

    python -m paper_2502_11018_amd.profiling stats RUN_kernel_trace.csv \\
            --stats RUN_kernel_stats.csv --steps K --out profiles/NAME.md \\
            --title TITLE --command "CMD" [--include REGEX --step-end REGEX]
        Markdown summary of a `rocprofv3 --kernel-trace --stats -f csv` run of
        bench.py: per-kernel durations over the last K steps (a step ends with
        the kernel matching --step-end, by default the acceptance walk).

    python -m paper_2502_11018_amd.profiling counters --pmc RUN_counter_collection.csv ... \\
            --trace RUN_kernel_trace.csv --group LABEL=REGEX ... --out profiles/NAME.md ...
        Per kernel group, the mean per dispatch of every counter of the --pmc
        passes (MFMA flops and utilisation, FETCH_SIZE) beside the mean
        kernel duration of a --kernel-trace run of the same command.

    python -m paper_2502_11018_amd.profiling traffic \\
            --kernel-regex REGEX --fetch BENCH_fetch.csv --write BENCH_write.csv \\
            --copy-fetch COPY_fetch.csv --copy-write COPY_write.csv --copy-bytes N \\
            --label gate_up_gemm --workload llama3-8b --source FILE [FILE ...] \\
            --out profiles/NAME.md --command "CMD ..."
        HBM traffic per dispatch of the kernels whose name matches REGEX, from
        two `rocprofv3 --pmc` passes (FETCH_SIZE, then WRITE_SIZE, KiB per
        dispatch), scaled by the same counters read on the copy kernel.  The
        summary ends with one machine-readable `traffic-record:` line that
        bench.py reads; it carries the sha256 of the kernel's source files so
        that a later change of the kernel voids the record.
"""

from __future__ import annotations

import argparse
import csv
import hashlib
import os
import re
import statistics
import sys

PKG = os.path.dirname(os.path.abspath(__file__))


def source_sha256(paths) -> str:
    """sha256 over the concatenated contents of one or more source files."""
    if isinstance(paths, str):
        paths = [paths]
    h = hashlib.sha256()
    for p in paths:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _rows(path):
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def _col(row, *names):
    for n in names:
        if n in row:
            return row[n]
    raise KeyError(f"none of {names} in {list(row)}")


def counter_per_dispatch(path: str, counter: str, kernel_regex: str):
    """Mean value (KiB) of `counter` over the dispatches of matching kernels."""
    rx = re.compile(kernel_regex)
    per = {}
    for r in _rows(path):
        if _col(r, "Counter_Name") != counter:
            continue
        name = _col(r, "Kernel_Name")
        if not rx.search(name):
            continue
        key = _col(r, "Dispatch_Id", "Correlation_Id")
        per[key] = per.get(key, 0.0) + float(_col(r, "Counter_Value"))
    if not per:
        raise SystemExit(f"{path}: no {counter} rows for kernels matching {kernel_regex!r}")
    vals = list(per.values())
    return statistics.fmean(vals), len(vals)


def cmd_copy(args):
    import torch

    n = args.mib << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    src.random_(0, 255)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(args.reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(f"copied {args.reps} x {n} bytes", flush=True)


def _short(name: str) -> str:
    return re.sub(r"^void ", "", name.split("(")[0]).replace("griffin::", "")


def cmd_stats(args):
    """Per-kernel durations over the last `steps` steps (a step ends with the
    kernel matching --step-end: the acceptance walk for a verify step),
    grouped by kernel and grid, plus the library's rows of rocprofv3's own
    whole-run statistics."""
    rx = re.compile(args.include)
    end_rx = re.compile(args.step_end)
    rows = [r for r in _rows(args.trace) if rx.search(_col(r, "Kernel_Name"))]
    rows.sort(key=lambda r: int(_col(r, "Start_Timestamp")))
    ends = [int(_col(r, "End_Timestamp")) for r in rows if end_rx.search(_col(r, "Kernel_Name"))]
    skip = args.skip_last
    if len(ends) < args.steps + skip + 1:
        raise SystemExit(f"{args.trace}: fewer than {args.steps + skip + 1} steps")
    t0 = ends[-args.steps - skip - 1]
    t1 = ends[-skip - 1] if skip else ends[-1]
    win = [r for r in rows if t0 < int(_col(r, "Start_Timestamp")) <= t1]
    before = [r for r in rows if int(_col(r, "Start_Timestamp")) <= t0]
    groups = {}
    prev = _short(_col(before[-1], "Kernel_Name")) if before else ""
    for r in win:  # keyed by kernel, grid and the kernel launched before it (tells O from down)
        name = _short(_col(r, "Kernel_Name"))
        key = (name, tuple(int(_col(r, f"Grid_Size_{a}")) // int(_col(r, f"Workgroup_Size_{a}")) for a in "XYZ"),
               prev)
        groups.setdefault(key, []).append((int(_col(r, "End_Timestamp")) - int(_col(r, "Start_Timestamp"))) / 1e3)
        prev = name
    busy = sum(sum(v) for v in groups.values()) / args.steps
    span = (int(_col(win[-1], "End_Timestamp")) - int(_col(win[0], "Start_Timestamp"))) / 1e3 / args.steps
    out = [f"# {args.title}", "", "Command:", "", "```", args.command, "```", "",
           (f"Last {args.steps} steps of the run" if not skip else
            f"{args.steps} steps of the run, ending {skip} steps before its last") +
           f": kernel busy time {busy:.1f} us per step, "
           f"first-kernel-start to last-kernel-end {span:.1f} us per step.", "",
           "| kernel | workgroups | after | launches/step | avg us | min us | max us | us/step |",
           "|---|---|---|---:|---:|---:|---:|---:|"]
    for (name, grid, after), v in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        out.append(f"| `{name}` | {grid[0]}x{grid[1]}x{grid[2]} | `{after}` | {len(v) / args.steps:g} | "
                   f"{statistics.fmean(v):.2f} | {min(v):.2f} | {max(v):.2f} | {sum(v) / args.steps:.1f} |")
    if args.stats:
        out += ["", "rocprofv3 `--stats` rows of the library's kernels (whole run, including warm-up and the "
                "chain steps that build the planted-tree pool):", "",
                "| kernel | calls | avg us | min us | max us | total ms |", "|---|---:|---:|---:|---:|---:|"]
        for r in sorted(_rows(args.stats), key=lambda r: -float(_col(r, "TotalDurationNs"))):
            if not rx.search(_col(r, "Name", "KernelName")):
                continue
            out.append(f"| `{_short(_col(r, 'Name', 'KernelName'))}` | {_col(r, 'Calls')} | "
                       f"{float(_col(r, 'AverageNs')) / 1e3:.2f} | {float(_col(r, 'MinNs')) / 1e3:.2f} | "
                       f"{float(_col(r, 'MaxNs')) / 1e3:.2f} | {float(_col(r, 'TotalDurationNs')) / 1e6:.2f} |")
    if args.note:
        out += ["", args.note]
    with open(args.out, "w") as f:
        f.write("\n".join(out) + "\n")
    print("\n".join(out))


def cmd_traffic(args):
    fk, nf = counter_per_dispatch(args.fetch, "FETCH_SIZE", args.kernel_regex)
    wk, nw = counter_per_dispatch(args.write, "WRITE_SIZE", args.kernel_regex)
    cf, _ = counter_per_dispatch(args.copy_fetch, "FETCH_SIZE", args.copy_regex)
    cw, _ = counter_per_dispatch(args.copy_write, "WRITE_SIZE", args.copy_regex)
    sf = args.copy_bytes / (cf * 1024.0)   # true bytes per counted byte
    sw = args.copy_bytes / (cw * 1024.0)
    fetch = fk * 1024.0 * sf
    write = wk * 1024.0 * sw
    sha = source_sha256(args.source)
    rel = ",".join(os.path.relpath(x, os.path.dirname(PKG)) for x in args.source)
    out = [f"# HBM traffic per dispatch: {args.label} ({args.workload})", "",
           "Commands (each a separate rocprofv3 pass):", "", "```", args.command, "```", "",
           f"* kernels matching `{args.kernel_regex}`: {nf} dispatches with FETCH_SIZE, {nw} with WRITE_SIZE",
           f"* FETCH_SIZE {fk:.1f} KiB/dispatch, WRITE_SIZE {wk:.1f} KiB/dispatch (raw)",
           f"* copy kernel ({args.copy_bytes} bytes read and written): FETCH_SIZE {cf:.1f} KiB, "
           f"WRITE_SIZE {cw:.1f} KiB -> scale {sf:.4f} (fetch), {sw:.4f} (write)",
           f"* scaled: fetch {fetch / 1e6:.2f} MB, write {write / 1e6:.2f} MB, total {(fetch + write) / 1e6:.2f} MB "
           f"per dispatch",
           f"* kernel sources `{rel}` sha256 {sha}", "",
           f"traffic-record: label={args.label} workload={args.workload} fetch_bytes={fetch:.0f} "
           f"write_bytes={write:.0f} source={rel} sha256={sha}"]
    with open(args.out, "w") as f:
        f.write("\n".join(out) + "\n")
    print("\n".join(out))


def _mean_duration_us(trace_csv: str, rx):
    durs = [(int(_col(r, "End_Timestamp")) - int(_col(r, "Start_Timestamp"))) / 1e3
            for r in _rows(trace_csv) if rx.search(_col(r, "Kernel_Name"))]
    return (statistics.fmean(durs), len(durs)) if durs else (None, 0)


def cmd_counters(args):
    """Per kernel group: the mean per dispatch of every counter in the given
    rocprofv3 --pmc CSVs, with the mean kernel-trace duration of the same
    group; MfmaFlopsBF16 becomes TFLOP/s against the bf16 dense peak and
    FETCH_SIZE (KiB) bytes scaled by the copy kernel's reading."""
    scale = 1.0
    if args.copy_fetch:
        cf, _ = counter_per_dispatch(args.copy_fetch, "FETCH_SIZE", args.copy_regex)
        scale = args.copy_bytes / (cf * 1024.0)
    out = [f"# {args.title}", "", "Commands (each a separate rocprofv3 pass):", "", "```", args.command, "```", "",
           "| kernel group | dispatches | mean us (trace) | counter | per dispatch | derived |",
           "|---|---:|---:|---|---:|---|"]
    for g in args.group:
        label, regex = g.split("=", 1)
        rx = re.compile(regex)
        dur, nd = _mean_duration_us(args.trace, rx)
        for path in args.pmc:
            names = sorted({_col(r, "Counter_Name") for r in _rows(path) if rx.search(_col(r, "Kernel_Name"))})
            for name in names:
                val, n = counter_per_dispatch(path, name, regex)
                derived = ""
                if name == "MfmaFlopsBF16" and dur:
                    derived = f"{val / (dur * 1e-6) / 1e12:.1f} TFLOP/s = {val / (dur * 1e-6) / 2.5e15:.1%} of 2.5 PFLOP/s"
                elif name == "MfmaUtil":
                    derived = "% of SIMD cycles with the MFMA unit busy"
                elif name == "FETCH_SIZE" and dur:
                    b = val * 1024.0 * scale
                    derived = f"{b / 1e6:.2f} MB (x{scale:.3f}), {b / (dur * 1e-6) / 1e9:.0f} GB/s = {b / (dur * 1e-6) / 8e12:.1%} of 8 TB/s"
                shown = f"{val:.4g}" if name != "MfmaFlopsBF16" else f"{val / 1e9:.2f} GFLOP"
                out.append(f"| {label} | {n} | {dur:.2f} | {name} | {shown} | {derived} |" if dur else
                           f"| {label} | {n} | — | {name} | {shown} | {derived} |")
    if args.note:
        out += ["", args.note]
    with open(args.out, "w") as f:
        f.write("\n".join(out) + "\n")
    print("\n".join(out))


def read_traffic_record(profiles_dir: str, label: str, workload: str, repo_root: str):
    """Scaled HBM bytes per dispatch from a committed summary, or None when
    there is none or the kernel source changed since the counters were taken."""
    if not os.path.isdir(profiles_dir):
        return None
    for fn in sorted(os.listdir(profiles_dir)):
        if not fn.endswith(".md"):
            continue
        with open(os.path.join(profiles_dir, fn)) as f:
            for line in f:
                if not line.startswith("traffic-record:"):
                    continue
                kv = dict(t.split("=", 1) for t in line.split()[1:])
                if kv.get("label") != label or kv.get("workload") != workload:
                    continue
                srcs = [os.path.join(repo_root, x) for x in kv["source"].split(",")]
                if not all(os.path.exists(x) for x in srcs) or source_sha256(srcs) != kv["sha256"]:
                    return None
                return float(kv["fetch_bytes"]) + float(kv["write_bytes"])
    return None


def main(argv=None):
    ap = argparse.ArgumentParser(prog="python -m paper_2502_11018_amd.profiling")
    sub = ap.add_subparsers(dest="cmd", required=True)
    c = sub.add_parser("copy")
    c.add_argument("--mib", type=int, default=1024)
    c.add_argument("--reps", type=int, default=5)
    s = sub.add_parser("stats")
    s.add_argument("trace", help="RUN_kernel_trace.csv")
    s.add_argument("--stats", default="", help="RUN_kernel_stats.csv")
    s.add_argument("--steps", type=int, required=True)
    s.add_argument("--include", default="griffin::")
    s.add_argument("--step-end", default="accept_kernel", help="regex of the kernel that ends a step")
    s.add_argument("--skip-last", type=int, default=0,
                   help="steps at the end of the run left out of the window (e.g. a later profiling pass)")
    s.add_argument("--out", required=True)
    s.add_argument("--title", required=True)
    s.add_argument("--command", required=True)
    s.add_argument("--note", default="")
    k = sub.add_parser("counters")
    k.add_argument("--pmc", nargs="+", required=True, help="rocprofv3 --pmc counter_collection CSVs")
    k.add_argument("--trace", required=True, help="kernel_trace CSV of the same command (durations)")
    k.add_argument("--group", nargs="+", required=True, help="LABEL=REGEX of kernel names")
    k.add_argument("--copy-fetch", default="")
    k.add_argument("--copy-regex", default="copy|Copy")
    k.add_argument("--copy-bytes", type=int, default=1 << 30)
    k.add_argument("--title", required=True)
    k.add_argument("--command", required=True)
    k.add_argument("--note", default="")
    k.add_argument("--out", required=True)
    t = sub.add_parser("traffic")
    t.add_argument("--kernel-regex", required=True)
    t.add_argument("--copy-regex", default="copy|Copy")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--copy-fetch", required=True)
    t.add_argument("--copy-write", required=True)
    t.add_argument("--copy-bytes", type=int, required=True)
    t.add_argument("--label", required=True)
    t.add_argument("--workload", required=True)
    t.add_argument("--source", required=True, nargs="+", help="kernel source files (hashed together)")
    t.add_argument("--out", required=True)
    t.add_argument("--command", required=True)
    args = ap.parse_args(argv)
    {"copy": cmd_copy, "stats": cmd_stats, "counters": cmd_counters, "traffic": cmd_traffic}[args.cmd](args)


if __name__ == "__main__":
    main(sys.argv[1:])
