"""Summaries of rocprofv3 output for the decode kernel (text for profiles/).

Two modes, both reading rocprofv3 CSV output (``--output-format csv``):

  trace    kernel-trace + stats of a bench.py run: the per-kernel table and the
           dispatches of the timed decode launches, matched to the bench's own
           HIP-event launch times (from its JSON line).
  traffic  two counter runs of the same command, one with --pmc FETCH_SIZE and
           one with --pmc WRITE_SIZE, that also ran bench.py --copy-probe MIB: the
           counters of that plain elementwise copy (MIB MiB read and written)
           give the scale from counter units to bytes, which is applied to the
           timed headline dispatch. Prints a JSON record for bench.py.

The kernel source hash ties a traffic record to the kernel it was taken on;
bench.py reports traffic only when the hash matches the current source.
"""
import argparse
import csv
import glob
import hashlib
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
KERNEL = "k_decode_persistent"
COPY_KERNEL = "neg"      # torch.neg over float32: reads and writes MIB MiB once
MARKER_KERNEL = "sigmoid"  # bench.py runs a one-element sigmoid right before each timed launch


def kernel_source_hash():
    h = hashlib.sha256()
    for f in ("ee_kernels.hip", "ee_internal.h"):
        with open(os.path.join(ROOT, "paper_2609_14144_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _rows(d, suffix):
    files = sorted(glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True))
    if not files:
        sys.exit(f"no *{suffix} under {d}")
    with open(files[0]) as f:
        return list(csv.DictReader(f))


def _bench_json(path):
    with open(path) as f:
        for line in f:
            line = line.strip()
            if line.startswith("{"):
                return json.loads(line)
    sys.exit(f"no JSON line in {path}")


def _timed(dispatches, bench):
    """The decode dispatches of the timed launches: every condition of the
    sweep is timed `len(kernel_ms_reps)` times, in order, and each timed
    launch is the first decode dispatch after bench.py's marker kernel.
    Returns [((name, condition, rep), dispatch)]."""
    conds = [(k, c, i) for k, c in bench["sweep"].items() if "realised_exit_rate" in c
             for i in range(len(c.get("kernel_ms_reps", [c["kernel_ms"]])))]
    rows = sorted(dispatches, key=lambda d: int(d["Dispatch_Id"]))
    out = []
    marks = [i for i, d in enumerate(rows) if MARKER_KERNEL in d["Kernel_Name"]]
    for m in marks:
        nxt = next((d for d in rows[m + 1:] if KERNEL in d["Kernel_Name"]), None)
        if nxt is not None:
            out.append(nxt)
    if len(out) != len(conds):
        sys.exit(f"found {len(out)} marked decode launches for {len(conds)} timed launches")
    return list(zip(conds, out))


def _rep_ms(c, rep):
    return c.get("kernel_ms_reps", [c["kernel_ms"]])[rep]


def trace(args):
    bench = _bench_json(args.bench)
    stats = _rows(args.dir, "kernel_stats.csv")
    disp = _rows(args.dir, "kernel_trace.csv")
    out = [f"# rocprofv3 kernel trace: {KERNEL}, {bench['config']['workload']}", "",
           "Command (run from the repository root on one MI355X):", "",
           f"    {args.command}", "",
           f"Kernel source hash: {kernel_source_hash()}", "",
           "## Per-kernel statistics (all dispatches of the run)", "",
           f"The {KERNEL} average mixes every launch of the run (calibration, prefill, "
           "warm-up and timed launches); the timed launches are matched one by one below.", "",
           "| kernel | calls | total ms | average us | min us | max us |",
           "|---|---|---|---|---|---|"]
    for r in sorted(stats, key=lambda r: -float(r["TotalDurationNs"]))[:12]:
        out.append(f"| {r['Name'][:70]} | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.3f} | "
                   f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
                   f"{float(r['MaxNs']) / 1e3:.2f} |")
    out += ["", "## Timed decode launches (one persistent launch of `steps` decode steps each)", "",
            "| condition | repetition | exit rate | steps | rocprof duration ms | bench HIP-event ms | difference |",
            "|---|---|---|---|---|---|---|"]
    for (name, c, rep), d in _timed(disp, bench):
        dur = (int(d["End_Timestamp"]) - int(d["Start_Timestamp"])) / 1e6
        ms = _rep_ms(c, rep)
        med = " (median)" if rep == c.get("median_rep", 0) else ""
        out.append(f"| {name} | {rep}{med} | {c['realised_exit_rate']:.3f} | {bench['steps']} | {dur:.3f} | "
                   f"{ms:.3f} | {100 * (dur / ms - 1):+.2f}% |")
    rf = bench["roofline"]
    out += ["", f"Headline (bench JSON): {bench['value']:.1f} {bench['unit']}; roofline achieved "
            f"{rf['achieved']:.1f} GB/s of {rf['peak']:.0f} GB/s (frac {rf['frac']:.4f}) from "
            f"{rf['algorithmic_bytes_per_launch'] / 1e9:.3f} GB of algorithmic bytes per launch "
            f"over {rf['launch_ms']:.3f} ms."]
    ceil = rf.get("ceiling")
    if ceil:
        probe = [r for r in stats if "k_stream_read" in r["Name"]]
        line = (f"Streaming-read ceiling (bench JSON, {ceil['probe']}): {ceil['GBs']:.0f} GB/s; "
                f"achieved / ceiling = {rf['frac_of_ceiling']:.3f}.")
        if probe:
            avg_us = float(probe[0]["AverageNs"]) / 1e3
            line += (f" The profiler's average for k_stream_read ({probe[0]['Calls']} calls) is "
                     f"{avg_us:.1f} us per {ceil['bytes'] / 2 ** 30:.0f} GiB = {ceil['bytes'] / avg_us / 1e3:.0f} GB/s.")
        out += ["", line]
    print("\n".join(out))


def _counter(d, name):
    rows = _rows(d, "counter_collection.csv")
    return [r for r in rows if r["Counter_Name"] == name]


def traffic(args):
    bench = _bench_json(args.bench)
    rec = {"kernel": KERNEL, "kernel_source_hash": kernel_source_hash(),
           "workload": bench["config"]["workload"], "steps": bench["steps"], "warmup": bench["warmup"],
           "prompt": bench["config"].get("prompt_tokens"),
           "command_fetch": args.command_fetch, "command_write": args.command_write,
           "copy_probe_mib": args.copy_mib}
    total = 0.0
    for key, d in (("FETCH_SIZE", args.fetch_dir), ("WRITE_SIZE", args.write_dir)):
        rows = _counter(d, key)
        copy = [r for r in rows if COPY_KERNEL in r["Kernel_Name"]]
        if not copy:
            sys.exit(f"{key}: no copy-probe dispatch")
        expect_kib = args.copy_mib * 1024.0
        scale = float(copy[0]["Counter_Value"]) / expect_kib  # counter units per KiB moved
        timed = _timed(rows, bench)
        (name, c, _), headline = next(((k, d) for k, d in timed if k[0] == "r0.5" and
                                       k[2] == bench["sweep"]["r0.5"].get("median_rep", 0)))
        b = float(headline["Counter_Value"]) / scale * 1024.0
        rec[key.lower()] = {"copy_counter_kib": float(copy[0]["Counter_Value"]), "copy_expected_kib": expect_kib,
                            "scale": scale, "raw_kib": float(headline["Counter_Value"]), "bytes": b,
                            "condition": name, "dispatch_id": int(headline["Dispatch_Id"])}
        total += b
    rec["hbm_bytes_per_launch"] = total
    rec["algorithmic_bytes_per_launch"] = bench["roofline"]["algorithmic_bytes_per_launch"]
    rec["ratio_to_algorithmic"] = total / bench["roofline"]["algorithmic_bytes_per_launch"]
    print(json.dumps(rec, indent=1))


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    sub = ap.add_subparsers(dest="mode", required=True)
    t = sub.add_parser("trace")
    t.add_argument("--dir", required=True)
    t.add_argument("--bench", required=True, help="file holding bench.py's JSON line")
    t.add_argument("--command", required=True)
    w = sub.add_parser("traffic")
    w.add_argument("--fetch-dir", required=True)
    w.add_argument("--write-dir", required=True)
    w.add_argument("--bench", required=True)
    w.add_argument("--copy-mib", type=float, required=True)
    w.add_argument("--command-fetch", required=True)
    w.add_argument("--command-write", required=True)
    a = ap.parse_args()
    trace(a) if a.mode == "trace" else traffic(a)


if __name__ == "__main__":
    main()
