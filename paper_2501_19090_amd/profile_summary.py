"""Summarise rocprofv3 output for the committed profiles.

    python -m paper_2501_19090_amd.profile_summary stats  <kernel_stats.csv> <out.md> <command...>
    python -m paper_2501_19090_amd.profile_summary traffic <fetch_dir> <write_dir> <kernel-substring>
           <launch-name> <out.txt> <command...>
    python -m paper_2501_19090_amd.profile_summary steady <kernel_trace.csv> <N> <out.md> <kernel-substring>...
    python -m paper_2501_19090_amd.profile_summary counters <out.md> <title> <command> <dir> <kernel-substring>...
    python -m paper_2501_19090_amd.profile_summary fullbench <bench_full.json> <out.md> <command...>

`stats` turns a --kernel-trace --stats CSV into a short markdown table.
`counters` appends to <out.md> a table of every counter a --pmc pass in <dir>
collected, averaged over the dispatches of each kernel whose name contains a
given substring.
`steady` appends to <out.md> the average duration of the last N dispatches
of each kernel whose name contains a given substring (the timed steps that
follow the warm-up, as bench.py times them).
`fullbench` turns the JSON report of `bench.py --full` into a markdown table
(every configuration and batch size: PIFA, low-rank U V and dense times,
speedups, TFLOP/s, GB/s and fractions of peak) with the source digest of the
kernels it was measured on.
`traffic` reads two --pmc passes (FETCH_SIZE, then WRITE_SIZE; KiB per
dispatch), takes the average for the kernel whose name contains
<kernel-substring>, and scales it by what the same counters read for the
calibration copy (a device-to-device copy of a known byte count, recorded by
bench.py --profile-run); the result is written as JSON text together with
the source digest of the kernels it was measured on.
"""
from __future__ import annotations

import csv
import glob
import json
import os
import sys

from paper_2501_19090_amd import build

COPY_BYTES = 512 << 20  # bench.py --profile-run copies this many bytes once


def _short(name: str) -> str:
    for a, b in [("_ZN4pifa", ""), ("ENS_10ScatterEpi", "|Epi"), ("IDF16bLi", "<bf16,"), ("IDF16_Li", "<f16,")]:
        name = name.replace(a, b)
    return name[:110]


def stats(csv_path: str, out_md: str, command: str) -> None:
    rows = list(csv.DictReader(open(csv_path)))
    lines = ["# rocprofv3 kernel statistics", "", "Command (run from the repository root on the GPU host):", "",
             "```", command, "```", "",
             "| kernel | calls | avg us | min us | max us | share % |", "|---|---:|---:|---:|---:|---:|"]
    for r in rows[:16]:
        lines.append("| `%s` | %s | %.2f | %.2f | %.2f | %.1f |" % (
            _short(r["Name"]), r["Calls"], float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
            float(r["MaxNs"]) / 1e3, float(r["Percentage"])))
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")


def steady(trace_csv: str, n: int, out_md: str, subs) -> None:
    rows = list(csv.DictReader(open(trace_csv)))
    lines = ["", "Steady state: average of the last %d dispatches of each kernel (after the warm-up); forward "
             "kernel digest `%s`:" % (n, build.forward_kernel_digest()), "",
             "| kernel | dispatches averaged | avg us |", "|---|---:|---:|"]
    for sub in subs:
        d = [(int(r["Start_Timestamp"]), int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
             for r in rows if sub in r["Kernel_Name"]]
        d.sort()
        last = [x for _, x in d[-n:]]
        if not last:
            raise SystemExit("steady: no dispatch of a kernel matching %r" % sub)
        lines.append("| `%s` | %d | %.2f |" % (_short(sub), len(last), sum(last) / len(last) / 1e3))
    with open(out_md, "a") as f:
        f.write("\n".join(lines) + "\n")


def counters(out_md: str, title: str, command: str, dirname: str, subs) -> None:
    files = glob.glob(os.path.join(dirname, "**", "*counter_collection.csv"), recursive=True)
    rows = [r for fn in files for r in csv.DictReader(open(fn))]
    names = sorted({r["Counter_Name"] for r in rows})
    # FETCH_SIZE / WRITE_SIZE (KiB) also as MB scaled by the calibration copy
    scale = {}
    for n in ("FETCH_SIZE", "WRITE_SIZE"):
        cv = [float(r["Counter_Value"]) for r in rows if r["Counter_Name"] == n and _is_copy(r["Kernel_Name"])]
        if n in names and cv:
            scale[n] = COPY_BYTES / (max(cv) * 1024.0)
    cols = names + ["%s MB" % n for n in names if n in scale] + ["avg us"]
    lines = ["", "## " + title, "", "Command (run from the repository root on the GPU host):", "", "```", command,
             "```", "", "| kernel | dispatches | " + " | ".join(cols) + " |",
             "|---|---:|" + "---:|" * len(cols)]
    for sub in subs:
        sel = [r for r in rows if sub in r["Kernel_Name"]]
        if not sel:
            continue
        disp = len({r.get("Dispatch_Id", r.get("Correlation_Id", i)) for i, r in enumerate(sel)})
        avg = {}
        for n in names:
            v = [float(r["Counter_Value"]) for r in sel if r["Counter_Name"] == n]
            avg[n] = sum(v) / len(v) if v else None
        vals = ["%.4g" % avg[n] if avg[n] is not None else "" for n in names]
        vals += ["%.2f" % (avg[n] * 1024.0 * scale[n] / 1e6) for n in names if n in scale]
        dur = {r.get("Dispatch_Id", i): int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for i, r in enumerate(sel)}
        vals.append("%.2f" % (sum(dur.values()) / len(dur) / 1e3))
        lines.append("| `%s` | %d | %s |" % (_short(sub), disp, " | ".join(vals)))
    if scale:
        lines.append("")
        lines.append("MB columns: the KiB counts times %s, the factors that map the counters of the run's "
                     "%d MiB device copy to its true bytes." % (
                         ", ".join("%s %.4f" % (n, f) for n, f in scale.items()), COPY_BYTES >> 20))
    lines.append("avg us: dispatch durations under counter collection (slower than unprofiled runs).")
    with open(out_md, "a") as f:
        f.write("\n".join(lines) + "\n")


def _is_copy(name: str) -> bool:
    # the calibration copy is a device-to-device memcpy (the runtime's copy
    # kernel); torch's elementwise dtype conversions are not, and in runs that
    # build a large layer they move more bytes than the calibration copy
    return "copyBuffer" in name


def _counter(dirname: str, counter: str):
    files = glob.glob(os.path.join(dirname, "**", "*counter_collection.csv"), recursive=True)
    out = []
    for fn in files:
        for r in csv.DictReader(open(fn)):
            if r["Counter_Name"] == counter:
                out.append((r["Kernel_Name"], float(r["Counter_Value"])))
    return out


def _avg(vals, pred):
    v = [x for n, x in vals if pred(n)]
    return (sum(v) / len(v), len(v)) if v else (None, 0)


def traffic(fetch_dir, write_dir, kernel_sub, launch_name, out_txt, command):
    fetch = _counter(fetch_dir, "FETCH_SIZE")
    write = _counter(write_dir, "WRITE_SIZE")
    k_fetch, nf = _avg(fetch, lambda n: kernel_sub in n)
    k_write, nw = _avg(write, lambda n: kernel_sub in n)
    if not nf or not nw:
        raise SystemExit("traffic: no dispatch of a kernel matching %r (FETCH %d, WRITE %d)" % (kernel_sub, nf, nw))
    is_copy = _is_copy
    # the calibration copy is the largest copy dispatch in the run
    c_fetch = max((x for n, x in fetch if is_copy(n)), default=None)
    c_write = max((x for n, x in write if is_copy(n)), default=None)
    rec = {
        "kernel": launch_name, "kernel_name_match": kernel_sub,
        "dispatches": {"fetch": nf, "write": nw},
        "fetch_kib_raw": k_fetch, "write_kib_raw": k_write,
        "copy_bytes": COPY_BYTES, "copy_fetch_kib_raw": c_fetch, "copy_write_kib_raw": c_write,
        "source_digest": build.source_digest(), "forward_kernel_digest": build.forward_kernel_digest(),
        "command": command,
    }
    if None not in (k_fetch, k_write, c_fetch, c_write):
        f_scale = COPY_BYTES / (c_fetch * 1024.0)
        w_scale = COPY_BYTES / (c_write * 1024.0)
        rec.update({"fetch_scale": f_scale, "write_scale": w_scale,
                    "hbm_read_bytes_per_launch": k_fetch * 1024.0 * f_scale,
                    "hbm_write_bytes_per_launch": k_write * 1024.0 * w_scale})
        rec["hbm_bytes_per_launch"] = rec["hbm_read_bytes_per_launch"] + rec["hbm_write_bytes_per_launch"]
    with open(out_txt, "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    print(json.dumps(rec, indent=1))


def fullbench(json_path: str, out_md: str, command: str) -> None:
    rows = json.load(open(json_path))
    lines = ["# Every configuration: PIFA against the same-engine low-rank and dense layers", "",
             "Command (run from the repository root on the GPU host):", "", "```", command, "```", "",
             "Kernel source digest: `%s`.  Times are microseconds per forward: M <= 128 rows replay "
             "HIP graphs over weight copies rotated past the 256 MB Infinity Cache; larger M are eager "
             "launches after warm-up on the same copy.  x U V and x dense are the time ratios "
             "(above 1: PIFA faster).  TFLOP/s uses PIFA's 2 M r (d_in + d_out - r) FLOPs, GB/s its "
             "weights, indices, X and Y; fractions are of 2516.6 TFLOP/s and 8000 GB/s."
             % rows[0].get("source_digest", build.source_digest()), "",
             "| config | d_in -> d_out, r | M | PIFA us | U V us | dense us | x U V | x dense | TFLOP/s | "
             "frac MFMA | GB/s | frac HBM |",
             "|---|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    for r in rows:
        lines.append("| %s | %d -> %d, %d | %d | %.1f | %.1f | %.1f | %.2f | %.2f | %.0f | %.3f | %.0f | %.3f |" % (
            r["config"], r["d_in"], r["d_out"], r["r"], r["M"], r["pifa_us"], r["uv_us"], r["dense_us"],
            r["speedup_vs_uv"], r["speedup_vs_dense"], r["pifa_tflops"], r["pifa_tflops"] / 2516.5824,
            r["pifa_gbps"], r["pifa_gbps"] / 8000.0))
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    mode = sys.argv[1]
    if mode == "stats":
        stats(sys.argv[2], sys.argv[3], " ".join(sys.argv[4:]))
    elif mode == "counters":
        counters(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5], sys.argv[6:])
    elif mode == "steady":
        steady(sys.argv[2], int(sys.argv[3]), sys.argv[4], sys.argv[5:])
    elif mode == "fullbench":
        fullbench(sys.argv[2], sys.argv[3], " ".join(sys.argv[4:]))
    elif mode == "traffic":
        traffic(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5], sys.argv[6], " ".join(sys.argv[7:]))
    else:
        raise SystemExit(__doc__)
