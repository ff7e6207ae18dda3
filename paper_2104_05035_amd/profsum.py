"""Summaries of rocprofv3 output for the measurement record.

    python -m paper_2104_05035_amd.profsum stats KERNEL_STATS_CSV BENCH_LOG OUT_MD TITLE COMMAND
        kernel-time table (rocprofv3 --kernel-trace --stats) with the bench.py
        JSON line of the same build (any --workload).

    python -m paper_2104_05035_amd.profsum traffic FETCH_CSV WRITE_CSV TAG SUBSTRING SOURCE OUT_MD CMD_F CMD_W
        HBM traffic of the kernel whose name contains SUBSTRING, from two
        rocprofv3 --pmc passes (FETCH_SIZE, then WRITE_SIZE; KiB per
        dispatch).  Each counter is scaled by what it reads for the largest
        device copy in the same run (bench.py --calib-copy copies 256 MiB),
        so the figure is bytes moved per launch.  The row records the SHA-1 of
        SOURCE; bench.py reports the figure only while that file is unchanged.
"""
import csv
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
TRAFFIC_MD = os.path.join(ROOT, "profiles", "hbm_traffic.md")
CALIB_BYTES = 256 * 1024 * 1024


def source_sha(path):
    with open(os.path.join(ROOT, path), "rb") as f:
        return hashlib.sha1(f.read()).hexdigest()[:12]


def _short(name):
    name = name.replace("(anonymous namespace)::", "")
    return name.split("(")[0].replace("void ", "").replace("rat3d::", "")


def stats(csv_path, bench_log, out, title, cmd):
    rows = list(csv.DictReader(open(csv_path)))
    bench = [ln for ln in open(bench_log) if ln.startswith("{")][-1].strip()
    b = json.loads(bench)
    work = b["config"]["workload"] if "config" in b else b["workload"]
    lines = ["# " + title, "",
             "Workload: %s; bf16 storage, fp32 accumulation." % work, "",
             "Command (repository root, one MI355X):", "", "    " + cmd, ""]
    if "roofline" in b:
        wu, bk, ts = b.get("warmup", 1), b.get("breakdown_steps", 3), b.get("steps", 3)
        sched = ("all of them with micro-batches not overlapped, like the step whose launches "
                 "the live timing brackets" if ts == 1 else
                 "all timed steps but the last with micro-batches overlapped")
        lines += ["Calls cover %d warm-up, %d breakdown and %d timed steps, %s.  Dominant kernel "
                  "per bench.py's live hipEvents: `%s`, %.1f us/launch (rocprofv3 average in the "
                  "table)." % (wu, bk, ts, sched, b["roofline"]["kernel"],
                               b["roofline"]["avg_launch_us"]), ""]
    else:
        lines += ["Calls cover 1 warm-up, 1 profiled (tagged) and 3 timed steps.", ""]
    lines += ["| kernel | calls | total ms | avg us | % |", "|---|---|---|---|---|"]
    for r in rows[:24]:
        lines.append("| `%s` | %s | %.1f | %.1f | %.2f |" % (
            _short(r["Name"]), r["Calls"], float(r["TotalDurationNs"]) / 1e6,
            float(r["AverageNs"]) / 1e3, float(r["Percentage"])))
    lines += ["", "bench.py line of the same build:", "", "```", bench, "```", ""]
    with open(out, "w") as f:
        f.write("\n".join(lines))


def _counter(csv_path, counter, substring):
    """(mean KiB per dispatch of the matching kernel, its dispatch count,
    KiB of the largest copy dispatch)."""
    per = {}
    for r in csv.DictReader(open(csv_path)):
        if r["Counter_Name"] != counter:
            continue
        key = (r["Dispatch_Id"], r["Kernel_Name"])
        per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
    vals = [v for (d, k), v in per.items() if substring in k]
    # the runtime's device copy (bench.py --calib-copy: 256 MiB); the bench's
    # own 1 GiB copy probe is a different kernel and is not the reference
    copies = [v for (d, k), v in per.items() if "rocclr_copyBuffer" in k]
    if not vals or not copies:
        raise SystemExit("no dispatches of %r or of a copy kernel in %s" % (substring, csv_path))
    return sum(vals) / len(vals), len(vals), max(copies)


def traffic(fetch_csv, write_csv, tag, substring, source, out, cmd_f, cmd_w):
    f_kib, n, f_cal = _counter(fetch_csv, "FETCH_SIZE", substring)
    w_kib, _, w_cal = _counter(write_csv, "WRITE_SIZE", substring)
    f_scale = CALIB_BYTES / (f_cal * 1024.0)
    w_scale = CALIB_BYTES / (w_cal * 1024.0)
    fetch = f_kib * 1024.0 * f_scale
    write = w_kib * 1024.0 * w_scale
    row = "| %s | %s | %s | %d | %.0f | %.0f | %.3f | %.3f | %.0f |" % (
        tag, source, source_sha(source), n, f_kib, w_kib, f_scale, w_scale, fetch + write)
    head = ["# HBM traffic per launch (rocprofv3 PMC)", "",
            "FETCH_SIZE and WRITE_SIZE are read in separate passes (KiB per dispatch, averaged "
            "over the kernel's dispatches in the run) and scaled by the factor that maps the "
            "same counter of a 256 MiB device copy in the same process onto 256 MiB.  bench.py "
            "reports `traffic` from the row whose tag and source SHA-1 match the build it runs.",
            "", "Commands (repository root, one MI355X):", ""]
    rows = []
    if os.path.exists(out):
        for ln in open(out):
            if ln.startswith("| ") and not ln.startswith("| tag") and ("| %s |" % tag) not in ln:
                rows.append(ln.rstrip("\n"))
    cmds = ["    " + cmd_f, "    " + cmd_w, ""]
    table = ["| tag | source | sha1 | dispatches | FETCH KiB | WRITE KiB | fetch scale | "
             "write scale | HBM bytes/launch |", "|---|---|---|---|---|---|---|---|---|"]
    with open(out, "w") as f:
        f.write("\n".join(head + cmds + table + rows + [row, ""]))
    print(row)


def lookup(tag):
    """HBM bytes per launch recorded for TAG, or None when absent or stale."""
    if not os.path.exists(TRAFFIC_MD):
        return None
    for ln in open(TRAFFIC_MD):
        cells = [c.strip() for c in ln.strip().strip("|").split("|")]
        if len(cells) == 9 and cells[0] == tag:
            try:
                if source_sha(cells[1]) != cells[2]:
                    return None
                return float(cells[8])
            except (OSError, ValueError):
                return None
    return None


if __name__ == "__main__":
    if sys.argv[1] == "stats":
        stats(*sys.argv[2:7])
    elif sys.argv[1] == "traffic":
        traffic(*sys.argv[2:10])
    else:
        raise SystemExit(__doc__)
