"""Turn rocprofv3 CSV output into the short text summaries kept under profiles/.

    python -m paper_2606_12487_amd.rocprof_summary stats STATS_CSV [--top N] [--title T] [--command C]
    python -m paper_2606_12487_amd.rocprof_summary traffic FETCH_CSV WRITE_CSV \
        COPY_FETCH_CSV COPY_WRITE_CSV --kernel SUBSTR --source FILE \
        --algorithmic-bytes B [--reduce mean|median] [--title T] [--command C]
    python -m paper_2606_12487_amd.rocprof_summary trace TRACE_CSV --kernel SUBSTR \
        --first N [--labels a,b,c] [--bytes B1,B2,B3] [--title T] [--command C]
    python -m paper_2606_12487_amd.rocprof_summary counters CSV [CSV ...] --kernel SUBSTR \
        --labels a,b,c [--skip N] [--title T] [--command C]

`stats` reads rocprofv3's kernel statistics (--kernel-trace --stats
--output-format csv) and prints one row per kernel.  `traffic` reads two
counter runs of a kernel (FETCH_SIZE, WRITE_SIZE: KiB per dispatch) and the
same counters for a device copy of 256 MiB, scales the kernel's figures by
known-bytes / counted-bytes of the copy, and prints HBM bytes per launch
together with the kernel source digest they belong to.  `trace` reads the
per-dispatch kernel trace and prints the mean duration of one kernel over its
first N dispatches (a benchmark's headline launches, which come first) and
over all of them; with --labels, the dispatches of a kernel launched at
several shapes in a fixed cycle are also averaged per position of the cycle,
and with --bytes (one figure per label) each average is also given as GB/s.
`counters` reads counter passes of a run that launches a
kernel at several shapes in a fixed cycle (after N other dispatches of it)
and prints each counter's mean per dispatch for each shape of the cycle.
"""

import argparse
import csv
import hashlib
import statistics
import sys

COPY_BYTES = 256 << 20


def _rows(path):
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def stats(path, title, command, top=0):
    rows = _rows(path)
    if top:
        rows = sorted(rows, key=lambda r: -float(r.get("TotalDurationNs", 0)))[:top]
    out = [f"# {title}" if title else "# rocprofv3 kernel statistics"]
    if command:
        out.append(f"# command: {command}")
    out.append(f"# source: {path.split('/')[-1]}")
    out.append("kernel | calls | total_us | average_us | min_us | max_us | percent")
    for r in rows:
        name = r.get("Name", "?")
        calls = int(float(r.get("Calls", 0)))
        tot = float(r.get("TotalDurationNs", 0)) / 1e3
        avg = float(r.get("AverageNs", 0)) / 1e3
        mn = float(r.get("MinNs", 0)) / 1e3
        mx = float(r.get("MaxNs", 0)) / 1e3
        pct = float(r.get("Percentage", 0))
        out.append(f"{name} | {calls} | {tot:.1f} | {avg:.2f} | {mn:.2f} | {mx:.2f} | {pct:.1f}")
    return "\n".join(out)


def _counter(path, counter, kernel, reduce="median"):
    vals = [float(r["Counter_Value"]) for r in _rows(path)
            if r["Counter_Name"] == counter and kernel in r["Kernel_Name"]]
    if not vals:
        raise SystemExit(f"no {counter} rows for kernels matching {kernel!r} in {path}")
    f = statistics.mean if reduce == "mean" else statistics.median
    return f(vals), len(vals)


def trace(path, kernel, first, title, command, labels=None, nbytes=None):
    rows = [r for r in _rows(path) if kernel in r["Kernel_Name"]]
    if not rows:
        raise SystemExit(f"no dispatches of kernels matching {kernel!r} in {path}")
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    dur = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in rows]
    head = dur[:first]
    out = [f"# {title}" if title else "# rocprofv3 kernel trace"]
    if command:
        out.append(f"# command: {command}")
    out += [f"kernel: {kernel}",
            f"dispatches_all: {len(dur)}",
            f"average_us_all: {statistics.mean(dur):.2f}",
            f"dispatches_first: {len(head)}",
            f"average_us_first: {statistics.mean(head):.2f}",
            f"min_us_first: {min(head):.2f}",
            f"max_us_first: {max(head):.2f}"]
    if labels:
        out.append("position | dispatches | average_us | min_us" + (" | GB/s" if nbytes else ""))
        for k, lab in enumerate(labels):
            d = dur[k::len(labels)]
            line = f"{lab} | {len(d)} | {statistics.mean(d):.2f} | {min(d):.2f}"
            if nbytes:
                line += f" | {nbytes[k] / (statistics.mean(d) * 1e-6) / 1e9:.1f}"
            out.append(line)
    return "\n".join(out)


def traffic(a, title, command):
    fetch, nf = _counter(a.fetch_csv, "FETCH_SIZE", a.kernel, a.reduce)
    write, nw = _counter(a.write_csv, "WRITE_SIZE", a.kernel, a.reduce)
    cfetch, _ = _counter(a.copy_fetch_csv, "FETCH_SIZE", a.copy_kernel)
    cwrite, _ = _counter(a.copy_write_csv, "WRITE_SIZE", a.copy_kernel)
    fscale = COPY_BYTES / (cfetch * 1024.0)
    wscale = COPY_BYTES / (cwrite * 1024.0)
    fb = fetch * 1024.0 * fscale
    wb = write * 1024.0 * wscale
    digest = hashlib.sha256(open(a.source, "rb").read()).hexdigest()[:16]
    out = [f"# {title}" if title else "# HBM traffic per launch"]
    if command:
        for c in command.split(" ;; "):
            out.append(f"# command: {c}")
    out += [
        f"kernel: {a.kernel}",
        f"source: {a.source.split('/')[-1]}",
        f"source_sha256_16: {digest}",
        f"dispatches_fetch: {nf}",
        f"dispatches_write: {nw}",
        f"fetch_kib_per_launch: {fetch:.1f}",
        f"write_kib_per_launch: {write:.1f}",
        f"copy_fetch_kib: {cfetch:.1f}",
        f"copy_write_kib: {cwrite:.1f}",
        f"fetch_scale: {fscale:.4f}",
        f"write_scale: {wscale:.4f}",
        f"hbm_read_bytes_per_launch: {fb:.0f}",
        f"hbm_write_bytes_per_launch: {wb:.0f}",
        f"hbm_bytes_per_launch: {fb + wb:.0f}",
        f"algorithmic_bytes_per_launch: {a.algorithmic_bytes}",
        f"traffic_over_algorithmic: {(fb + wb) / a.algorithmic_bytes:.3f}",
    ]
    return "\n".join(out)


def counters(paths, kernel, labels, skip, title, command):
    per = {}   # counter -> dispatch id -> summed value
    for path in paths:
        for r in _rows(path):
            if kernel in r["Kernel_Name"]:
                d = per.setdefault(r["Counter_Name"], {})
                i = int(r["Dispatch_Id"])
                d[i] = d.get(i, 0.0) + float(r["Counter_Value"])
    out = [f"# {title}" if title else "# rocprofv3 counters per dispatch"]
    if command:
        for c in command.split(" ;; "):
            out.append(f"# command: {c}")
    out.append("counter | " + " | ".join(labels))
    for name in sorted(per):
        ids = sorted(per[name])[skip:]
        cols = [[] for _ in labels]
        for k, i in enumerate(ids):
            cols[k % len(labels)].append(per[name][i])
        out.append(name + " | " + " | ".join(
            f"{statistics.mean(c):.0f}" if c else "-" for c in cols))
    return "\n".join(out)


def main(argv=None):
    p = argparse.ArgumentParser()
    sub = p.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("--top", type=int, default=0, help="only the N kernels with the most total time")
    s.add_argument("--title", default="")
    s.add_argument("--command", default="")
    t = sub.add_parser("traffic")
    t.add_argument("fetch_csv")
    t.add_argument("write_csv")
    t.add_argument("copy_fetch_csv")
    t.add_argument("copy_write_csv")
    t.add_argument("--kernel", required=True)
    t.add_argument("--copy-kernel", default="")
    t.add_argument("--source", required=True)
    t.add_argument("--algorithmic-bytes", type=int, required=True)
    t.add_argument("--reduce", choices=["median", "mean"], default="median")
    t.add_argument("--title", default="")
    t.add_argument("--command", default="")
    r = sub.add_parser("trace")
    r.add_argument("csv")
    r.add_argument("--kernel", required=True)
    r.add_argument("--first", type=int, required=True)
    r.add_argument("--labels", default="")
    r.add_argument("--bytes", default="")
    r.add_argument("--title", default="")
    r.add_argument("--command", default="")
    c = sub.add_parser("counters")
    c.add_argument("csv", nargs="+")
    c.add_argument("--kernel", required=True)
    c.add_argument("--labels", required=True)
    c.add_argument("--skip", type=int, default=0)
    c.add_argument("--title", default="")
    c.add_argument("--command", default="")
    a = p.parse_args(argv)
    if a.cmd == "counters":
        print(counters(a.csv, a.kernel, a.labels.split(","), a.skip, a.title, a.command))
        return
    if a.cmd == "stats":
        print(stats(a.csv, a.title, a.command, a.top))
    elif a.cmd == "trace":
        labels = a.labels.split(",") if a.labels else None
        nbytes = [float(b) for b in a.bytes.split(",")] if a.bytes else None
        print(trace(a.csv, a.kernel, a.first, a.title, a.command, labels, nbytes))
    else:
        print(traffic(a, a.title, a.command))


if __name__ == "__main__":
    sys.exit(main())
