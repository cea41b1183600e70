"""Summarise rocprofv3 output (kernel-trace database or CSV) as a short text
table: per kernel name, calls, total and mean duration.

    python -m paper_1302_1700_amd.profsum <results.db | kernel_trace.csv | dir> [--pmc]
    python -m paper_1302_1700_amd.profsum copy <MiB>

With --pmc, counter values per kernel dispatch are averaged per kernel name
(FETCH_SIZE / WRITE_SIZE and the like).  `copy` runs a plain device-to-device
copy of a tensor of the given size (read once, written once): the calibration
point for the FETCH_SIZE / WRITE_SIZE counters.
"""
import csv
import glob
import os
import sqlite3
import sys
from collections import defaultdict


def _find(path, pattern):
    if os.path.isdir(path):
        hits = sorted(glob.glob(os.path.join(path, "**", pattern), recursive=True))
        return hits[0] if hits else None
    return path


def kernel_stats(path):
    db = _find(path, "*_results.db")
    rows = defaultdict(list)
    if db and db.endswith(".db"):
        con = sqlite3.connect(db)
        for name, dur in con.execute("select name, duration from kernels"):
            rows[name].append(dur)
    else:
        trace = _find(path, "*kernel_trace.csv")
        with open(trace) as f:
            for r in csv.DictReader(f):
                rows[r["Kernel_Name"]].append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    out = []
    for name, d in rows.items():
        out.append((name, len(d), sum(d), sum(d) / len(d)))
    out.sort(key=lambda r: -r[2])
    return out


def pmc_stats(path):
    db = _find(path, "*_results.db")
    acc = defaultdict(lambda: defaultdict(list))
    if db and db.endswith(".db"):
        con = sqlite3.connect(db)
        q = ("select k.name, p.counter_name, p.value from pmc_events p join kernels k "
             "on p.event_id = k.id")
        try:
            for name, cname, v in con.execute(q):
                acc[name][cname].append(v)
        except sqlite3.Error:
            cols = [r[1] for r in con.execute("pragma table_info(counters_collection)")]
            for r in con.execute("select * from counters_collection"):
                d = dict(zip(cols, r))
                acc[d.get("kernel_name")][d.get("counter_name")].append(d.get("value"))
    else:
        f = _find(path, "*counter_collection.csv")
        with open(f) as fh:
            per = defaultdict(lambda: defaultdict(float))
            for r in csv.DictReader(fh):
                per[(r["Kernel_Name"], r["Dispatch_Id"])][r["Counter_Name"]] += float(r["Counter_Value"])
            for (name, _), cs in per.items():
                for c, v in cs.items():
                    acc[name][c].append(v)
    return {k: {c: sum(v) / len(v) for c, v in cs.items()} for k, cs in acc.items()}


def copy_probe(mib):
    import torch
    n = mib * (1 << 20) // 4
    src = torch.rand(n, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print("copied %d MiB x 3" % mib)


def main():
    args = [a for a in sys.argv[1:] if not a.startswith("--")]
    if args and args[0] == "copy":
        copy_probe(int(args[1]))
        return
    if "--pmc" in sys.argv:
        for k, cs in pmc_stats(args[0]).items():
            print(k)
            for c, v in sorted(cs.items()):
                print("    %-28s %.6g" % (c, v))
        return
    print("%-90s %7s %12s %10s" % ("kernel", "calls", "total_us", "mean_us"))
    for name, n, tot, mean in kernel_stats(args[0]):
        print("%-90s %7d %12.1f %10.2f" % (name[:90], n, tot / 1e3, mean / 1e3))


if __name__ == "__main__":
    main()
