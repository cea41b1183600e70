"""Summarise rocprofv3 output (kernel-trace database or CSV) as a short text
table: per kernel name, calls, total and mean duration.

    python -m paper_1302_1700_amd.profsum <results.db | kernel_trace.csv | dir> [--pmc]
    python -m paper_1302_1700_amd.profsum util <pmc dir>
    python -m paper_1302_1700_amd.profsum copy <MiB>
    python -m paper_1302_1700_amd.profsum traffic <fetch_dir> <write_dir> <copy_fetch_dir>
           <copy_write_dir> <copy_MiB> <bench_log> [--out profiles/traffic.json]

With --pmc, counter values per kernel dispatch are averaged per kernel name
(FETCH_SIZE / WRITE_SIZE and the like).  `copy` runs a plain device-to-device
copy of a tensor of the given size (read once, written once): the calibration
point for the FETCH_SIZE / WRITE_SIZE counters.  `traffic` turns a FETCH_SIZE
pass and a WRITE_SIZE pass of bench.py over a workload, plus the same two
passes of the copy probe, into HBM bytes per launch of the scan: each counter
is scaled by (bytes the copy moved) / (what the counter read for it).  The
dispatches of the library's kernels are matched to the scan's launches by
their order (bench.py's JSON line, in <bench_log>, lists the launches; its
warm-up and timed scans run them in that order), so a kernel instance used by
several layers gets one entry per layer; each entry records the digest of the
kernel sources it was taken on.
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


def pmc_dispatches(path):
    """[(dispatch id, kernel name, {counter: value})] in dispatch order, the
    counter values summed over the dispatch's records."""
    db = _find(path, "*_results.db")
    per = {}
    if db and db.endswith(".db"):
        con = sqlite3.connect(db)
        for did, name, cname, v in con.execute(
                "select dispatch_id, name, counter_name, counter_value from pmc_events"):
            e = per.setdefault(did, [name, defaultdict(float)])
            e[1][cname] += v
    else:
        f = _find(path, "*counter_collection.csv")
        with open(f) as fh:
            for r in csv.DictReader(fh):
                did = int(r["Dispatch_Id"])
                e = per.setdefault(did, [r["Kernel_Name"], defaultdict(float)])
                e[1][r["Counter_Name"]] += float(r["Counter_Value"])
    return [(d, per[d][0], dict(per[d][1])) for d in sorted(per)]


def bench_line(log):
    """The JSON line bench.py printed (the last line that parses)."""
    import json
    res = None
    with open(log) as f:
        for line in f:
            line = line.strip()
            if line.startswith("{"):
                try:
                    res = json.loads(line)
                except ValueError:
                    pass
    if res is None:
        raise ValueError("no bench.py JSON line in %s" % log)
    return res


def copy_probe(mib):
    """Calibration kernels of known traffic on a tensor of `mib` MiB: a
    device-to-device copy (reads and writes it once), a sum (reads it once,
    writes one value) and a fill (writes it once), three times each."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.rand(n, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    for _ in range(3):
        src.sum()
    for _ in range(3):
        dst.fill_(1.0)
    torch.cuda.synchronize()
    print("copied, summed and filled %d MiB x 3" % mib)


def source_digest():
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc")
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".hip", ".h")):
            with open(os.path.join(csrc, f), "rb") as fh:
                h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def per_launch(path, bench, counter):
    """Mean of one counter per launch of the scan, over the plain scans of a
    bench.py run (warm-up and timed steps: every launch once per scan, in
    order); [(kernel name, mean)] in launch order."""
    return [(k, cs[counter]) for k, cs in per_launch_counters(path, bench)]


def per_launch_counters(path, bench):
    """[(kernel name, {counter: mean over the plain scans})] in launch order."""
    launches = bench["launches"]
    n = len(launches)
    disp = [d for d in pmc_dispatches(path) if d[1].startswith("void fs::")]
    scans = (bench["warmup"] + bench["steps"]) * n
    if len(disp) < scans:
        raise ValueError("%s: %d dispatches of the library, %d scans of %d launches expected"
                         % (path, len(disp), bench["warmup"] + bench["steps"], n))
    vals = [defaultdict(list) for _ in range(n)]
    names = [None] * n
    for i, (_, name, cs) in enumerate(disp[:scans]):
        L = launches[i % n]
        if L["name"].split("<")[0] not in name:
            raise ValueError("dispatch %d is %s, launch %d of the scan is %s" % (i, name, i % n, L["name"]))
        for c, v in cs.items():
            vals[i % n][c].append(v)
        names[i % n] = name
    return [(names[i], {c: sum(v) / len(v) for c, v in vs.items()}) for i, vs in enumerate(vals)]


def traffic(fetch_dir, write_dir, cfetch_dir, cwrite_dir, copy_mib, bench_log, out):
    import json
    copy_bytes = copy_mib * (1 << 20)
    cf = pmc_stats(cfetch_dir)
    cw = pmc_stats(cwrite_dir)
    ck = [k for k in cf if "copyBuffer" in k or "copy" in k.lower()]
    fscale = copy_bytes / (cf[ck[0]]["FETCH_SIZE"] * 1024.0)
    wscale = copy_bytes / (cw[ck[0]]["WRITE_SIZE"] * 1024.0)
    # second calibration points: a read-only reduction and a write-only fill
    # of the same tensor (the copy's factors are the ones applied)
    # (the kernels of those names that moved the most: torch also launches
    # small fills and reductions of its own)
    rk = sorted((k for k in cf if "reduce" in k.lower()), key=lambda k: -cf[k]["FETCH_SIZE"])
    fk = sorted((k for k in cw if "fill" in k.lower()), key=lambda k: -cw[k]["WRITE_SIZE"])
    fscale2 = copy_bytes / (cf[rk[0]]["FETCH_SIZE"] * 1024.0) if rk else None
    wscale2 = copy_bytes / (cw[fk[0]]["WRITE_SIZE"] * 1024.0) if fk else None
    print("calibration: copy FETCH x%.4f WRITE x%.4f; read-only sum FETCH x%s; write-only fill WRITE x%s"
          % (fscale, wscale, "%.4f" % fscale2 if fscale2 else "-", "%.4f" % wscale2 if wscale2 else "-"))
    bench = bench_line(bench_log)
    workload = bench["config"]["workload"]
    fe = per_launch(fetch_dir, bench, "FETCH_SIZE")
    wr = per_launch(write_dir, bench, "WRITE_SIZE")
    entries = []
    if os.path.exists(out):
        with open(out) as f:
            entries = [e for e in json.load(f) if e.get("workload") != workload]
    dig = source_digest()
    for L, (k, f), (_, w) in zip(bench["launches"], fe, wr):
        fb = f * 1024.0 * fscale
        wb = w * 1024.0 * wscale
        entries.append({"workload": workload, "launch": L["name"], "layer": L["layer"], "kernel": k,
                        "source_digest": dig, "fetch_bytes_per_launch": fb, "write_bytes_per_launch": wb,
                        "bytes_per_launch": fb + wb, "algorithmic_bytes": L["bytes"],
                        "fetch_scale": fscale, "write_scale": wscale,
                        "fetch_scale_sum": fscale2, "write_scale_fill": wscale2})
        print("L%-2d %-58s fetch %10.3f MB  write %10.3f MB  (algorithmic %10.3f MB)"
              % (L["layer"], L["name"][:58], fb / 1e6, wb / 1e6, L["bytes"] / 1e6))
    with open(out, "w") as f:
        json.dump(entries, f, indent=1)
    print("scales: FETCH x%.4f  WRITE x%.4f  -> %s" % (fscale, wscale, out))


def utilisation(path, simds=1024, xcds=8, bench_log=None):
    """Per kernel name (or, given the bench.py log of the run, per launch of
    the scan: 'L<layer> <launch>'), from one SQ counter pass (SQ_WAVES,
    SQ_INSTS_VALU, SQ_INSTS_MFMA, SQ_INSTS_SALU, SQ_INSTS_LDS,
    SQ_INSTS_VMEM_RD, SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE): the matrix
    cores' busy fraction over the dispatch (busy cycles summed over all
    SIMDs, against the GPU-active cycles of one XCD times the SIMD count) and
    the instructions each wave issued."""
    rows = []
    if bench_log:
        bench = bench_line(bench_log)
        items = [("L%d %s" % (L["layer"], L["name"]), cs)
                 for L, (_, cs) in zip(bench["launches"], per_launch_counters(path, bench))]
    else:
        items = [(k, cs) for k, cs in pmc_stats(path).items() if k and k.startswith("void fs::")]
    for k, cs in items:
        waves = cs.get("SQ_WAVES", 0.0) or 1.0
        active = cs.get("GRBM_GUI_ACTIVE", 0.0) / xcds
        busy = cs.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
        mfma = cs.get("SQ_INSTS_MFMA", 0.0)
        rows.append((k, busy / (active * simds) if active else 0.0, mfma / waves,
                     (cs.get("SQ_INSTS_VALU", 0.0) - mfma) / waves, cs.get("SQ_INSTS_SALU", 0.0) / waves,
                     cs.get("SQ_INSTS_LDS", 0.0) / waves, cs.get("SQ_INSTS_VMEM_RD", 0.0) / waves,
                     busy / mfma if mfma else 0.0, waves))
    print("%-78s %6s %7s %7s %6s %5s %5s %6s %8s" % ("kernel", "mfma%", "mfma/w", "valu/w", "salu/w",
                                                      "lds/w", "vmr/w", "cyc/mf", "waves"))
    for r in sorted(rows, key=lambda r: -r[1]):
        print("%-78s %5.1f%% %7.1f %7.1f %6.1f %5.1f %5.1f %6.1f %8.0f" % ((r[0][:78], 100 * r[1]) + r[2:]))


def main():
    args = [a for a in sys.argv[1:] if not a.startswith("--")]
    if args and args[0] == "traffic":
        out = "profiles/traffic.json"
        if "--out" in sys.argv:
            out = sys.argv[sys.argv.index("--out") + 1]
            args = [a for a in args if a != out]
        traffic(args[1], args[2], args[3], args[4], int(args[5]), args[6], out)
        return
    if args and args[0] == "copy":
        copy_probe(int(args[1]))
        return
    if args and args[0] == "util":
        utilisation(args[1], bench_log=args[2] if len(args) > 2 else None)
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
