"""Summarise rocprofv3 output (kernel-trace database or CSV) as a short text
table: per kernel name, calls, total and mean duration.

    python -m paper_1302_1700_amd.profsum <results.db | kernel_trace.csv | dir> [--pmc]
    python -m paper_1302_1700_amd.profsum util <pmc dir>
    python -m paper_1302_1700_amd.profsum copy <MiB>
    python -m paper_1302_1700_amd.profsum traffic <fetch_dir> <write_dir> <copy_fetch_dir>
           <copy_write_dir> <copy_MiB> <workload> [--out profiles/traffic.json]

With --pmc, counter values per kernel dispatch are averaged per kernel name
(FETCH_SIZE / WRITE_SIZE and the like).  `copy` runs a plain device-to-device
copy of a tensor of the given size (read once, written once): the calibration
point for the FETCH_SIZE / WRITE_SIZE counters.  `traffic` turns a FETCH_SIZE
pass and a WRITE_SIZE pass of a workload, plus the same two passes of the copy
probe, into HBM bytes per launch: each counter is scaled by (bytes the copy
moved) / (what the counter read for it), and the entry records the digest of
the kernel sources it was taken on.
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


def source_digest():
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc")
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".hip", ".h")):
            with open(os.path.join(csrc, f), "rb") as fh:
                h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def traffic(fetch_dir, write_dir, cfetch_dir, cwrite_dir, copy_mib, workload, out):
    import json
    copy_bytes = copy_mib * (1 << 20)
    cf = pmc_stats(cfetch_dir)
    cw = pmc_stats(cwrite_dir)
    ck = [k for k in cf if "copyBuffer" in k or "copy" in k.lower()]
    fscale = copy_bytes / (cf[ck[0]]["FETCH_SIZE"] * 1024.0)
    wscale = copy_bytes / (cw[ck[0]]["WRITE_SIZE"] * 1024.0)
    fe = pmc_stats(fetch_dir)
    wr = pmc_stats(write_dir)
    entries = []
    if os.path.exists(out):
        with open(out) as f:
            entries = [e for e in json.load(f) if e.get("workload") != workload]
    dig = source_digest()
    for k in fe:
        if not k or not k.startswith("void fs::"):
            continue
        fb = fe[k]["FETCH_SIZE"] * 1024.0 * fscale
        wb = wr.get(k, {}).get("WRITE_SIZE", 0.0) * 1024.0 * wscale
        entries.append({"kernel": k, "workload": workload, "source_digest": dig,
                        "fetch_bytes_per_launch": fb, "write_bytes_per_launch": wb,
                        "bytes_per_launch": fb + wb, "fetch_scale": fscale, "write_scale": wscale})
        print("%-80s fetch %10.3f MB  write %10.3f MB" % (k[:80], fb / 1e6, wb / 1e6))
    with open(out, "w") as f:
        json.dump(entries, f, indent=1)
    print("scales: FETCH x%.4f  WRITE x%.4f  -> %s" % (fscale, wscale, out))


def utilisation(path, simds=1024, xcds=8):
    """Per kernel name, from one SQ counter pass (SQ_WAVES, SQ_INSTS_VALU,
    SQ_INSTS_MFMA, SQ_INSTS_SALU, SQ_INSTS_LDS, SQ_INSTS_VMEM_RD,
    SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE): the matrix cores' busy
    fraction over the dispatch (busy cycles summed over all SIMDs, against
    the GPU-active cycles of one XCD times the SIMD count) and the
    instructions each wave issued."""
    rows = []
    for k, cs in pmc_stats(path).items():
        if not k or not k.startswith("void fs::"):
            continue
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
        utilisation(args[1])
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
