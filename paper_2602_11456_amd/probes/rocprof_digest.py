"""Digests of rocprofv3 output for the library's kernels (measurement
tooling, not part of the library).

    python3 -m paper_2602_11456_amd.probes.rocprof_digest stats KERNEL_STATS_CSV
        per-kernel calls and average duration (rocprofv3 --kernel-trace --stats)
    python3 -m paper_2602_11456_amd.probes.rocprof_digest pipeline KERNEL_TRACE_CSV [COPY_TRACE_CSV]
        per call of the chunked pipeline: span, busy time per kernel and per
        stream, and any device-to-host DMA copies inside it (rocprofv3
        --kernel-trace [--memory-copy-trace] of bench.py --only-pipeline)
    python3 -m paper_2602_11456_amd.probes.rocprof_digest traffic FETCH_CSV WRITE_CSV COPY_BYTES OUT_JSON
        HBM bytes per dispatch from two rocprofv3 --pmc runs (FETCH_SIZE,
        then WRITE_SIZE, in KiB), each scaled by what the same counter reads
        for the device-to-device copies of COPY_BYTES bytes that
        bench.py --copy-calibration adds at the end of the run
    python3 -m paper_2602_11456_amd.probes.rocprof_digest counters PMC_CSV
        per-kernel averages of every counter of a rocprofv3 --pmc run
"""
from __future__ import annotations

import collections
import csv
import hashlib
import json
import os
import re
import statistics
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "csrc")


def short(name: str) -> str:
    """Kernel name without namespace, return type and arguments."""
    n = name.replace("void ", "").replace("aurora::", "")
    return n.split("(")[0]


def stats(path):
    for r in csv.DictReader(open(path)):
        if "aurora" not in r["Name"]:
            continue
        print(f"{short(r['Name']):60s} calls {int(r['Calls']):6d}  "
              f"avg {float(r['AverageNs']) / 1e3:10.1f} us  "
              f"total {float(r['TotalDurationNs']) / 1e6:9.2f} ms")


def pipeline(trace_path, copy_path=None):
    """Per pipeline call (each starts with run_reset_kernel): its span from
    the first kernel's start to the last one's end, and per kernel and per
    stream the dispatches and busy time."""
    rows = list(csv.DictReader(open(trace_path)))
    ev = []
    for r in rows:
        m = re.findall(r"([A-Za-z_]\w*)(?:<[^()]*>)?\(", r["Kernel_Name"])
        name = m[0] if m else r["Kernel_Name"][:40]
        q = r.get("Stream_Id") or r.get("Queue_Id")
        ev.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), name, q))
    copies = []
    if copy_path:
        for r in csv.DictReader(open(copy_path)):
            if "DEVICE_TO_HOST" in r.get("Direction", "") or "D2H" in r.get("Direction", ""):
                copies.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]),
                               int(r.get("Size", 0) or 0)))
    ev.sort()
    calls, cur = [], None
    for e in ev:
        if e[2] == "run_reset_kernel":
            cur = []
            calls.append(cur)
        if cur is not None and e[2] != "__amd_rocclr_copyBuffer":
            cur.append(e)
    for ci, c in enumerate(calls):
        names = collections.defaultdict(list)
        streams = collections.defaultdict(list)
        for s, e, n, q in c:
            names[n].append(e - s)
            streams[q].append(e - s)
        kind = "coded" if "coded_group_kernel" in names else "plain"
        t0 = min(s for s, *_ in c)
        t1 = max(e for _, e, *_ in c)
        print(f"call {ci} ({kind}): {len(c)} kernels, first kernel start to last kernel end "
              f"{(t1 - t0) / 1e6:.2f} ms")
        for n, d in sorted(names.items(), key=lambda x: -sum(x[1])):
            print(f"   {n:28s} x{len(d):4d}  avg {statistics.mean(d) / 1e3:8.1f} us  "
                  f"med {statistics.median(d) / 1e3:8.1f}  busy {sum(d) / 1e6:6.2f} ms")
        for q, d in sorted(streams.items(), key=lambda x: -sum(x[1])):
            print(f"   stream {q}: {len(d)} kernels, busy {sum(d) / 1e6:6.2f} ms")
        cc = [x for x in copies if t0 <= x[0] <= t1]
        if cc:
            nbytes = sum(b for *_, b in cc)
            busy = sum(e - s for s, e, _ in cc)
            print(f"   D2H copies x{len(cc)}: {nbytes / 1e9:.3f} GB, busy {busy / 1e6:.2f} ms")


def traffic(fetch_csv, write_csv, copy_bytes, out_json):
    def load(path, counter):
        per = collections.defaultdict(list)
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] == counter:
                per[r["Kernel_Name"]].append(float(r["Counter_Value"]))
        return per
    F = load(fetch_csv, "FETCH_SIZE")
    W = load(write_csv, "WRITE_SIZE")
    cf = [v for k, vs in F.items() if "copyBuffer" in k for v in vs]
    cw = [v for k, vs in W.items() if "copyBuffer" in k for v in vs]
    # the calibration copies only: FETCH_SIZE reads about half the copied
    # bytes there, WRITE_SIZE about all of them
    big_f = [v for v in cf if 0.4 < v * 1024 / copy_bytes < 0.6]
    big_w = [v for v in cw if 0.8 < v * 1024 / copy_bytes < 1.2]
    fetch_factor = copy_bytes / (sum(big_f) / len(big_f) * 1024)
    write_factor = copy_bytes / (sum(big_w) / len(big_w) * 1024)
    kernels = {}
    for k in F:
        if "aurora" not in k:
            continue
        f = sum(F[k]) / len(F[k])
        w = sum(W.get(k, [0])) / max(len(W.get(k, [0])), 1)
        kernels[short(k)] = {"dispatches": len(F[k]), "fetch_kib": f, "write_kib": w,
                             "bytes_per_dispatch": f * 1024 * fetch_factor
                             + w * 1024 * write_factor}
    h = hashlib.sha256()
    for f in ("extract.hip", "delta_internal.h", "apply.hip"):
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    # one planned extract call: the tensor table and tile map are the plan's,
    # built once, so only the stage, scan and finalize kernels run per call
    per_call = sum(v["bytes_per_dispatch"] for k, v in kernels.items()
                   if any(s in k for s in ("stage_kernel<true, true, false>",
                                           "group_sum_kernel<unsigned int>",
                                           "group_scan_kernel",
                                           "finalize_kernel<long, true, true, false>")))
    out = {"bytes_per_call": per_call, "fetch_factor": fetch_factor,
           "write_factor": write_factor,
           "calibration": f"3 device-to-device copies of {copy_bytes} bytes",
           "kernels": kernels, "kernel_source_sha256": h.hexdigest()}
    with open(out_json, "w") as f:
        json.dump(out, f, indent=1)
    print(f"fetch factor {fetch_factor:.4f}, write factor {write_factor:.4f}")
    for k, v in kernels.items():
        print(f"{k:60s} n={v['dispatches']:3d} read "
              f"{v['fetch_kib'] * 1024 * fetch_factor / 1e9:8.4f} GB write "
              f"{v['write_kib'] * 1024 * write_factor / 1e9:8.4f} GB")
    print(f"extract call (stage, scans, finalize): {per_call / 1e9:.3f} GB")


def counters(path):
    per = collections.defaultdict(lambda: collections.defaultdict(list))
    for r in csv.DictReader(open(path)):
        per[short(r["Kernel_Name"])][r["Counter_Name"]].append(float(r["Counter_Value"]))
    for k, cs in per.items():
        if "aurora" not in k and "::" in k:
            continue
        vals = "  ".join(f"{c}={statistics.mean(v):.4g}" for c, v in sorted(cs.items()))
        n = max(len(v) for v in cs.values())
        print(f"{k:60s} x{n:3d}  {vals}")


def main(argv):
    if len(argv) < 2:
        print(__doc__)
        return 2
    cmd, args = argv[1], argv[2:]
    if cmd == "stats":
        stats(*args)
    elif cmd == "pipeline":
        pipeline(*args)
    elif cmd == "traffic":
        traffic(args[0], args[1], int(args[2]), args[3])
    elif cmd == "counters":
        counters(*args)
    else:
        print(__doc__)
        return 2
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv))
