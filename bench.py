#!/usr/bin/env python3
"""Benchmark of the sparse delta checkpoint hot path on one MI355X.

Workload: a Qwen3-8B-shaped bf16 weight set (399 tensors, 8,190,735,360
words, untied embedding and LM head) with 1% of the words of every tensor
changed, drawn on the GPU by ``paper_2602_11456_amd.synth``.  Inputs are
resident in HBM before timing starts.

One step = delta_extract_multi over the whole set (int64 global indices)
followed by delta_apply_multi of the result into a rollout copy.  Apply
assigns the new words, so re-applying the same delta every step is exact
and idempotent.

Timing: W untimed warm-up steps, then K timed steps between two
synchronisations; HIP events on the launch stream bracket every extract and
every apply.  Printed: one JSON line with GB/s scanned by extract (4 bytes
per word: both copies read once) as ``value``, the extract kernel's
roofline figures, apply throughput, and the CPU oracle timed on a bounded
sample of the same weight set.

    python bench.py [--steps K] [--warmup W] [--gpus 1]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

METRIC = "delta extract GB/s scanned (% of HBM peak) + apply GB/s, Qwen3-8B shape @1%"
HBM_PEAK_GBPS = 8000.0
ROOT = os.path.dirname(os.path.abspath(__file__))
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "extract_qwen3-8b_traffic.json")
CEILINGS_PROBE = os.path.join(ROOT, "paper_2602_11456_amd", "probes", "ceilings")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--density", type=float, default=0.01)
    ap.add_argument("--model", default="qwen3-8b")
    ap.add_argument("--clustered", action="store_true",
                    help="80%% of the changes in 5%% of the rows (the clustered Qwen3-8B set)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="oracle time budget for the CPU baseline sample")
    ap.add_argument("--traffic", default=TRAFFIC_FILE,
                    help="JSON file with measured HBM bytes per extract call")
    ap.add_argument("--no-pipeline", action="store_true",
                    help="skip the chunked extract -> pinned host pipeline measurement "
                         "(Qwen3-14B-shaped set)")
    ap.add_argument("--pipeline-reps", type=int, default=5)
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip the write-ceiling probe of apply")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the other weight sets (Qwen3-8B at 0.1%% and 10%%, clustered, "
                         "Qwen3-4B)")
    ap.add_argument("--only-pipeline", action="store_true",
                    help="measure only the pipelines on the Qwen3-14B-shaped set and print "
                         "their figures (for profiling; not the benchmark line)")
    ap.add_argument("--no-extras", action="store_true",
                    help="time only the headline step (extract + apply); skip the LEB128, "
                         "hash, fused-layout and delta-chain measurements")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="after timing, copy BYTES device-to-device three times (a known "
                         "traffic reference for hardware counters)")
    return ap.parse_args()


def kernel_source_digest():
    """Digest of the extract and apply kernels' sources: stored traffic
    figures are only used while the kernels they were measured on are
    unchanged."""
    import hashlib
    h = hashlib.sha256()
    for f in ("extract.hip", "delta_internal.h", "apply.hip"):
        with open(os.path.join(ROOT, "paper_2602_11456_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measure_ceilings():
    """The scatter's write ceilings on this device, from the measurement
    probe (paper_2602_11456_amd/probes/ceilings.hip, built with the
    library): partial and full 64-byte line writes per second at the
    spacing of a 1% delta over the Qwen3-8B set's size, with no loads.  Run
    as a child process before this process touches the GPU."""
    import subprocess
    if not os.path.exists(CEILINGS_PROBE):
        return {"error": f"{CEILINGS_PROBE} is not built (run __graft_entry__.build())"}
    try:
        r = subprocess.run([CEILINGS_PROBE], capture_output=True, text=True, timeout=120)
    except subprocess.TimeoutExpired:
        return {"error": "the ceilings probe timed out"}
    if r.returncode != 0:
        return {"error": f"the ceilings probe failed ({r.returncode}): {r.stderr.strip()[-300:]}"}
    return json.loads(r.stdout.strip().splitlines()[-1])


def apply_path(words, count):
    """Which path delta_apply_multi_sorted takes for `count` entries over
    `words` words: the tile merge from one word in 32, the scatter below."""
    return "tile merge" if count > 0 and count >= words // 32 else "scatter"


def apply_roofline(N, K, app_s, apply_bytes, apply_achieved, apply_traffic, lines, ceiling,
                   ceilings):
    """The apply's roofline for the path it took: the scatter against the
    measured rate of partial-line writes, the tile merge against HBM peak
    for its bytes (every word read and written once, plus the delta)."""
    if apply_path(N, K) == "tile merge":
        moved = 4 * N + 10 * K
        return {
            "kernel": "apply_merge_kernel (16384-word tiles read, patched in LDS, written whole)",
            "bound": "hbm",
            "achieved": round(moved / app_s / 1e9, 2),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(moved / app_s / 1e9 / HBM_PEAK_GBPS, 4),
            "traffic": None,
            "algorithmic_bytes": moved,
            "note": "a delta of at least one word in 32 touches nearly every 64-byte line; "
                    "the merge reads and writes every word once instead of one partial-line "
                    "write per touched line",
        }
    return {
        "kernel": "apply_multi_kernel (scattered 2-byte stores)",
        "bound": "hbm",
        "achieved": round(apply_achieved, 2),
        "peak": HBM_PEAK_GBPS,
        "unit": "GB/s",
        "frac": round(apply_achieved / HBM_PEAK_GBPS, 4),
        "traffic": apply_traffic,
        "algorithmic_bytes": apply_bytes,
        "lines_touched": lines,
        "line_writes_per_s": round(lines / app_s, 1),
        "ceiling_line_writes_per_s": ceiling,
        "frac_of_ceiling": round(lines / app_s / ceiling, 4) if ceiling else None,
        "ceilings_probe": ceilings,
        "note": "each touched 64-byte line costs one partial-line write at the memory; "
                "the ceiling is the rate of such writes with no loads at all, measured "
                "in this run by paper_2602_11456_amd/probes/ceilings (full-line writes "
                "are faster, but making a line full needs its old words: a read)",
    }


def touched_lines(weights, idx, numels):
    """Distinct 64-byte lines of the weight tensors that a delta's entries
    fall in (counted with torch on the GPU, outside any timed region): the
    fewest write transactions a scatter of the delta can issue."""
    import itertools
    import torch
    if idx.numel() == 0:
        return 0
    dev = idx.device
    bases = torch.tensor([0] + list(itertools.accumulate(numels))[:-1], dtype=torch.int64,
                         device=dev)
    ptrs = torch.tensor([w.data_ptr() for w in weights], dtype=torch.int64, device=dev)
    t = torch.searchsorted(bases, idx, right=True) - 1
    line = (ptrs[t] + 2 * (idx - bases[t])) >> 6
    del t
    return int((line[1:] != line[:-1]).sum().item()) + 1


def cpu_info():
    """CPU model (from /proc/cpuinfo) and the cores this process may run on."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        nproc = len(os.sched_getaffinity(0))
    except AttributeError:
        nproc = os.cpu_count() or 1
    return model, nproc


def cpu_baseline(ws, budget_s, reps=4):
    """The CPU oracle on the same weight set, timed on the host's cores.

    Single thread: tensor by tensor, each scanned ``reps`` times back to
    back while its host copy is resident, for half the budget.  All cores:
    the threaded oracle (contiguous per-thread ranges, concatenated in
    order) over batches of whole tensors of about 2 G words, each batch
    scanned ``reps`` times, for the other half.  Host copies are not timed.
    GB/s scanned = 4 bytes per word over the oracle's own time."""
    import numpy as np
    import torch
    import oracle

    oracle.build(force=False)
    model, nproc = cpu_info()
    threads = int(os.environ.get("OMP_NUM_THREADS") or 0) or nproc
    threads = max(1, min(threads, nproc))

    def host(t):
        return t.view(torch.int16).reshape(-1).cpu().numpy().view(np.uint16)

    # single thread
    words1 = 0
    spent1 = 0.0
    tensors1 = 0
    for p, q, k in zip(ws.prev, ws.new, ws.planted):
        hp, hq = host(p), host(q)
        for _ in range(reps):
            t0 = time.perf_counter()
            _, _, cnt = oracle.extract(hp, hq, np.int64, capacity=k)
            spent1 += time.perf_counter() - t0
            words1 += hp.size
            if cnt != k:
                raise RuntimeError(f"oracle found {cnt} changed words, {k} planted")
        tensors1 += 1
        if spent1 >= budget_s / 2:
            break
    # all cores, batches of whole tensors
    wordsm = 0
    spentm = 0.0
    tensorsm = 0
    batch_words = 2 << 30
    i = 0
    T = len(ws.prev)
    while i < T and spentm < budget_s / 2:
        j, n = i, 0
        while j < T and (j == i or n + ws.prev[j].numel() <= batch_words):
            n += ws.prev[j].numel()
            j += 1
        hps = [host(p) for p in ws.prev[i:j]]
        hqs = [host(q) for q in ws.new[i:j]]
        k = sum(ws.planted[i:j])
        for _ in range(reps):
            t0 = time.perf_counter()
            _, _, _, cnt = oracle.extract_multi(hps, hqs, capacity=k, threads=threads)
            spentm += time.perf_counter() - t0
            wordsm += n
            if cnt != k:
                raise RuntimeError(f"threaded oracle found {cnt} changed words, {k} planted")
        del hps, hqs
        tensorsm += j - i
        i = j
    single = 4 * words1 / spent1 / 1e9
    multi = 4 * wordsm / spentm / 1e9
    return {
        "value": round(multi, 3),
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"threaded oracle on {threads} threads: the first {tensorsm} of {T} tensors "
                  f"of the same weight set in batches of up to {batch_words} words, each batch "
                  f"scanned {reps} times ({wordsm} words, {4 * wordsm / 1e9:.1f} GB) in "
                  f"{spentm:.1f} s; single-threaded C loop: the first {tensors1} tensors, each "
                  f"scanned {reps} times ({4 * words1 / 1e9:.1f} GB) in {spent1:.1f} s",
        "single_thread_GBps": round(single, 3),
        "all_cores_GBps": round(multi, 3),
        "nproc": nproc,
        "cpu_model": model,
    }


def pipeline_measurement(args, dev):
    """Chunked extract -> pinned host memory with 4 HIP streams passed (3
    of them busy: reading, finishing, delivering) on the Qwen3-14B-shaped
    set at 1% (2^27-word chunks), host-synchronous calls
    over a tensor plan built once (as a training loop keeps its weights)
    timed with the wall clock, next to a pinned device-to-host copy of the
    same number of bytes (the host-link ceiling)."""
    import torch
    import paper_2602_11456_amd as ad
    from paper_2602_11456_amd import synth

    ws = synth.make_weight_set("qwen3-14b", args.density, seed=synth.config_seed(5), device=dev)
    torch.cuda.synchronize()
    K = ws.total_planted
    chunk, nstreams = 1 << 27, 4
    plan = ad.MultiPlan(ws.prev, ws.new)
    staging = torch.empty(ad.delta_pipeline_staging_bytes(plan.numels, chunk, nstreams),
                          dtype=torch.uint8, device=dev)
    streams = [torch.cuda.Stream(device=dev) for _ in range(nstreams)]
    h_idx = torch.empty(K + 4096, dtype=torch.int64, pin_memory=True)
    h_val = torch.empty(K + 4096, dtype=torch.bfloat16, pin_memory=True)
    times = []
    for rep in range(args.pipeline_reps + 1):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        i, v = ad.delta_extract_pipelined_plan(plan, chunk, nstreams, h_idx, h_val,
                                               staging, streams)
        t = time.perf_counter() - t0
        if i.numel() != K:
            raise RuntimeError(f"pipeline found {i.numel()} changed words, {K} planted")
        if rep:
            times.append(t)
    out_bytes = K * 10
    # host-link ceiling: one pinned D2H copy of the same bytes
    src = torch.empty(out_bytes, dtype=torch.uint8, device=dev)
    dst = torch.empty(out_bytes, dtype=torch.uint8, pin_memory=True)
    ctimes = []
    for rep in range(3):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        dst.copy_(src, non_blocking=True)
        torch.cuda.synchronize()
        ctimes.append(time.perf_counter() - t0)
    t = sorted(times)[len(times) // 2]
    tc = min(ctimes)
    del src, dst, h_idx, i

    # the same pipeline with the indices gap + LEB128 coded before the copy
    staging = None
    torch.cuda.empty_cache()
    staging = torch.empty(ad.delta_pipeline_leb128_staging_bytes(plan.numels, chunk, nstreams),
                          dtype=torch.uint8, device=dev)
    h_bytes = torch.empty(3 * K + 4096, dtype=torch.uint8, pin_memory=True)
    ltimes = []
    for rep in range(args.pipeline_reps + 1):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        b, v2, counts, used = ad.delta_extract_pipelined_leb128_plan(
            plan, chunk, nstreams, h_bytes, h_val, staging, streams)
        tl = time.perf_counter() - t0
        if v2.numel() != K:
            raise RuntimeError(f"coded pipeline found {v2.numel()} changed words, {K} planted")
        if rep:
            ltimes.append(tl)
    tl = sorted(ltimes)[len(ltimes) // 2]
    coded_bytes = b.numel() + 2 * K
    return {
        "workload": f"qwen3-14b weight set, {len(ws.prev)} tensors, {ws.total} bf16 words, "
                    f"{args.density:.2%} changed, {chunk}-word chunks, {nstreams} streams passed "
                    "of which 3 carry work (one reads every chunk, one finishes each read "
                    "chunk, one delivers into pinned host memory; a process has 4 hardware "
                    "queues, and more busy streams would share them and serialise)",
        "streams_passed": nstreams,
        "streams_busy": min(nstreams, 3),
        "ms": round(t * 1e3, 3),
        "GBps_scanned": round(4 * ws.total / t / 1e9, 1),
        "d2h_GBps": round(out_bytes / t / 1e9, 2),
        "d2h_ceiling_GBps": round(out_bytes / tc / 1e9, 2),
        "d2h_bytes": out_bytes,
        "leb128": {
            "ms": round(tl * 1e3, 3),
            "GBps_scanned": round(4 * ws.total / tl / 1e9, 1),
            "d2h_bytes": coded_bytes,
            "index_bytes_per_entry": round(b.numel() / K, 4),
            "d2h_GBps": round(coded_bytes / tl / 1e9, 2),
        },
    }


def leb128_measurement(ad, plan, idx, val, d_offs, numels, rollout, stream, reps):
    """Gap + LEB128 encode of the extracted global indices with one segment
    per tensor (tensor-local first index), then decode, each timed with HIP
    events on the launch stream; the decode must return the indices.  Also
    the extract that writes the coded indices itself
    (delta_extract_multi_leb128), whose bytes must equal the encoder's."""
    import torch
    lib = ad.library()
    dev = idx.device
    K = idx.numel()
    T = len(numels)
    bases = torch.tensor([0] + list(_prefix(numels))[:-1], dtype=torch.int64, device=dev)
    h = stream.cuda_stream
    enc_ws = torch.empty(max(lib.delta_leb128_encode_workspace_bytes(K), 1), dtype=torch.uint8,
                         device=dev)
    cap = 10 * K
    buf = torch.empty(max(cap, 1), dtype=torch.uint8, device=dev)
    nbytes = torch.zeros(1, dtype=torch.int64, device=dev)
    seg_bytes = torch.zeros(T + 1, dtype=torch.int64, device=dev)

    def encode():
        st = lib.delta_leb128_encode(idx.data_ptr(), K, d_offs.data_ptr(), bases.data_ptr(), T,
                                     buf.data_ptr(), cap, nbytes.data_ptr(), seg_bytes.data_ptr(),
                                     None, enc_ws.data_ptr(), enc_ws.numel(), h)
        if st:
            raise RuntimeError(lib.delta_last_error().decode())

    encode()
    stream.synchronize()
    nb = int(nbytes.item())
    dec_ws = torch.empty(lib.delta_leb128_decode_workspace_bytes(nb, K, T), dtype=torch.uint8,
                         device=dev)
    out = torch.empty(max(K, 1), dtype=torch.int64, device=dev)
    cnt = torch.zeros(1, dtype=torch.int64, device=dev)
    flag = torch.zeros(1, dtype=torch.int32, device=dev)

    def decode():
        st = lib.delta_leb128_decode(buf.data_ptr(), nb, d_offs.data_ptr(), bases.data_ptr(), T,
                                     out.data_ptr(), K, cnt.data_ptr(), flag.data_ptr(),
                                     dec_ws.data_ptr(), dec_ws.numel(), h)
        if st:
            raise RuntimeError(lib.delta_last_error().decode())

    decode()
    stream.synchronize()
    if int(cnt.item()) != K or int(flag.item()) or not torch.equal(out[:K], idx):
        raise RuntimeError("LEB128 decode does not return the extracted indices")
    # decode-in-apply onto the rollout copy (idempotent), against decode +
    # apply of the decoded indices
    apply_ws = torch.empty(ad.delta_apply_leb128_multi_workspace_bytes(nb, T), dtype=torch.uint8,
                           device=dev)
    multi_ws = torch.empty(max(ad.delta_apply_multi_workspace_bytes(T), 1), dtype=torch.uint8,
                           device=dev)
    flag2 = torch.zeros(1, dtype=torch.int32, device=dev)
    code = buf[:nb]

    def apply_coded():
        ad.delta_apply_leb128_multi(rollout, code, d_offs, bases, val, error_flag=flag2,
                                    workspace=apply_ws, stream=stream)

    apply_coded()
    stream.synchronize()
    if int(flag2.item()):
        raise RuntimeError("decode-in-apply flagged an error")
    # the sender's side in one call: extract straight to the coded stream
    cws = torch.empty(ad.delta_extract_multi_leb128_workspace_bytes(numels), dtype=torch.uint8,
                      device=dev)
    ccode = torch.empty(nb + 64, dtype=torch.uint8, device=dev)
    cval = torch.empty(K + 64, dtype=val.dtype, device=dev)
    ccnt = torch.zeros(1, dtype=torch.int64, device=dev)
    cnb = torch.zeros(1, dtype=torch.int64, device=dev)
    coffs = torch.zeros(T + 1, dtype=torch.int64, device=dev)
    cboffs = torch.zeros(T + 1, dtype=torch.int64, device=dev)

    def extract_coded():
        ad.delta_extract_multi_leb128_into(plan, ccode, cval, ccnt, cnb, cws, coffs, cboffs,
                                           stream)

    extract_coded()
    stream.synchronize()
    if (int(ccnt.item()) != K or int(cnb.item()) != nb or not torch.equal(ccode[:nb], code)
            or not torch.equal(cboffs, seg_bytes) or not torch.equal(coffs, d_offs)
            or not torch.equal(cval[:K].view(torch.int16), val.view(torch.int16))):
        raise RuntimeError("the coded extract differs from extract + encode")
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(reps)]
    for e0, e1, e2, e3, e4, e5 in ev:
        e0.record(stream)
        encode()
        e1.record(stream)
        decode()
        e2.record(stream)
        apply_coded()
        e3.record(stream)
        ad.delta_apply_multi(rollout, out[:K], val, workspace=multi_ws, stream=stream)
        e4.record(stream)
        extract_coded()
        e5.record(stream)
    stream.synchronize()
    med = lambda xs: sorted(xs)[len(xs) // 2]
    enc = med([e[0].elapsed_time(e[1]) for e in ev])
    dec = med([e[1].elapsed_time(e[2]) for e in ev])
    app_coded = med([e[2].elapsed_time(e[3]) for e in ev])
    app_plain = med([e[3].elapsed_time(e[4]) for e in ev])
    ext_coded = med([e[4].elapsed_time(e[5]) for e in ev])
    N = sum(numels)
    return {
        "workload": f"the {K} extracted int64 global indices, one segment per tensor",
        "bytes": nb,
        "bytes_per_entry": round(nb / K, 4),
        "encode_ms": round(enc, 4),
        "decode_ms": round(dec, 4),
        # encode reads the indices (twice: sizes, then bytes) and writes the bytes
        "encode_GBps_algorithmic": round((8 * K + nb) / (enc / 1e3) / 1e9, 1),
        "decode_GBps_algorithmic": round((nb + 8 * K) / (dec / 1e3) / 1e9, 1),
        "apply_from_code_ms": round(app_coded, 4),
        "decode_then_apply_ms": round(dec + app_plain, 4),
        # delta_extract_multi_leb128: both copies read once, the words and the
        # code written (no index stream)
        "extract_coded_ms": round(ext_coded, 4),
        "extract_coded_GBps_scanned": round(4 * N / (ext_coded / 1e3) / 1e9, 1),
        "extract_coded_GBps_algorithmic": round((4 * N + 2 * K + nb) / (ext_coded / 1e3) / 1e9,
                                                1),
    }


def compose_measurement(ad, rollout, N, K_entries, stream, reps, chain=4):
    """Sec. 5.4 catch-up over a chain of `chain` deltas, each ~1% of the
    Qwen3-8B index space at uniformly random positions (drawn on the GPU):
    delta_compose timed with HIP events, then one apply of the composed
    delta, against replaying the chain delta by delta and against applying
    the chain in one pass (delta_apply_chain, checked first on a second
    copy of the rollout to leave exactly what the composed delta leaves)."""
    import torch
    dev = rollout[0].device
    g = torch.Generator(device=dev)
    g.manual_seed(11456 + 54)
    deltas = []
    for d in range(chain):
        idx = torch.unique(torch.randint(0, N, (K_entries,), device=dev, generator=g))
        val = torch.randint(-32768, 32767, (idx.numel(),), device=dev, generator=g,
                            dtype=torch.int16).view(torch.bfloat16)
        deltas.append((idx, val))
    counts = [i.numel() for i, _ in deltas]
    lib = ad.library()
    ws = torch.empty(ad.delta_compose_workspace_bytes(counts), dtype=torch.uint8, device=dev)
    cap = sum(counts)
    out_i = torch.empty(cap, dtype=torch.int64, device=dev)
    out_v = torch.empty(cap, dtype=torch.bfloat16, device=dev)
    cnt = torch.zeros(1, dtype=torch.int64, device=dev)
    ip = ad._ptr_array([i.data_ptr() for i, _ in deltas])
    vp = ad._ptr_array([v.data_ptr() for _, v in deltas])
    ca = ad._u64_array(counts)
    h = stream.cuda_stream

    def compose():
        st = lib.delta_compose(ip, vp, ca, chain, out_i.data_ptr(), out_v.data_ptr(), cap,
                               cnt.data_ptr(), None, ws.data_ptr(), ws.numel(), h)
        if st:
            raise RuntimeError(lib.delta_last_error().decode())

    compose()
    stream.synchronize()
    k = int(cnt.item())
    apply_ws = torch.empty(max(ad.delta_apply_multi_workspace_bytes(len(rollout)), 1),
                           dtype=torch.uint8, device=dev)
    chain_ws = torch.empty(ad.delta_apply_chain_workspace_bytes(counts, len(rollout)),
                           dtype=torch.uint8, device=dev)
    flag = torch.zeros(1, dtype=torch.int32, device=dev)
    second = [t.clone() for t in rollout]
    ad.delta_apply_multi(rollout, out_i[:k], out_v[:k], workspace=apply_ws, stream=stream)
    ad.delta_apply_chain(second, deltas, error_flag=flag, workspace=chain_ws, stream=stream)
    stream.synchronize()
    if int(flag.item()) or not all(torch.equal(a.view(torch.int16), b.view(torch.int16))
                                   for a, b in zip(rollout, second)):
        raise RuntimeError("the one-pass chain apply differs from applying the composed delta")
    del second
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(reps)]
    for e0, e1, e2, e3, e4 in ev:
        e0.record(stream)
        compose()
        e1.record(stream)
        ad.delta_apply_multi(rollout, out_i[:k], out_v[:k], workspace=apply_ws, stream=stream)
        e2.record(stream)
        for idx, val in deltas:
            ad.delta_apply_multi(rollout, idx, val, workspace=apply_ws, stream=stream)
        e3.record(stream)
        ad.delta_apply_chain(rollout, deltas, workspace=chain_ws, stream=stream)
        e4.record(stream)
    stream.synchronize()
    med = lambda xs: sorted(xs)[len(xs) // 2]
    tc = med([e[0].elapsed_time(e[1]) for e in ev])
    ta = med([e[1].elapsed_time(e[2]) for e in ev])
    tr = med([e[2].elapsed_time(e[3]) for e in ev])
    tch = med([e[3].elapsed_time(e[4]) for e in ev])
    moved = (sum(counts) + k) * 10   # every input entry read once, the result written once
    # longer chains: the one-pass catch-up (merged tile by tile once the
    # chain holds one word in 24) against replaying it delta by delta
    longer = {}
    for K2 in (8, 16):
        while len(deltas) < K2:
            idx = torch.unique(torch.randint(0, N, (K_entries,), device=dev, generator=g))
            val = torch.randint(-32768, 32767, (idx.numel(),), device=dev, generator=g,
                                dtype=torch.int16).view(torch.bfloat16)
            deltas.append((idx, val))
        ch = deltas[:K2]
        cws = torch.empty(ad.delta_apply_chain_workspace_bytes([i.numel() for i, _ in ch],
                                                               len(rollout)),
                          dtype=torch.uint8, device=dev)
        ad.delta_apply_chain(rollout, ch, workspace=cws, stream=stream)
        tl = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(3)]
        for e0, e1, e2 in tl:
            e0.record(stream)
            ad.delta_apply_chain(rollout, ch, workspace=cws, stream=stream)
            e1.record(stream)
            for idx, val in ch:
                ad.delta_apply_multi(rollout, idx, val, workspace=apply_ws, stream=stream)
            e2.record(stream)
        stream.synchronize()
        longer[str(K2)] = {
            "entries": sum(i.numel() for i, _ in ch),
            "catch_up_one_pass_ms": round(med([e[0].elapsed_time(e[1]) for e in tl]), 4),
            "replay_chain_ms": round(med([e[1].elapsed_time(e[2]) for e in tl]), 4),
        }
        del cws
    return {
        "workload": f"{chain} deltas of ~1% random positions of the {N}-word index space "
                    f"({sum(counts)} entries), composed into {k}",
        "compose_ms": round(tc, 4),
        "compose_GBps_one_pass": round(moved / (tc / 1e3) / 1e9, 1),
        "entries_per_s": round(sum(counts) / (tc / 1e3), 1),
        "apply_composed_ms": round(ta, 4),
        "replay_chain_ms": round(tr, 4),
        "catch_up_compose_plus_apply_ms": round(tc + ta, 4),
        "catch_up_one_pass_ms": round(tch, 4),
        "longer_chains": longer,
    }


def single_tensor_measurement(ad, synth, stream, reps):
    """One 2048 x 2048 bf16 tensor with 1% of its words changed, int32
    indices.  Its two copies (16.8 MB) fit in the 256 MB last-level cache:
    "warm" repeats the call; "cold" first writes a 1 GiB scratch buffer,
    which evicts them.  Times are the GPU's: HIP events on the launch stream
    around each call, with a short spin kernel enqueued first so that the
    host has enqueued the whole call before the GPU reaches it (as in a
    stream of calls); the host's own enqueue time and the time with the host
    enqueuing inside the bracket are reported beside.  delta_extract (two
    launches: scan, then a per-tile finalize) and delta_extract_noalloc
    (the same kernels on the library's fixed scratch), each also replayed
    from a HIP graph."""
    import torch
    dev = torch.device("cuda")
    n = 2048 * 2048
    prev, new, pos = synth.make_pair(n, 0.01, seed=synth.config_seed(1), device=dev)
    K = pos.numel()
    idx = torch.empty(K + 64, dtype=torch.int32, device=dev)
    val = torch.empty(K + 64, dtype=torch.bfloat16, device=dev)
    cnt = torch.zeros(1, dtype=torch.int64, device=dev)
    ws = torch.empty(ad.delta_extract_workspace_bytes(n), dtype=torch.uint8, device=dev)
    scratch = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    lib = ad.library()
    med = lambda xs: sorted(xs)[len(xs) // 2]
    spin = 200_000   # cycles of the spin kernel ahead of each timed call

    def run(call, graph):
        out = {}
        for _ in range(3):
            call()
        stream.synchronize()
        if int(cnt.item()) != K:
            raise RuntimeError("config 1: wrong count")
        t = []
        for _ in range(reps):
            t0 = time.perf_counter()
            call()
            t.append(time.perf_counter() - t0)
            stream.synchronize()
        out["host_enqueue_us"] = round(med(t) * 1e6, 2)
        for mode in ("warm", "cold", "host_bound"):
            # the whole call, then (a second pass) the scan kernel alone,
            # bracketed by the library's own events
            times = []
            for scan in (False, True):
                ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)]
                      for _ in range(reps)]
                with torch.cuda.stream(stream):
                    for i, (e0, e1) in enumerate(ev):
                        if mode == "cold":
                            scratch.fill_(i & 0xFF)
                        if scan:
                            e0.record(stream)   # torch creates an event on its first record
                            e1.record(stream)
                            if lib.delta_set_scan_events(e0.cuda_event, e1.cuda_event):
                                raise RuntimeError(lib.delta_last_error().decode())
                        if mode != "host_bound":
                            torch.cuda._sleep(spin)
                        if not scan:
                            e0.record(stream)
                        call()
                        if not scan:
                            e1.record(stream)
                stream.synchronize()
                lib.delta_set_scan_events(None, None)
                times.append(med([e0.elapsed_time(e1) for e0, e1 in ev]))
            call_ms, scan_ms = times
            if mode == "host_bound":
                out["host_bound_ms"] = round(call_ms, 4)
                continue
            out[mode] = {"ms": round(call_ms, 4), "scan_kernel_ms": round(scan_ms, 4),
                         "GBps_scanned": round(4 * n / (call_ms / 1e3) / 1e9, 1)}
        # the same call captured once into a HIP graph (on a side stream, as
        # capture requires) and replayed on the launch stream
        cs = torch.cuda.Stream()
        cs.wait_stream(stream)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cs):
            graph(cs)
        stream.wait_stream(cs)
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(reps)]
        with torch.cuda.stream(stream):
            for e0, e1 in ev:
                torch.cuda._sleep(spin)
                e0.record(stream)
                g.replay()
                e1.record(stream)
        stream.synchronize()
        if int(cnt.item()) != K:
            raise RuntimeError("config 1: wrong count after graph replays")
        gm = med([e0.elapsed_time(e1) for e0, e1 in ev])
        out["graph_warm"] = {"ms": round(gm, 4), "GBps_scanned": round(4 * n / (gm / 1e3) / 1e9, 1)}
        del g
        return out

    noalloc = run(lambda: ad.delta_extract_noalloc_into(prev, new, idx, val, cnt, stream),
                  lambda s: ad.delta_extract_noalloc_into(prev, new, idx, val, cnt, s))
    extract = run(lambda: ad.delta_extract_into(prev, new, idx, val, cnt, ws, stream),
                  lambda s: ad.delta_extract_into(prev, new, idx, val, cnt, ws, s))
    del scratch
    return {"workload": f"one 2048 x 2048 bf16 tensor, {K} changed words (1%), int32 indices",
            "entry": "delta_extract (two launches: scan, per-tile finalize)",
            "warm": extract["warm"], "cold": extract["cold"],
            "delta_extract": dict(extract, launches=2),
            "delta_extract_noalloc": noalloc}


def hash_measurement(ad, buf, stream, reps):
    """XXH64 segment hashes (Sec. 5.2 integrity) of the extracted delta's
    bytes, timed with HIP events, for two segment sizes."""
    import torch
    lib = ad.library()
    nbytes = buf.numel()
    res = {"workload": f"XXH64 segments of the {nbytes}-byte (idx, val) streams of the delta"}
    for seg in (1 << 20, 1 << 16, 1 << 14):
        n = (nbytes + seg - 1) // seg
        out = torch.empty(n, dtype=torch.int64, device=buf.device)
        h = stream.cuda_stream
        call = lambda: lib.delta_hash_segments(buf.data_ptr(), nbytes, seg, 1, out.data_ptr(), h)
        call()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(reps)]
        for e0, e1 in ev:
            e0.record(stream)
            call()
            e1.record(stream)
        stream.synchronize()
        t = sorted(e0.elapsed_time(e1) for e0, e1 in ev)[reps // 2]
        res[f"seg_{seg}"] = {"ms": round(t, 4), "GBps": round(nbytes / (t / 1e3) / 1e9, 1),
                             "segments": n}
    return res


def fused_measurement(ad, synth, ws, model, out_idx, out_val, work, stream, reps):
    """Extraction straight into the fused inference index space (Sec. 5.1:
    qkv_proj, gate_up_proj) on the same weight set, timed with HIP events."""
    import ctypes
    import torch
    targets, sources = synth.qwen3_fused_layout(model)
    plan = ad.MultiPlan(ws.prev, ws.new)
    lib = ad.library()
    tgt = (ctypes.c_int32 * plan.T)(*[f for f, _ in sources])
    boff = ad._u64_array([o for _, o in sources])
    tn = ad._u64_array([n for _, n in targets])
    cnt = torch.zeros(1, dtype=torch.int64, device=out_idx.device)
    offs = torch.zeros(len(targets) + 1, dtype=torch.int64, device=out_idx.device)
    cap = out_idx.numel()
    h = stream.cuda_stream

    def call():
        st = lib.delta_extract_fused(plan.prev_ptrs, plan.next_ptrs, plan.numel_arr, plan.T, tgt,
                                     boff, tn, len(targets), out_idx.data_ptr(),
                                     out_val.data_ptr(), cap, cnt.data_ptr(), offs.data_ptr(),
                                     work.data_ptr(), work.numel(), h)
        if st:
            raise RuntimeError(lib.delta_last_error().decode())

    call()
    stream.synchronize()
    if int(cnt.item()) != ws.total_planted:
        raise RuntimeError("fused extract count differs from the planted changes")
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for e0, e1 in ev:
        e0.record(stream)
        call()
        e1.record(stream)
    stream.synchronize()
    t = sorted(e0.elapsed_time(e1) for e0, e1 in ev)[reps // 2]
    return {"workload": f"{len(ws.prev)} training tensors into {len(targets)} fused targets",
            "ms": round(t, 4), "GBps_scanned": round(4 * ws.total / (t / 1e3) / 1e9, 1)}


def _prefix(xs):
    s = 0
    for x in xs:
        s += x
        yield s


def count_measurement(ad, lib, plan, work, stream, reps, K, scanned, stage_ms):
    """delta_count_changed_multi on the same set: the extract's reads and
    compares with nothing staged or written, i.e. the read cost of the scan
    at the same tile shape; its count must equal the extract's."""
    import torch
    cnt = torch.zeros(1, dtype=torch.int64, device=work.device)
    ad.delta_count_changed_multi_into(plan, cnt, work, stream)
    stream.synchronize()
    if int(cnt.item()) != K:
        raise RuntimeError(f"count {int(cnt.item())} differs from the extract's {K}")
    call, kern = [], []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s0.record(stream)
        s1.record(stream)
        if lib.delta_set_scan_events(s0.cuda_event, s1.cuda_event):
            raise RuntimeError(lib.delta_last_error().decode())
        e0.record(stream)
        ad.delta_count_changed_multi_into(plan, cnt, work, stream)
        e1.record(stream)
        stream.synchronize()
        lib.delta_set_scan_events(None, None)
        call.append(e0.elapsed_time(e1))
        kern.append(s0.elapsed_time(s1))
    call_ms = sum(call) / len(call)
    kern_ms = sum(kern) / len(kern)
    return {
        "workload": "delta_count_changed_multi over the same set (both copies read once, "
                    "nothing staged or written)",
        "ms": round(call_ms, 4),
        "count_kernel_ms": round(kern_ms, 4),
        "count_kernel_GBps": round(scanned / (kern_ms / 1e3) / 1e9, 2),
        "count_kernel_frac_of_peak": round(scanned / (kern_ms / 1e3) / 1e9 / HBM_PEAK_GBPS, 4),
        "stage_kernel_vs_count_kernel": round(kern_ms / stage_ms, 4),
    }


def sweep_measurement(ad, synth, dev, stream, reps):
    """The other weight sets of the benchmark suite beside the headline:
    the Qwen3-8B set at 0.1% and 10% density, the clustered Qwen3-8B set
    (80% of the changes in 5% of the rows) and the Qwen3-4B set, each
    extracted (delta_extract_multi, int64 global indices) and applied
    (delta_apply_multi) ``reps`` times after one warm-up, HIP events around
    every call; the count and the applied rollout are checked."""
    import torch
    out = {}
    cases = [("qwen3-8b_d0.1pct", "qwen3-8b", 0.001, False, 3),
             ("qwen3-8b_d10pct", "qwen3-8b", 0.10, False, 3),
             ("qwen3-8b_clustered", "qwen3-8b", 0.01, True, 4),
             ("qwen3-4b", "qwen3-4b", 0.01, False, 2)]
    for key, model, density, clustered, cfg in cases:
        ws = synth.make_weight_set(model, density, seed=synth.config_seed(cfg), device=dev,
                                   clustered=clustered)
        N, Kp = ws.total, ws.total_planted
        plan = ad.MultiPlan(ws.prev, ws.new).prepare()
        out_idx = torch.empty(Kp + 1024, dtype=torch.int64, device=dev)
        out_val = torch.empty(Kp + 1024, dtype=torch.bfloat16, device=dev)
        cnt = torch.zeros(1, dtype=torch.int64, device=dev)
        work = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=dev)
        roll = [p.clone() for p in ws.prev]
        aws = torch.empty(max(ad.delta_apply_multi_sorted_workspace_bytes(plan.T), 1),
                          dtype=torch.uint8, device=dev)
        ad.delta_extract_multi_into(plan, out_idx, out_val, cnt, work, None, stream)
        torch.cuda.synchronize()
        K = int(cnt.item())
        if K != Kp:
            raise RuntimeError(f"{key}: extract found {K} changed words, {Kp} planted")
        ad.delta_apply_multi(roll, out_idx[:K], out_val[:K], workspace=aws, stream=stream,
                             sorted_indices=True)
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(reps)]
        for e0, e1, e2 in ev:
            e0.record(stream)
            ad.delta_extract_multi_into(plan, out_idx, out_val, cnt, work, None, stream)
            e1.record(stream)
            ad.delta_apply_multi(roll, out_idx[:K], out_val[:K], workspace=aws, stream=stream,
                                 sorted_indices=True)
            e2.record(stream)
        torch.cuda.synchronize()
        for r, q in zip(roll, ws.new):
            if not torch.equal(r.view(torch.int16), q.view(torch.int16)):
                raise RuntimeError(f"{key}: rollout differs from the updated weights")
        med = lambda xs: sorted(xs)[len(xs) // 2]
        te = med([a.elapsed_time(b) for a, b, _ in ev])
        ta = med([b.elapsed_time(c) for _, b, c in ev])
        alg = 4 * N + 10 * K
        out[key] = {"words": N, "changed": K, "extract_ms": round(te, 4),
                    "extract_GBps_scanned": round(4 * N / (te / 1e3) / 1e9, 1),
                    "extract_pct_hbm_peak": round(100 * alg / (te / 1e3) / 1e9 / HBM_PEAK_GBPS, 2),
                    "apply_ms": round(ta, 4),
                    "apply_path": apply_path(N, K),
                    "apply_GBps_algorithmic": round(12 * K / (ta / 1e3) / 1e9, 1),
                    "apply_changed_words_per_s": round(K / (ta / 1e3), 1)}
        log(f"{key}: extract {te:.3f} ms, apply {ta:.3f} ms")
        del ws, plan, out_idx, out_val, work, roll
        torch.cuda.empty_cache()
    return out


def torch_reference_measurement(ws, reps=3):
    """Informational: the same extract written with torch operations only
    (compare, nonzero, gather per tensor; nonzero waits for the host), not
    part of the library."""
    import torch
    times = []
    for _ in range(reps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        total = 0
        for p, q in zip(ws.prev, ws.new):
            pv, qv = p.reshape(-1).view(torch.int16), q.reshape(-1).view(torch.int16)
            i = torch.nonzero(pv != qv).reshape(-1)
            v = qv[i]
            total += i.numel()
            del i, v
        torch.cuda.synchronize()
        times.append((time.perf_counter() - t0) * 1e3)
    ms = sorted(times)[len(times) // 2]
    return {"workload": "torch.nonzero(prev != new) and a gather, tensor by tensor",
            "ms": round(ms, 3), "changed": total,
            "GBps_scanned": round(4 * ws.total / (ms / 1e3) / 1e9, 1)}


def extras(args, ad, synth, ws, rollout, plan, out_idx, out_val, d_offs, work, stream, K, N,
           result):
    """The measurements beside the headline step: LEB128 coding, integrity
    hashing, the fused layout and delta chains (the last one overwrites the
    rollout copy)."""
    import torch
    result["leb128"] = leb128_measurement(ad, plan, out_idx[:K], out_val[:K], d_offs,
                                          plan.numels, rollout, stream, args.steps)
    # the delta's two streams as one byte buffer, as an artifact holds them
    payload = torch.cat([out_idx[:K].view(torch.uint8), out_val[:K].view(torch.uint8)])
    result["hash"] = hash_measurement(ad, payload, stream, args.steps)
    del payload
    result["fused"] = fused_measurement(ad, synth, ws, args.model, out_idx, out_val, work, stream,
                                        args.steps)
    result["compose"] = compose_measurement(ad, rollout, N, K, stream, max(args.steps // 2, 3))
    result["single_tensor"] = single_tensor_measurement(ad, synth, stream, max(args.steps, 20))
    result["torch_reference"] = torch_reference_measurement(ws)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the hot path has no multi-GPU form in this library)", file=sys.stderr)
        return 2

    # the probe runs first, in a process of its own, before this one touches the GPU
    ceilings = None if (args.no_ceilings or args.only_pipeline) else measure_ceilings()
    if ceilings is not None:
        log(f"write ceilings: {ceilings}")

    import torch
    import paper_2602_11456_amd as ad
    from paper_2602_11456_amd import synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    ad.library()   # fail loudly if the HIP library is missing
    if args.only_pipeline:
        print(json.dumps({"pipeline": pipeline_measurement(args, dev)}), flush=True)
        return 0
    # The pipelines run first, in the fresh process: their three busy
    # streams share the process's four hardware queues with every stream
    # created before them, and two busy streams on one queue serialise
    # (the plain pipeline measured 29.4-33.6 ms depending on the streams a
    # process had made before).
    pipeline = None
    if not args.no_pipeline:
        pipeline = pipeline_measurement(args, dev)
        torch.cuda.empty_cache()

    t0 = time.time()
    ws = synth.make_weight_set(args.model, args.density,
                               seed=synth.config_seed(4 if args.clustered else 3), device=dev,
                               clustered=args.clustered)
    torch.cuda.synchronize()
    N = ws.total
    K_planted = ws.total_planted
    log(f"generated {len(ws.prev)} tensors, {N} words, {K_planted} changed "
        f"in {time.time() - t0:.1f} s")

    # the tensor table is built once for the set, as a training loop keeps
    # its weights (delta_multi_plan); every timed step does the whole extract
    plan = ad.MultiPlan(ws.prev, ws.new).prepare()
    cap = K_planted + 1024
    out_idx = torch.empty(cap, dtype=torch.int64, device=dev)
    out_val = torch.empty(cap, dtype=torch.bfloat16, device=dev)
    d_count = torch.zeros(1, dtype=torch.int64, device=dev)
    d_offs = torch.zeros(plan.T + 1, dtype=torch.int64, device=dev)
    work = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=dev)
    rollout = [p.clone() for p in ws.prev]
    apply_ws = torch.empty(max(ad.delta_apply_multi_sorted_workspace_bytes(plan.T), 1),
                           dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def extract():
        ad.delta_extract_multi_into(plan, out_idx, out_val, d_count, work, d_offs, stream)

    def apply(k):
        # the extract's indices are strictly increasing: the sorted entry point
        ad.delta_apply_multi(rollout, out_idx[:k], out_val[:k], workspace=apply_ws,
                             stream=stream, sorted_indices=True)

    # warm-up (also checks the count once)
    extract()
    torch.cuda.synchronize()
    K = int(d_count.item())
    if K != K_planted:
        raise RuntimeError(f"extract found {K} changed words, {K_planted} planted")
    for _ in range(max(args.warmup - 1, 0)):
        extract()
        apply(K)
    apply(K)
    torch.cuda.synchronize()

    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
            torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    # the scan kernel's own launches, bracketed by the library on the same
    # stream (delta_set_scan_events)
    scan_evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                for _ in range(args.steps)]
    for s0, s1 in scan_evs:   # torch creates an event on its first record
        s0.record(stream)
        s1.record(stream)
    lib = ad.library()
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    for (e0, e1, e2), (s0, s1) in zip(evs, scan_evs):
        if lib.delta_set_scan_events(s0.cuda_event, s1.cuda_event):
            raise RuntimeError(lib.delta_last_error().decode())
        e0.record(stream)
        extract()
        e1.record(stream)
        apply(K)
        e2.record(stream)
    t_end.record(stream)
    torch.cuda.synchronize()
    lib.delta_set_scan_events(None, None)

    ext_ms = [e0.elapsed_time(e1) for e0, e1, _ in evs]
    scan_ms = [s0.elapsed_time(s1) for s0, s1 in scan_evs]
    app_ms = [e1.elapsed_time(e2) for _, e1, e2 in evs]
    total_ms = t_start.elapsed_time(t_end)
    ext_avg = sum(ext_ms) / len(ext_ms)
    app_avg = sum(app_ms) / len(app_ms)

    # correctness of the timed state: the rollout equals the new weights
    for r, q in zip(rollout, ws.new):
        if not torch.equal(r.view(torch.int16), q.view(torch.int16)):
            raise RuntimeError("rollout copy differs from the updated weights")

    w = 8   # int64 indices
    scanned = 4 * N
    alg_bytes = scanned + K * (w + 2)
    ext_s = ext_avg / 1e3
    value = scanned / ext_s / 1e9
    achieved = alg_bytes / ext_s / 1e9
    apply_bytes = K * (w + 2) + 2 * K
    traffic = None
    scan_traffic = None
    if args.traffic and os.path.exists(args.traffic):
        with open(args.traffic) as f:
            rec = json.load(f)
        if rec.get("kernel_source_sha256") == kernel_source_digest():
            traffic = rec.get("bytes_per_call")
            for name, k in rec.get("kernels", {}).items():
                if name == "stage_kernel<true, true, false>":   # the planned headline call's
                    scan_traffic = round(k["bytes_per_dispatch"])
    # the dominant kernel: the scan (stage_kernel), whose algorithmic bytes
    # are both copies read once
    scan_avg = sum(scan_ms) / len(scan_ms)
    scan_achieved = scanned / (scan_avg / 1e3) / 1e9

    lines = touched_lines(rollout, out_idx[:K], plan.numels)
    apply_traffic = None
    if args.traffic and os.path.exists(args.traffic):
        with open(args.traffic) as f:
            rec = json.load(f)
        if rec.get("kernel_source_sha256") == kernel_source_digest():
            for name, k in rec.get("kernels", {}).items():
                if "apply_multi_kernel" in name:
                    apply_traffic = round(k["bytes_per_dispatch"])
    ceiling = (ceilings["partial_line_writes_per_s"]
               if ceilings and "partial_line_writes_per_s" in ceilings else None)
    app_s = app_avg / 1e3
    apply_achieved = apply_bytes / app_s / 1e9

    ext_sorted = sorted(ext_ms)
    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(total_ms / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u16",
        "data": "synthetic",
        "config": {
            "workload": f"{args.model} weight set, {len(ws.prev)} tensors, {N} bf16 words, "
                        + (f"{args.density:.2%} of words changed, 80% of them in 5% of the rows"
                           if args.clustered else
                           f"{args.density:.2%} of words changed per tensor")
                        + ", int64 global indices",
            "tensors": len(ws.prev),
            "words": N,
            "changed": K,
            "density": args.density,
            "index": "int64",
            "tensor_table": "built once for the set before the timed steps "
                            "(delta_multi_plan_create), as a training loop keeps its weights",
        },
        "extract": {
            "ms": round(ext_avg, 4),
            "ms_p10": round(ext_sorted[len(ext_sorted) // 10], 4),
            "ms_p90": round(ext_sorted[(9 * len(ext_sorted)) // 10], 4),
            "GBps_scanned": round(value, 2),
            "GBps_algorithmic": round(achieved, 2),
            "pct_hbm_peak": round(100 * achieved / HBM_PEAK_GBPS, 2),
        },
        "apply": {
            "ms": round(app_avg, 4),
            "GBps_algorithmic": round(apply_achieved, 2),
            "changed_words_per_s": round(K / app_s, 1),
            "path": apply_path(N, K),
            "roofline": apply_roofline(N, K, app_s, apply_bytes, apply_achieved, apply_traffic,
                                       lines, ceiling, ceilings),
        },
        "roofline": {
            "kernel": "stage_kernel (reads and compares both copies)",
            "bound": "hbm",
            "achieved": round(scan_achieved, 2),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(scan_achieved / HBM_PEAK_GBPS, 4),
            "traffic": scan_traffic,
            "ms": round(scan_avg, 4),
            "algorithmic_bytes": scanned,
        },
        "roofline_extract_call": {
            "kernels": "stage + group sum + group scan + finalize (the tensor table is the "
                       "plan's, built once)",
            "bound": "hbm",
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": traffic,
            "algorithmic_bytes": alg_bytes,
        },
    }
    result["count_only"] = count_measurement(ad, lib, plan, work, stream, args.steps, K, scanned,
                                             scan_avg)
    if not args.no_extras:
        extras(args, ad, synth, ws, rollout, plan, out_idx, out_val, d_offs, work, stream, K, N,
               result)
    if args.copy_calibration > 0:
        n = args.copy_calibration // 2
        src = torch.empty(n, dtype=torch.int16, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if not args.no_cpu_baseline:
        del rollout
        rollout = None
        result["cpu_baseline"] = cpu_baseline(ws, args.cpu_seconds)
    del ws, plan, out_idx, out_val, work
    rollout = None
    torch.cuda.empty_cache()
    if not args.no_sweep:
        result["sweep"] = sweep_measurement(ad, synth, dev, stream, 5)
    if pipeline is not None:
        result["pipeline"] = pipeline
    result["device"] = device_info(dev)
    print(json.dumps(result), flush=True)
    return 0


def device_info(dev):
    """The device's properties as the runtime reports them (CU count, cache
    and memory sizes), next to the figures they bound."""
    import torch
    p = torch.cuda.get_device_properties(dev)
    return {
        "name": p.name,
        "arch": getattr(p, "gcnArchName", ""),
        "compute_units": p.multi_processor_count,
        "hbm_bytes": p.total_memory,
        "l2_bytes": getattr(p, "L2_cache_size", None),
        "lds_bytes_per_workgroup": getattr(p, "shared_memory_per_block", None),
        "torch": torch.__version__,
        "hip": torch.version.hip,
    }


if __name__ == "__main__":
    sys.exit(main())
