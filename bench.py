#!/usr/bin/env python3
"""Benchmark of the batched prefix-cache replay hot path on one MI355X.

One step = the whole path over one batch of synthetic traces, inputs already
resident in HBM: block offsets and chained keys for every trace (hashing),
then replay of every instance (LRU, S3-FIFO, PrefixShield) from an empty
cache.  Prints one JSON line.

  python bench.py [--steps K] [--warmup W] [--workload scale1024|onetouch4096|chat|...]

The default workload is the 1,024-instance batch: 16 one-touch traces of
50,000 requests, each replayed by 64 concurrent 4096-block instances (LRU,
S3-FIFO, PrefixShield at 62 refill rates).  value = block probes / s of the
whole step (requests/s is reported beside it).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
ROOT = os.path.dirname(os.path.abspath(__file__))
# Counter summaries of the replay kernel per workload (rocprofv3, committed
# under profiles/): calibrated HBM bytes (FETCH_SIZE / WRITE_SIZE against a
# device copy) and LDS / occupancy figures.  Each is valid only for the batch
# and the kernel source it was measured on.
PROFILES = os.path.join(ROOT, "profiles")
# what the replay kernel is built from: its sources and its compiler flags
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_01657_amd", *f) for f in
                  (("csrc", "pc_replay.hip"), ("csrc", "pc_replay_global.hip"), ("csrc", "pc_internal.h"),
                   ("build.py",))]
HASH_BYTES_PER_BLOCK = 64 + 8  # 16 int32 tokens in, one uint64 key out
HASH_BYTES_PER_REQ = 8 + 4 + 4 + 8 + 8   # tok_off, len, ns, key_off read, key_off write
REPLAY_BYTES_PER_PROBE = 8     # the key
REPLAY_BYTES_PER_REQ = 8 + 1 + 1 + 4     # key offset, group, contract, prefix id


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="scale1024")
    ap.add_argument("--seeds", type=int, default=None, help="number of traces (default: the workload's)")
    ap.add_argument("--requests", type=int, default=None, help="requests per trace (default: the workload's)")
    ap.add_argument("--capacities", default=None,
                    help="comma-separated capacities in blocks (workloads with a capacity sweep, e.g. chat)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-requests", type=int, default=0,
                    help="requests per trace in the oracle baseline (0: all of them)")
    ap.add_argument("--cpu-sample-traces", type=int, default=0,
                    help="traces whose instances the oracle baseline replays (0: enough for one instance "
                         "per host thread)")
    ap.add_argument("--phase-profile", action="store_true",
                    help="use the phase-counter library and add per-phase cycles, reclamation latency per "
                         "evicting request and state bytes per cached block to the JSON line")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MiB (3 times) and exit: the "
                         "known-size kernel that HBM byte counters are scaled against")
    return ap.parse_args()


def kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def profile_keys(path, workload, n_traces, n_req):
    """The key: value lines of a committed counter summary, or None when it
    is missing or was taken on another batch or kernel source."""
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#") and not line.startswith(" "):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256") != kernel_source_hash():
        return None
    if kv.get("batch") != f"{workload} traces={n_traces} requests={n_req}":
        return None
    return kv


def measured_traffic(workload, n_traces, n_req):
    """HBM bytes per replay launch (calibrated FETCH_SIZE + WRITE_SIZE)."""
    kv = profile_keys(os.path.join(PROFILES, f"replay_kernel_{workload}_hbm_traffic.txt"), workload, n_traces, n_req)
    try:
        return int(kv["traffic_bytes_per_launch"]) if kv else None
    except (KeyError, ValueError):
        return None


def measured_lds(workload, n_traces, n_req):
    """LDS side of the replay roofline from the committed counter summary:
    the fraction of kernel cycles a CU's LDS is busy, the share of those
    cycles lost to bank conflicts, and workgroups (instances) per busy CU."""
    kv = profile_keys(os.path.join(PROFILES, f"replay_kernel_{workload}_lds_occupancy.txt"), workload, n_traces,
                      n_req)
    if not kv:
        return None
    try:
        return {"lds_busy_frac": float(kv["lds_busy_per_cu_frac"]),
                "bank_conflict_frac_of_busy": float(kv["lds_bank_conflict_frac"]),
                "instances_per_cu": float(kv["mean_workgroups_per_active_cu"]),
                "source": f"profiles/replay_kernel_{workload}_lds_occupancy.txt"}
    except (KeyError, ValueError):
        return None


def calibrate_copy(mib):
    import torch
    n = mib << 20
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "device copy", "bytes_read_per_launch": n, "bytes_written_per_launch": n,
                      "launches": 3}))


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: this build measures one GPU only; replay instances are independent and "
              "would shard across GPUs with no collective, but no multi-GPU run is part of it.",
              file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy_mib:
        calibrate_copy(args.calibrate_copy_mib)
        return
    import torch
    import paper_2608_01657_amd as P
    if args.phase_profile:
        P.use_phase_counters()
    from paper_2608_01657_amd import device as dv
    from paper_2608_01657_amd import tracegen as tg

    t0 = time.time()
    seeds = list(range(args.seeds)) if args.seeds else None
    kw = {}
    if args.capacities:
        kw["capacities"] = [int(c) for c in args.capacities.split(",")]
    traces, insts = tg.workload(args.workload, seeds=seeds, n_requests=args.requests, **kw)
    gen_s = time.time() - t0
    print(f"[bench] generated {len(traces)} traces, {len(insts)} instances in {gen_s:.1f}s", file=sys.stderr,
          flush=True)

    # every trace in one set of device buffers: one offsets call and one
    # hash call per step for the whole batch
    ts = dv.TraceSet(traces)
    ts.hash()                           # sizes the key buffer
    torch.cuda.synchronize()
    assert int(ts.dt.status.item()) == 0
    batch = dv.ReplayBatch(ts.views, insts)
    stream = torch.cuda.current_stream()

    n_req_total = sum(traces[i.trace].n_req for i in insts)
    n_blocks_hash = ts.dt.n_keys
    n_req_hash = ts.dt.n_req

    def step(ev=None):
        if ev:
            ev[0].record(stream)
        ts.hash()
        if ev:
            ev[1].record(stream)
        batch.launch()
        if ev:
            ev[2].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for k in range(args.steps):
        step(evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    hash_each = [e[0].elapsed_time(e[1]) for e in evs]
    replay_each = [e[1].elapsed_time(e[2]) for e in evs]
    hash_ms = float(np.mean(hash_each))
    replay_ms = float(np.mean(replay_each))
    step_ms = wall * 1000.0 / args.steps

    res = batch.results()
    assert all(st == 0 for _, _, st in res), "an instance reported an error status"
    probes = sum(sum(g["probes"] for g in gr) for gr, _, _ in res)
    hits = sum(sum(g["hits"] for g in gr) for gr, _, _ in res)

    # roofline: replay kernel (dominant) against HBM with its algorithmic bytes
    replay_bytes = probes * REPLAY_BYTES_PER_PROBE + n_req_total * REPLAY_BYTES_PER_REQ
    replay_gbs = replay_bytes / (replay_ms * 1e-3) / 1e9
    hash_bytes = n_blocks_hash * HASH_BYTES_PER_BLOCK + n_req_hash * HASH_BYTES_PER_REQ
    hash_gbs = hash_bytes / (hash_ms * 1e-3) / 1e9
    dominant = "replay" if replay_ms >= hash_ms else "hash"
    # the replay kernel of the layout most instances use (one launch per
    # footprint class; a single class runs on the caller's stream)
    _, layouts = P.pc_replay_state_bytes(batch.tdesc, batch.idesc)
    lay = max(set(layouts), key=layouts.count)
    roof = {"kernel": f"replay_kernel<{lay}> ({P.LAYOUT_NAMES[lay]} layout)" if dominant == "replay" else "hash_kernel",
            "layout_instances": {P.LAYOUT_NAMES[x]: layouts.count(x) for x in sorted(set(layouts))},
            "bound": "hbm",
            "achieved": round(replay_gbs if dominant == "replay" else hash_gbs, 3),
            "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round((replay_gbs if dominant == "replay" else hash_gbs) / HBM_PEAK_GBS, 6),
            "traffic": measured_traffic(args.workload, len(traces), traces[0].n_req) if dominant == "replay" else None,
            "lds": measured_lds(args.workload, len(traces), traces[0].n_req) if dominant == "replay" else None,
            "bytes_per_launch": int(replay_bytes if dominant == "replay" else hash_bytes),
            "avg_launch_ms": round(replay_ms if dominant == "replay" else hash_ms, 4)}
    roof_hash = {"kernel": "hash_kernel (+ block offsets), all traces in one call", "bound": "hbm",
                 "achieved": round(hash_gbs, 2),
                 "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(hash_gbs / HBM_PEAK_GBS, 4),
                 "bytes_per_launch": int(hash_bytes), "avg_ms": round(hash_ms, 4),
                 "tokens_per_s": (n_blocks_hash * 16) / (hash_ms * 1e-3)}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(traces, insts, args.cpu_sample_requests, args.cpu_sample_traces)

    phases = phase_report(batch, insts, traces, replay_ms) if args.phase_profile else None
    if phases is not None:
        phases["oracle_reclamation"] = oracle_reclamation(traces, insts)

    value = probes / (step_ms * 1e-3)
    out = {
        "metric": "block probes/sec (batched replay, 1 GPU)",
        "value": value,
        "unit": "probes/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": step_ms,
        "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {"workload": args.workload, "traces": len(traces), "instances": len(insts),
                   "requests_per_trace": traces[0].n_req, "capacity_blocks": sorted({i.capacity for i in insts}),
                   "block_tokens": 16, "policies": sorted({tg.POLICY_NAMES[i.policy] for i in insts})},
        "requests_per_s": n_req_total / (step_ms * 1e-3),
        "replay_probes_per_s": probes / (replay_ms * 1e-3),
        "replay_requests_per_s": n_req_total / (replay_ms * 1e-3),
        "hash_ms": hash_ms, "replay_ms": replay_ms,
        "hash_ms_median_min_max": [float(np.median(hash_each)), float(min(hash_each)), float(max(hash_each))],
        "replay_ms_median_min_max": [float(np.median(replay_each)), float(min(replay_each)), float(max(replay_each))],
        "probes_per_step": probes, "hits_per_step": hits, "requests_per_step": n_req_total,
        "roofline": roof,
        "roofline_hash": roof_hash,
        "cpu_baseline": cpu,
    }
    if phases is not None:
        out["phase_profile"] = phases
    print(json.dumps(out))


def phase_report(batch, insts, traces, replay_ms):
    """Per policy: mean cycles per request of each phase, the reclamation
    cycles of a request that evicts (converted to microseconds with the
    shader clock's rate, measured by every instance as its span in shader
    cycles over its span on the 100 MHz real-time clock), and state bytes
    per cached block."""
    import paper_2608_01657_amd as P
    from paper_2608_01657_amd import tracegen as tg
    pcs = batch.phase_counters()
    totals = [sum(pc[f"cycles_{n}"] for n in P.PHASE_NAMES) for pc in pcs]
    mhz = sum(pc["span_cycles"] for pc in pcs) / (sum(pc["span_ticks_100mhz"] for pc in pcs) / 100.0)
    sbytes, layout = P.pc_replay_state_bytes(batch.tdesc, batch.idesc)
    rep = {"clock_cycles_per_us": round(mhz, 1),
           "instance_span_ms_mean": round(float(np.mean([pc["span_ticks_100mhz"] for pc in pcs])) / 1e5, 3),
           "replay_ms": round(replay_ms, 3)}
    for pol in sorted({i.policy for i in insts}):
        ks = [k for k, i in enumerate(insts) if i.policy == pol]
        nreq = sum(traces[insts[k].trace].n_req for k in ks)
        ev = sum(pcs[k]["evicting_requests"] for k in ks)
        r = {n: round(sum(pcs[k][f"cycles_{n}"] for k in ks) / nreq, 1) for n in P.PHASE_NAMES}
        r["us_per_request"] = round(sum(totals[k] for k in ks) / nreq / mhz, 3)
        r["reclaim_us_per_evicting_request"] = round(sum(pcs[k]["cycles_reclamation"] for k in ks) / max(ev, 1) / mhz, 3)
        r["evicting_requests"] = ev
        r["state_bytes_per_block"] = round(float(np.mean([sbytes[k] / insts[k].capacity for k in ks])), 1)
        r["state_layout"] = sorted({P.LAYOUT_NAMES[layout[k]] for k in ks})
        for n in P.PHASE_EVENTS[1:]:
            r[n] = sum(pcs[k][n] for k in ks)
        rep[tg.POLICY_NAMES[pol]] = r
    return rep


def oracle_reclamation(traces, insts):
    """The oracle's reclamation (Alg. 2 one victim selection at a time, with
    its per-group and per-segment lists) timed per request that evicts, on
    the instances of the first trace, one host thread per instance: mean and
    95th percentile per policy, and per victim."""
    import oracle
    from paper_2608_01657_amd import tracegen as tg
    tr = traces[0]
    sample = [i for i in insts if i.trace == 0]
    keys, off = oracle.hash_trace(tr)
    with ThreadPoolExecutor(max_workers=max(1, min(os.cpu_count() or 1, len(sample)))) as ex:
        outs = list(ex.map(lambda i: oracle.replay_trace(tr, keys, off, i, per_request=True, time_reclaim=True),
                           sample))
    rep = {}
    for pol in sorted({i.policy for i in sample}):
        ns = [o.reclaim_ns[o.per_request[:, 2] > 0] for i, o in zip(sample, outs) if i.policy == pol]
        nv = sum(int(o.per_request[:, 2].sum()) for i, o in zip(sample, outs) if i.policy == pol)
        allns = np.concatenate(ns) if ns else np.zeros(0)
        if allns.size:
            rep[tg.POLICY_NAMES[pol]] = {"us_per_evicting_request": round(float(allns.mean()) / 1e3, 3),
                                         "p95_us": round(float(np.percentile(allns, 95)) / 1e3, 3),
                                         "ns_per_victim": round(float(allns.sum()) / max(nv, 1), 1),
                                         "evicting_requests": int(allns.size)}
    rep["sample"] = f"trace 0, its {len(sample)} instances, one host thread each ({cpu_model()})"
    return rep


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(traces, insts, sample_requests, sample_traces):
    """The oracle (plain single-threaded C per instance) on the host cores,
    one instance per thread on every host core: hash of the sampled traces
    (their first `sample_requests` requests, all if 0), then replay of every
    instance of those traces.  The sample is the first traces of the
    workload, enough of them for one instance per thread (the instances of
    one trace are the workload's mix of policies and parameters)."""
    import oracle
    from paper_2608_01657_amd import tracegen as tg

    nproc = os.cpu_count() or 1
    n_tr = sample_traces
    if n_tr <= 0:
        n_tr, per = 0, 0
        while n_tr < len(traces) and per < nproc:
            per += sum(1 for i in insts if i.trace == n_tr)
            n_tr += 1
    n_tr = max(1, min(n_tr, len(traces)))
    sub = []
    for tr in traces[:n_tr]:
        n = tr.n_req if sample_requests <= 0 else min(sample_requests, tr.n_req)
        sub.append(tg.Trace(tr.name, tr.tokens, tr.tok_off[:n], tr.length[:n], tr.group[:n], tr.contract[:n],
                            tr.prefix[:n], tr.n_groups, tr.n_prefix, None if tr.tick is None else tr.tick[:n]))
    sample = [i for i in insts if i.trace < n_tr]
    threads = max(1, min(nproc, len(sample)))
    t0 = time.perf_counter()
    c0 = time.process_time()
    def timed(f, *a):
        t = time.perf_counter()
        r = f(*a)
        return r, time.perf_counter() - t

    with ThreadPoolExecutor(max_workers=threads) as ex:
        hashed_t = list(ex.map(lambda tr: timed(oracle.hash_trace, tr), sub))
        hashed = [h for h, _ in hashed_t]
        rep_t = list(ex.map(lambda i: timed(oracle.replay_trace, sub[i.trace], hashed[i.trace][0],
                                            hashed[i.trace][1], i), sample))
    wall = time.perf_counter() - t0
    cpu_s = time.process_time() - c0
    results = [r for r, _ in rep_t]
    probes = sum(sum(g["probes"] for g in r.groups) for r in results)
    reqs = sum(sub[i.trace].n_req for i in sample)
    # each call runs on one thread: per-instance replay rates, hashed tokens
    # (full blocks) per second of one thread
    per_inst = [sum(g["probes"] for g in r.groups) / dt for r, dt in rep_t if dt > 0]
    hashed_tokens = sum(int((tr.length.astype(np.int64) // 16).sum()) * 16 for tr in sub)
    hash_s = sum(dt for _, dt in hashed_t)
    return {"value": probes / wall, "unit": "probes/s", "cores": threads, "kind": "oracle",
            "nproc": nproc, "cpu_model": cpu_model(),
            "requests_per_s": reqs / wall, "probes_per_s_per_thread": probes / cpu_s if cpu_s > 0 else None,
            "instance_probes_per_s_median": float(np.median(per_inst)) if per_inst else None,
            "hash_tokens_per_s_per_thread": hashed_tokens / hash_s if hash_s > 0 else None,
            "wall_s": wall,
            "sample": f"{'all' if all(s.n_req == t.n_req for s, t in zip(sub, traces)) else 'the first'} "
                      f"{sub[0].n_req} requests of trace{'s' if n_tr > 1 else ''} 0"
                      f"{'-' + str(n_tr - 1) if n_tr > 1 else ''} of {len(traces)}, all {len(sample)} of their "
                      f"instances (of {len(insts)}): oracle hash + replay, {probes} probes, "
                      f"{cpu_s:.1f}s CPU in {wall:.2f}s wall on {threads} threads"}


if __name__ == "__main__":
    main()
