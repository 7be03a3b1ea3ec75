"""Policy-level experiments on the synthetic stand-ins, run on the GPU.

    python -m paper_2608_01657_amd.experiments [--seeds N] [--json FILE]

What the paper measures with vLLM on its own traces (Sec. V-B to V-D), this
measures on the replay engine with the seeded synthetic traces of tracegen:

  attacks   victim hit ratio (mean over victim requests of cached tokens /
            prompt tokens) under no attack, one-touch pollution, low-and-slow
            rotation and replay pollution, for LRU, S3-FIFO, StaticQuota,
            PrefixShield and the two ablations (no segmentation, no debt
            gate), with paired
            bootstrap CIs over seeds (Sec. V-B, Table I; Sec. V-D, Fig. 3)
            The polluter's debt-gated and promoted blocks are reported for
            PrefixShield with and without the gate (Sec. V-D).
  benign    all-request hit ratio on the conversational trace and its bursty
            variant at C = 4096 (Sec. V-C, Table II)

The traces are stand-ins, not the paper's, so the numbers are context for
the policies' behaviour, not a reproduction.  Everything is computed by the
HIP path; no host fallback exists.
"""
from __future__ import annotations

import argparse
import json
import sys
from collections import defaultdict

import numpy as np


def _run(traces, insts, per_request=True):
    from . import device as dv
    dts = [dv.upload(tr) for tr in traces]
    for t in dts:
        dv.cut_and_hash(t)
    b = dv.ReplayBatch(dts, insts, per_request=per_request)
    b.launch()
    res = b.results()
    pr = b.per_request_arrays() if per_request else None
    for gr, inst, st in res:
        if st != 0:
            raise RuntimeError(f"replay status {st}")
    return res, pr


def attacks(seeds, n_requests=4000):
    from . import metrics, tracegen as tg
    out = {}
    for kind in tg.ATTACK_KINDS:
        traces, insts = tg.workload("attack_" + kind, seeds=seeds, n_requests=n_requests)
        res, pr = _run(traces, insts)
        per = defaultdict(list)   # label -> [victim hit ratio per seed]
        gate = defaultdict(lambda: [0, 0])   # label -> polluter [gated, promoted]
        for k, spec in enumerate(insts):
            per[spec.label].append(metrics.mean_hit_ratio(pr[k], traces[spec.trace], group=0))
            gate[spec.label][0] += res[k][0][1]["gated"]
            gate[spec.label][1] += res[k][0][1]["promotions"]
        row = {lab: 100 * float(np.mean(v)) for lab, v in per.items()}
        cmp = {}
        for a, b in [("prefixshield", "lru"), ("prefixshield", "s3fifo"), ("prefixshield", "staticquota"),
                     ("prefixshield", "prefixshield_noseg"), ("prefixshield", "prefixshield_nogate")]:
            m, lo, hi = metrics.paired_bootstrap(per[a], per[b])
            cmp[f"{a} - {b}"] = [100 * m, 100 * lo, 100 * hi]
        out[kind] = {"victim_hit_pct": row, "paired_pp": cmp,
                     "polluter_gated_promoted": {lab: gate[lab] for lab in ("prefixshield", "prefixshield_nogate")}}
    return out


def benign(seeds, n_requests=100000):
    from . import metrics, tracegen as tg
    ALL4 = tg.ALL_POLICIES + (tg.POLICY_STATICQUOTA,)
    out = {}
    for name in ("chat", "chat_bursty"):
        if name == "chat":
            traces, insts = tg.workload(name, seeds=seeds, n_requests=n_requests, capacities=[4096],
                                        policies=ALL4)
        else:
            traces, insts = tg.workload(name, seeds=seeds, n_requests=n_requests, policies=ALL4)
        res, pr = _run(traces, insts)
        per = defaultdict(list)
        for k, spec in enumerate(insts):
            per[spec.label.split("_C")[0]].append(metrics.mean_hit_ratio(pr[k], traces[spec.trace]))
        m, lo, hi = metrics.paired_bootstrap(per["prefixshield"], per["s3fifo"])
        out[name] = {"hit_pct": {lab: 100 * float(np.mean(v)) for lab, v in per.items()},
                     "paired_pp": {"prefixshield - s3fifo": [100 * m, 100 * lo, 100 * hi]}}
    return out


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--seeds", type=int, default=10)
    ap.add_argument("--benign-seeds", type=int, default=4)
    ap.add_argument("--json", default=None)
    args = ap.parse_args(argv)
    out = {"attacks": attacks(list(range(args.seeds))),
           "benign": benign(list(range(args.benign_seeds)))}
    for kind, r in out["attacks"].items():
        print(f"attack {kind:9s} victim hit %: " + "  ".join(f"{k}={v:.2f}" for k, v in r["victim_hit_pct"].items()))
        for k, (m, lo, hi) in r["paired_pp"].items():
            print(f"    {k:38s} {m:+7.2f} pp  [{lo:+.2f}, {hi:+.2f}]")
        print("    polluter blocks gated / promoted: " +
              "  ".join(f"{k}={v[0]}/{v[1]}" for k, v in r["polluter_gated_promoted"].items()))
    for name, r in out["benign"].items():
        print(f"benign {name:11s} hit %: " + "  ".join(f"{k}={v:.2f}" for k, v in r["hit_pct"].items()))
        for k, (m, lo, hi) in r["paired_pp"].items():
            print(f"    {k:38s} {m:+7.2f} pp  [{lo:+.2f}, {hi:+.2f}]")
    if args.json:
        with open(args.json, "w") as f:
            json.dump(out, f, indent=1)
    return 0


if __name__ == "__main__":
    sys.exit(main())
