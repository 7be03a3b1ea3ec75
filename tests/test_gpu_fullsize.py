"""GPU parity at the full sizes of the five workloads.

Every instance is a full-length trace.  The one-touch 4096-block batch is
replayed exactly as bench.py times it (16 traces x 3 policies = 48
instances, 50,000 requests each, one batch) and every instance is compared
with the oracle.  The larger batches are replayed on a sample of their seeds
(the trace length, capacities, policies and refill sweep are the full ones);
there the oracle checks a sample of instances and every instance is checked
against invariants that hold at any size."""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle
from gpu_util import assert_same
from paper_2608_01657_amd import device as dv
from paper_2608_01657_amd import tracegen as tg

pytestmark = pytest.mark.gpu

WORKERS = min(16, os.cpu_count() or 1)


def _hash_all(traces, check_keys=(0,)):
    """Hash every trace on the GPU; keys of the traces in `check_keys` are
    compared with the oracle's.  Returns device traces and oracle keys."""
    dts = [dv.upload(tr) for tr in traces]
    for t in dts:
        dv.cut_and_hash(t)
    with ThreadPoolExecutor(WORKERS) as ex:
        okeys = list(ex.map(oracle.hash_trace, traces))
    for i, t in enumerate(dts):
        assert int(t.status.item()) == 0
        assert np.array_equal(t.key_off.cpu().numpy(), okeys[i][1]), f"trace {i}: key offsets differ"
        if i in check_keys:
            keys = t.keys[:t.n_keys].cpu().numpy().view(np.uint64)
            assert np.array_equal(keys, okeys[i][0]), f"trace {i}: keys differ"
    return dts, okeys


def _invariants(groups, inst, spec, n_req):
    """Properties of any replay: conservation of probes, charges and
    residency (every block is keyed in its group's namespace, so an orphan's
    owner is its requester)."""
    tot = lambda f: sum(g[f] for g in groups)
    assert tot("requests") == n_req
    for g in groups:
        assert g["hits"] + g["misses"] == g["probes"]
        assert g["charged"] == g["misses"] - g["dups"]
        assert g["resident_end"] == g["charged"] - g["evicted_owned"] - g["orphans"]
        assert 0 <= g["resident_end"] <= g["resident_max"] <= spec.capacity
        assert g["debt_end_q16"] <= g["debt_max_q16"]
    assert tot("evicted_owned") == tot("evictions_caused") == inst["evictions"]
    assert 0 <= inst["resident_end"] <= inst["resident_max"] <= spec.capacity
    assert inst["resident_end"] == tot("resident_end")
    if spec.policy != tg.POLICY_PREFIXSHIELD:
        assert tot("promotions") == 0 and tot("gated") == 0


def _replay_and_compare(traces, insts, dts, okeys, oracle_ids):
    b = dv.ReplayBatch(dts, insts)
    b.launch()
    res = b.results()

    def orc(k):
        spec = insts[k]
        return k, oracle.replay_trace(traces[spec.trace], okeys[spec.trace][0], okeys[spec.trace][1], spec)

    with ThreadPoolExecutor(WORKERS) as ex:
        outs = list(ex.map(orc, oracle_ids))
    for k, o in outs:
        assert_same(res[k], o, f"instance {k} ({insts[k].label}, seed trace {insts[k].trace})")
    for k, (groups, inst, status) in enumerate(res):
        assert status == 0
        _invariants(groups, inst, insts[k], traces[insts[k].trace].n_req)
    return res


def test_onetouch4096_bench_batch_all_instances():
    traces, insts = tg.workload("onetouch4096")
    assert len(insts) == 48 and all(t.n_req == 50000 for t in traces)
    dts, okeys = _hash_all(traces, check_keys=range(len(traces)))
    _replay_and_compare(traces, insts, dts, okeys, range(len(insts)))


def test_twopass_full_length_sampled_seeds():
    traces, insts = tg.workload("twopass", seeds=[0, 1, 2, 3])
    assert all(t.n_req == 80000 for t in traces)
    dts, okeys = _hash_all(traces)
    _replay_and_compare(traces, insts, dts, okeys, range(len(insts)))


def test_delayed_full_length_refill_sweep():
    traces, insts = tg.workload("delayed", seeds=[0, 1])
    assert all(t.n_req == 200000 for t in traces) and len(insts) == 48
    dts, okeys = _hash_all(traces)
    # oracle: every policy at the lowest and highest refill rate of seed 0
    sample = [k for k, i in enumerate(insts) if i.trace == 0 and ("_rho1" == i.label[-5:] or i.label.endswith("_rho128"))]
    assert len(sample) == 6
    _replay_and_compare(traces, insts, dts, okeys, sample)


def test_chat_full_length_all_capacities():
    """Capacities up to 16,384 blocks: the larger ones keep their state in the
    workspace instead of LDS.  StaticQuota too: 16 partitions, so at 1,024
    blocks a 64-block partition truncates most long prompts."""
    traces, insts = tg.workload("chat", seeds=[0, 1], policies=tg.ALL_POLICIES + (tg.POLICY_STATICQUOTA,))
    assert all(t.n_req == 100000 for t in traces) and len(insts) == 40
    dts, okeys = _hash_all(traces)
    sample = [k for k, i in enumerate(insts) if i.trace == 0]
    _replay_and_compare(traces, insts, dts, okeys, sample)


def test_scale1024_sampled():
    """1,024 concurrent 4096-block instances (16 traces x 64 policy variants);
    the oracle checks LRU, S3-FIFO and three refill rates of one trace."""
    traces, insts = tg.workload("scale1024")
    assert len(insts) == 1024
    dts, okeys = _hash_all(traces)
    sample = [k for k, i in enumerate(insts) if i.trace == 5 and
              (i.policy != tg.POLICY_PREFIXSHIELD or i.label.split("rho")[-1] in ("1/4", "16/4", "62/4"))]
    assert len(sample) == 5
    _replay_and_compare(traces, insts, dts, okeys, sample)


def test_tiers_full_length_all_instances():
    """Three contract tiers (normalized debt, Eq. 5; a group with two
    contracts), full length, every instance against the oracle."""
    traces, insts = tg.workload("tiers", seeds=[0, 1])
    assert all(t.n_req == 50000 for t in traces) and len(insts) == 6
    dts, okeys = _hash_all(traces, check_keys=(0, 1))
    _replay_and_compare(traces, insts, dts, okeys, range(len(insts)))


def test_attack_traces_all_variants_per_request():
    """The paper-scale attack traces (C = 511), every variant including the
    two ablations and StaticQuota, per-request outputs too."""
    for kind in tg.ATTACK_KINDS:
        traces, insts = tg.workload("attack_" + kind, seeds=[0, 1])
        assert len(insts) == 12
        dts, okeys = _hash_all(traces, check_keys=(0, 1))
        b = dv.ReplayBatch(dts, insts, per_request=True)
        b.launch()
        res = b.results()
        pr = b.per_request_arrays()
        for k, spec in enumerate(insts):
            o = oracle.replay_trace(traces[spec.trace], okeys[spec.trace][0], okeys[spec.trace][1], spec,
                                    per_request=True)
            assert_same(res[k], o, f"{kind} {spec.label}")
            assert np.array_equal(pr[k], o.per_request), f"{kind} {spec.label}: per-request outputs differ"


def test_chat_bursty_ticks_full_length():
    """Conversational traces with bursty arrival ticks (Eq. 1's clock), full length."""
    traces, insts = tg.workload("chat_bursty", seeds=[0])
    assert traces[0].n_req == 100000 and traces[0].tick is not None
    dts, okeys = _hash_all(traces)
    _replay_and_compare(traces, insts, dts, okeys, range(len(insts)))


def test_selector_contention_all_instances():
    """Every request reclaims under contention from 8 / 32 indebted groups
    (the selector measurement sizes), full length, all instances."""
    for name in ("selector512x8", "selector4096x32"):
        traces, insts = tg.workload(name, seeds=[0])
        assert traces[0].n_req == 20000
        dts, okeys = _hash_all(traces)
        _replay_and_compare(traces, insts, dts, okeys, range(len(insts)))


PHASE_CHILD = r"""
import json, sys, numpy as np
sys.path.insert(0, sys.argv[1]); sys.path.insert(0, sys.argv[1] + "/tests")
import paper_2608_01657_amd as P
P.use_phase_counters()
import oracle
from gpu_util import assert_same
from paper_2608_01657_amd import device as dv, tracegen as tg
traces, insts = tg.workload("selector512x8", seeds=[0], n_requests=3000)
t = dv.upload(traces[0]); dv.cut_and_hash(t)
b = dv.ReplayBatch([t], insts, per_request=True); b.launch()
res = b.results(); pr = b.per_request_arrays(); pcs = b.phase_counters()
k, off = oracle.hash_trace(traces[0])
out = []
for i, spec in enumerate(insts):
    o = oracle.replay_trace(traces[0], k, off, spec, per_request=True)
    assert_same(res[i], o, spec.label)
    assert np.array_equal(pr[i], o.per_request)
    assert pcs[i]["evicting_requests"] == int((o.per_request[:, 2] > 0).sum())
    assert all(pcs[i]["cycles_" + n] > 0 for n in P.PHASE_NAMES if n != "reclamation")
    out.append(pcs[i])
print(json.dumps(out))
"""


def test_phase_counter_library_replays_identically():
    """The phase-counter build changes no result, and its event counts agree
    with the per-request outputs (requests that evicted)."""
    import json
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, "-c", PHASE_CHILD, root], capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-3000:]
    pcs = json.loads(r.stdout.strip().splitlines()[-1])
    assert len(pcs) == 3
