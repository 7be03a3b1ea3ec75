"""GPU parity at the full sizes of the five workloads and the 1,024-instance
scale batch: every instance of every workload is compared with the oracle.

Each workload is replayed as bench.py times it: all its traces keyed on the
GPU, then every instance in one pc_replay_batch launch.  The oracle keys every
trace (compared with the GPU's keys in full) and replays every instance, one
host thread per instance.  Traces are generated one seed at a time and their
token arrays dropped once keyed, so host memory holds only keys and request
descriptors; the oracle works on the seeds already keyed while the next seed
is generated.  Every instance is also checked against invariants that hold
at any size."""
import dataclasses
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_same
from paper_2608_01657_amd import device as dv
from paper_2608_01657_amd import tracegen as tg

pytestmark = pytest.mark.gpu

WORKERS = min(16, os.cpu_count() or 1)


def _log(msg):
    print(f"[fullsize {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


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


@dataclasses.dataclass
class _Requests:
    """A trace without its tokens: what the replay (both sides) reads."""
    name: str
    group: np.ndarray
    contract: np.ndarray
    prefix: np.ndarray
    n_groups: int
    n_prefix: int
    tick: object
    n_req: int


def _full_workload(name, n_seeds, policies=tg.ALL_POLICIES, as_set=False):
    """Every seed of workload `name`: keys on both sides (compared in full),
    all instances replayed in one GPU launch and every one compared with the
    oracle.  as_set: the traces are keyed together in one call, as bench.py
    does (host memory then holds every trace's tokens until then).  Returns
    the number of instances compared."""
    t0 = time.time()
    pool = ThreadPoolExecutor(WORKERS)
    dts, reqs, insts, key_futs, orc_futs, kept = [], [], [], [], [], []

    def oracle_replay(k, spec):
        okeys, ooff = key_futs[spec.trace].result()
        return k, oracle.replay_trace(reqs[spec.trace], okeys, ooff, spec)

    try:
        for i in range(n_seeds):
            trs, its = tg.workload(name, seeds=[i], policies=policies)
            tr = trs[0]
            ti = len(reqs)
            key_futs.append(pool.submit(oracle.hash_trace, tr))
            if as_set:
                kept.append(tr)
            else:
                t = dv.upload(tr)
                dv.cut_and_hash(t)
                t.tokens = t.tokens[:0]      # keys are made: the replay never reads tokens
                dts.append(t)
            reqs.append(_Requests(tr.name, tr.group, tr.contract, tr.prefix, tr.n_groups, tr.n_prefix, tr.tick,
                                  tr.n_req))
            del tr, trs
            for spec in its:
                k = len(insts)
                insts.append(dataclasses.replace(spec, trace=ti))
                orc_futs.append(pool.submit(oracle_replay, k, insts[k]))
            if i % 8 == 7 or i == n_seeds - 1:
                _log(f"{name}: {i + 1}/{n_seeds} seeds generated and keyed ({time.time() - t0:.0f}s)")
        if as_set:
            ts = dv.TraceSet(kept).hash()
            kept.clear()
            torch.cuda.synchronize()
            assert int(ts.dt.status.item()) == 0, f"{name}: hash status"
            for i in range(len(reqs)):
                okeys, ooff = key_futs[i].result()
                assert np.array_equal(ts.trace_key_off(i), ooff), f"{name} seed {i}: key offsets differ"
                bad = np.flatnonzero(ts.trace_keys(i) != okeys)
                assert bad.size == 0, f"{name} seed {i}: {bad.size} keys differ, first at {bad[:5]}"
            dts = ts.views
        torch.cuda.synchronize()
        for i, t in enumerate(dts if not as_set else []):
            assert int(t.status.item()) == 0, f"{name} seed {i}: hash status"
            okeys, ooff = key_futs[i].result()
            assert np.array_equal(t.key_off.cpu().numpy(), ooff), f"{name} seed {i}: key offsets differ"
            keys = t.keys[:t.n_keys].cpu().numpy().view(np.uint64)
            bad = np.flatnonzero(keys != okeys)
            assert bad.size == 0, f"{name} seed {i}: {bad.size} keys differ, first at {bad[:5]}"
        b = dv.ReplayBatch(dts, insts)
        b.launch()
        res = b.results()
        _log(f"{name}: {len(insts)} instances replayed on the GPU ({time.time() - t0:.0f}s)")
        for n_done, f in enumerate(orc_futs):
            k, o = f.result()
            spec = insts[k]
            assert_same(res[k], o, f"{name} instance {k} ({spec.label}, seed {spec.trace})")
            _invariants(res[k][0], res[k][1], spec, reqs[spec.trace].n_req)
            if n_done % 256 == 255:
                _log(f"{name}: {n_done + 1}/{len(insts)} instances equal to the oracle ({time.time() - t0:.0f}s)")
        _log(f"{name}: all {len(insts)} instances equal to the oracle ({time.time() - t0:.0f}s)")
        return len(insts)
    finally:
        pool.shutdown(wait=True, cancel_futures=True)


@pytest.mark.timeout(900)
def test_onetouch4096_bench_batch_all_instances():
    """Config 2: 16 seeds x 3 policies = 48 concurrent 4096-block instances."""
    assert _full_workload("onetouch4096", 16, as_set=True) == 48


@pytest.mark.timeout(900)
def test_twopass_all_instances():
    """Config 3: 32 seeds x 3 policies = 96 instances of 80,000 requests."""
    assert _full_workload("twopass", 32) == 96


@pytest.mark.timeout(900)
def test_delayed_all_instances():
    """Config 4: 8 seeds x 8 refill rates x 3 policies = 192 instances of
    200,000 requests; the middle rates clear the polluter's debt inside the
    50,000-request gap (Sec. V-D's delayed replay)."""
    assert _full_workload("delayed", 8) == 192


@pytest.mark.timeout(900)
def test_chat_all_instances():
    """Config 5: 64 seeds x 5 capacities (1K-16K blocks; 8K and 16K keep
    their state in the workspace) x 3 policies = 960 instances of 100,000
    requests."""
    assert _full_workload("chat", 64) == 960


@pytest.mark.timeout(900)
def test_scale1024_all_instances():
    """1,024 concurrent 4096-block instances (16 traces x LRU, S3-FIFO and
    PrefixShield at 62 refill rates), keyed and replayed as bench.py times
    them."""
    assert _full_workload("scale1024", 16, as_set=True) == 1024


def test_chat_staticquota_full_length():
    """StaticQuota on the conversational traces: 16 partitions, so at 1,024
    blocks a 64-block partition truncates most long prompts; every capacity."""
    traces, insts = tg.workload("chat", seeds=[0, 1], policies=(tg.POLICY_STATICQUOTA,))
    assert all(t.n_req == 100000 for t in traces) and len(insts) == 10
    dts, okeys = _hash_all(traces)
    _replay_and_compare(traces, insts, dts, okeys, range(len(insts)))


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
