"""Helpers shared by the GPU tests: run the HIP path and the oracle on the
same seeded inputs and compare."""
import numpy as np

import oracle
from paper_2608_01657_amd import device as dv
from paper_2608_01657_amd import tracegen as tg


def gpu_hash(trace):
    t = dv.upload(trace)
    dv.cut_and_hash(t)
    assert int(t.status.item()) == 0
    keys = t.keys[:t.n_keys].cpu().numpy().view(np.uint64)
    return t, keys, t.key_off.cpu().numpy()


def replay_gpu(dtraces, instances, per_request=False):
    b = dv.ReplayBatch(dtraces, instances, per_request=per_request)
    b.launch()
    res = b.results()
    pr = b.per_request_arrays() if per_request else None
    return res, pr


def assert_same(gpu_res, orc_res, label=""):
    groups, inst, status = gpu_res
    assert status == 0, f"{label}: GPU status {status}"
    for g, (a, b) in enumerate(zip(groups, orc_res.groups)):
        assert a == b, f"{label} group {g}: gpu {a} != oracle {b}"
    assert inst == orc_res.inst, f"{label}: gpu {inst} != oracle {orc_res.inst}"


# Instances that fill the batch beyond what the GPU's CUs hold at once, so
# that the planner lays every instance out for the most instances per CU
# (the hybrid layout for large capacities) as in a large batch; they replay
# an empty trace.
N_DENSE_PAD = 600


def _pad_trace():
    return tg.KeyTrace(np.zeros(0, np.uint64), np.zeros(1, np.int64), np.zeros(0, np.uint8), np.zeros(0, np.uint8),
                       np.zeros(0, np.uint32), 1, 1)


def run_key_traces(kts, instances_per_trace, per_request=True, dense=False):
    """Replay key traces on both sides; every instance compared in full.
    dense: in a batch padded beyond the GPU's CUs (see N_DENSE_PAD)."""
    kts = list(kts)
    instances_per_trace = list(instances_per_trace)
    n_real = sum(len(x) for x in instances_per_trace)
    if dense:
        kts.append(_pad_trace())
        instances_per_trace.append([tg.Instance(0, tg.POLICY_PREFIXSHIELD, 4096) for _ in range(N_DENSE_PAD)])
    dts = [dv.upload_keys(kt) for kt in kts]
    insts = []
    for ti, lst in enumerate(instances_per_trace):
        for inst in lst:
            inst.trace = ti
            insts.append(inst)
    res, pr = replay_gpu(dts, insts, per_request=per_request)
    res, insts = res[:n_real], insts[:n_real]
    for k, inst in enumerate(insts):
        kt = kts[inst.trace]
        o = oracle.replay_key_trace(kt, inst, per_request=per_request)
        assert_same(res[k], o, f"instance {k} ({tg.POLICY_NAMES[inst.policy]}, C={inst.capacity}, flags={inst.flags})")
        if per_request:
            assert np.array_equal(pr[k], o.per_request), f"instance {k}: per-request outputs differ"
    return res


POLICIES = [tg.POLICY_LRU, tg.POLICY_S3FIFO, tg.POLICY_PREFIXSHIELD, tg.POLICY_STATICQUOTA]


def random_key_batch(chunk):
    """25 crafted key traces (seeds 25*chunk ...) with frequent hits, orphans,
    duplicates and truncation, each replayed by every policy and flag with
    1-3 contracts, ticks, eps and S3-FIFO parameters drawn per instance.
    Returns (key traces, instances per trace)."""
    kts, per = [], []
    for seed in range(chunk * 25, chunk * 25 + 25):
        rng = np.random.default_rng(seed)
        nc = int(rng.integers(1, 4))
        kt = tg.random_key_trace(seed, n_req=int(rng.integers(1, 120)), max_blocks=int(rng.integers(1, 80)),
                                 n_groups=int(rng.integers(1, 6)), n_prefix=12, n_contracts=nc,
                                 key_universe=int(rng.integers(4, 200)), with_ticks=bool(seed % 2))
        insts = []
        for pol in POLICIES:
            for flags in ([0, 1, 2, 3] if pol == tg.POLICY_PREFIXSHIELD else [0]):
                cap = int(rng.integers(1, 90))
                contracts = [(int(rng.integers(3, 3 * tg.Q16)), int(rng.integers(0, 40)) * tg.Q16)
                             for _ in range(nc)]
                # S3-FIFO also with a one-block small queue (0), no ghost
                # (1000), every head moving (threshold 0) and none (4)
                insts.append(tg.Instance(0, pol, cap, contracts=contracts, flags=flags,
                                         eps_q16=int(rng.choice([0, tg.Q16 // 2, 3 * tg.Q16])),
                                         s3_small_permille=int(rng.choice([0, 1, 100, 250, 500, 1000])),
                                         s3_move_threshold=int(rng.choice([0, 1, 2, 4]))))
        kts.append(kt)
        per.append(insts)
    return kts, per


def step_boundary_batch():
    """6 key traces of 40 requests of 255-257 and 511-513 blocks (both sides
    of the 256-position lookup step) with shared prefixes, duplicates within
    a request and keys reused across requests; every policy and PrefixShield
    flag at capacities 200, 256, 300 and 700.  Returns (key traces,
    instances per trace)."""
    kts, per = [], []
    for seed in range(6):
        rng = np.random.default_rng(9000 + seed)
        G = 3
        reqs, groups = [], []
        hist = []
        for r in range(40):
            n = int(rng.choice([255, 256, 257, 511, 512, 513]))
            if hist and rng.random() < 0.6:
                src = hist[int(rng.integers(0, len(hist)))]
                ks = list(src[:int(rng.integers(0, len(src) + 1))])
            else:
                ks = []
            while len(ks) < n:
                ks.append(int(rng.integers(1, 1500)))    # small universe: reuse and duplicates
            ks = ks[:n]
            hist.append(ks)
            reqs.append(ks)
            groups.append(int(rng.integers(0, G)))
        keys = np.array([k for r in reqs for k in r], dtype=np.uint64)
        off = np.concatenate([[0], np.cumsum([len(r) for r in reqs])]).astype(np.int64)
        R = len(reqs)
        kts.append(tg.KeyTrace(keys, off, np.array(groups, np.uint8), (np.arange(R) % 2).astype(np.uint8),
                               (np.array(groups) * 3 + np.arange(R) % 3).astype(np.uint32), G, 3 * G))
        contracts = [(tg.Q16, 64 * tg.Q16), (tg.Q16 // 4, 16 * tg.Q16)]
        insts = []
        for pol in POLICIES:
            for cap in (200, 256, 300, 700):
                for flags in ([0, 1, 2] if pol == tg.POLICY_PREFIXSHIELD else [0]):
                    insts.append(tg.Instance(0, pol, cap, contracts=contracts, flags=flags))
        per.append(insts)
    return kts, per


def many_groups_batch():
    """6 key traces with 64 accounting groups and 4 contracts of different
    refill rates (normalized debt, Eq. 5; ties in projected debt), every
    policy and PrefixShield flag.  Returns (key traces, instances per
    trace)."""
    kts, per = [], []
    for seed in range(6):
        rng = np.random.default_rng(1000 + seed)
        kt = tg.random_key_trace(1000 + seed, n_req=300, max_blocks=12, n_groups=64, n_prefix=128,
                                 n_contracts=4, key_universe=60)
        insts = []
        for pol in POLICIES:
            for flags in ([0, 1, 2] if pol == tg.POLICY_PREFIXSHIELD else [0]):
                contracts = [(tg.Q16 // (c + 1), int(rng.integers(0, 4)) * tg.Q16) for c in range(4)]
                insts.append(tg.Instance(0, pol, int(rng.integers(8, 200)), contracts=contracts, flags=flags))
        kts.append(kt)
        per.append(insts)
    return kts, per


def workload_parity(name, seeds, n_requests, per_request=False, **kw):
    """Keys and replay of a named workload on both sides, every key and every
    instance compared.  Returns the number of instances."""
    traces, insts = tg.workload(name, seeds=seeds, n_requests=n_requests, **kw)
    dts, okeys = [], []
    for tr in traces:
        t, keys, off = gpu_hash(tr)
        ok_, ooff = oracle.hash_trace(tr)
        assert np.array_equal(keys, ok_) and np.array_equal(off, ooff)
        dts.append(t)
        okeys.append((ok_, ooff))
    res, pr = replay_gpu(dts, insts, per_request=per_request)
    for k, inst in enumerate(insts):
        o = oracle.replay_trace(traces[inst.trace], okeys[inst.trace][0], okeys[inst.trace][1], inst,
                                per_request=per_request)
        assert_same(res[k], o, f"{name} instance {k} {inst.label}")
        if per_request:
            assert np.array_equal(pr[k], o.per_request), f"{name} instance {k}: per-request outputs differ"
    return len(insts)
