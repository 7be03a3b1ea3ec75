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
