"""Child process of test_gpu_race.py (run as a script, not collected): it
selects the race-detection build of the library, in which every replay
barrier is followed by a pseudo-random per-wavefront delay, and replays
batches that exercise every policy, flag and state layout, each compared
with the oracle in full.  A result that depends on the order in which the
wavefronts of a workgroup reach shared state differs here.

    python tests/jitter_child.py <repo root>
"""
import json
import sys
import time

root = sys.argv[1]
sys.path.insert(0, root)
sys.path.insert(0, root + "/tests")

import paper_2608_01657_amd as P  # noqa: E402

P.use_jitter_build()

import oracle  # noqa: E402
from gpu_util import (assert_same, gpu_hash, many_groups_batch, random_key_batch, replay_gpu,  # noqa: E402
                      run_key_traces, step_boundary_batch, workload_parity)
from paper_2608_01657_amd import tracegen as tg  # noqa: E402


def log(msg):
    print(msg, file=sys.stderr, flush=True)


t0 = time.time()
done = {}
log("step boundary, launch 1 starting")
# lookup-step boundaries at small capacities (the free-queue log fills and
# is compacted often), replayed three times: each launch draws other delays
for rep in range(3):
    n = len(run_key_traces(*step_boundary_batch()))
    done["step_boundary"] = done.get("step_boundary", 0) + n
    log(f"step boundary, launch {rep + 1}: {n} instances ({time.time() - t0:.0f}s)")
# the same in a batch wide enough for the hybrid layout
n = len(run_key_traces(*step_boundary_batch(), dense=True))
done["step_boundary_dense"] = n
log(f"step boundary, dense batch: {n} instances ({time.time() - t0:.0f}s)")
for chunk in range(4):
    n = len(run_key_traces(*random_key_batch(chunk)))
    done["random"] = done.get("random", 0) + n
log(f"random key traces: {done['random']} instances ({time.time() - t0:.0f}s)")
# 64 groups on 4 contracts: ties in projected debt, many queues
log("many groups starting")
done["many_groups"] = len(run_key_traces(*many_groups_batch()))
# contention from 8 / 32 indebted groups on every request, the attack
# traces with every PrefixShield variant and StaticQuota, three contract tiers
for name, n_req in (("selector512x8", None), ("selector4096x32", None), ("attack_onetouch", None),
                    ("attack_lowslow", None), ("attack_replay", None), ("tiers", 20000)):
    log(f"{name} starting")
    done[name] = workload_parity(name, [0], n_req, per_request=True)
    log(f"{name}: {done[name]} instances ({time.time() - t0:.0f}s)")
# conversational trace at full length, every capacity (all-LDS, hybrid or
# workspace state) and policy
log("chat seed 0 starting")
traces, insts = tg.workload("chat", seeds=[0])
t, keys, off = gpu_hash(traces[0])
okeys, ooff = oracle.hash_trace(traces[0])
assert (keys == okeys).all() and (off == ooff).all()
res, _ = replay_gpu([t], insts)
for k, spec in enumerate(insts):
    o = oracle.replay_trace(traces[0], okeys, ooff, spec)
    assert_same(res[k], o, f"chat {spec.label}")
done["chat_full_length"] = len(insts)
log(f"chat seed 0: {len(insts)} instances ({time.time() - t0:.0f}s)")
print(json.dumps(done))
