"""pc_replay_batch_static (the entry point that allocates nothing: its
workspace is the library's static device array) against pc_replay_batch on
the same batch, every stats record and per-request quadruple bit for bit,
on two calls in a row, the second with a smaller batch (the array keeps the
first call's contents, which the second must not see)."""
import numpy as np
import pytest
import torch

import paper_2608_01657_amd as P
from paper_2608_01657_amd import device as dv
from paper_2608_01657_amd import tracegen as tg

pytestmark = pytest.mark.gpu


def _batch(n_req, caps, seed):
    kts = [tg.random_key_trace(seed + i, n_req=n_req, max_blocks=600, n_groups=5, n_prefix=40, n_contracts=2,
                               key_universe=3000, with_ticks=bool(i % 2)) for i in range(2)]
    dts = [dv.upload_keys(kt) for kt in kts]
    insts = []
    for ti in range(len(kts)):
        for pol in (tg.POLICY_LRU, tg.POLICY_S3FIFO, tg.POLICY_PREFIXSHIELD, tg.POLICY_STATICQUOTA):
            for cap in caps:
                insts.append(tg.Instance(ti, pol, cap, contracts=[(tg.Q16 // 3, 8 * tg.Q16), (tg.Q16, 0)]))
    return dts, insts


def _run_both(dts, insts):
    b = dv.ReplayBatch(dts, insts, per_request=True)
    b.launch()
    ref = b.results()
    ref_pr = b.per_request.cpu().numpy()
    n = len(insts)
    stats = torch.full((n * P.PC_STATS_RECORD_BYTES // 8,), -7, dtype=torch.int64, device=dts[0].keys.device)
    pr = torch.full_like(b.per_request, -7)
    P.pc_replay_batch_static(b.tdesc, b.idesc, stats, pr)
    G, S = P.pc_get_stats(stats, n, -1, 64)
    got = P.stats_to_dicts(G, S, [dts[i.trace].n_groups for i in insts])
    return ref, ref_pr, got, pr.cpu().numpy()


def test_static_workspace_matches_pc_replay_batch_twice():
    torch.cuda.set_device(0)
    # first call: LDS and workspace layouts (C = 9000 keeps its state in the
    # array), S3-FIFO ghost rings, prefix bitmaps
    dts, insts = _batch(400, (64, 700, 9000), 31)
    ws = P.pc_replay_workspace_bytes([dv.trace_desc(t) for t in dts], [P.make_instance_desc(i) for i in insts])
    assert ws <= P.PC_STATIC_WORKSPACE_BYTES
    ref, ref_pr, got, pr = _run_both(dts, insts)
    assert all(st == 0 for _, _, st in ref)
    assert got == ref
    assert np.array_equal(pr, ref_pr)
    # second call, smaller: fewer requests, instances and capacities
    dts2, insts2 = _batch(150, (40, 300), 77)
    ref2, ref_pr2, got2, pr2 = _run_both(dts2, insts2)
    assert all(st == 0 for _, _, st in ref2)
    assert got2 == ref2
    assert np.array_equal(pr2, ref_pr2)
