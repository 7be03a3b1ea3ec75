"""The C oracle (indexed per-group/per-segment queues) against the scan-based
Python brute force on random tiny traces: every counter must be equal.

This pins the oracle's queue/index logic (Alg. 2's FirstSegmentQueue and
GlobalFirstSegmentQueue, the LRU free-queue order, S3-FIFO's queues and
ghost) against a selector that simply scans every candidate, as the paper's
prototype does (Sec. IV)."""
import itertools

import numpy as np
import pytest

import oracle
from brute_force import brute_replay
from paper_2608_01657_amd import tracegen as tg

POLICIES = [tg.POLICY_LRU, tg.POLICY_S3FIFO, tg.POLICY_PREFIXSHIELD, tg.POLICY_STATICQUOTA]


def _compare(kt, inst):
    res = oracle.replay_key_trace(kt, inst, per_request=True)
    bst, bis, bpr = brute_replay(kt.keys, kt.key_off, kt.group, kt.contract, kt.prefix,
                                 kt.n_groups, inst, tick=kt.tick)
    for g in range(kt.n_groups):
        assert res.groups[g] == bst[g], (g, res.groups[g], bst[g])
    assert res.inst == bis
    assert [tuple(x) for x in res.per_request.tolist()] == [tuple(x) for x in bpr]


def _instances(rng, n_contracts):
    out = []
    for pol in POLICIES:
        for flags in ([0, 1, 2, 3] if pol == tg.POLICY_PREFIXSHIELD else [0]):
            cap = int(rng.integers(1, 13))
            contracts = []
            for _ in range(n_contracts):
                rho = int(rng.integers(1, 3 * tg.Q16))
                beta = int(rng.integers(0, 6)) * tg.Q16 + int(rng.integers(0, 2)) * int(rng.integers(0, tg.Q16))
                contracts.append((rho, beta))
            eps = int(rng.choice([0, 0, tg.Q16 // 2, 2 * tg.Q16]))
            # S3-FIFO: a small queue of one block (0), no ghost at all (1000),
            # every head moving (threshold 0) and none ever moving (4 > the
            # frequency cap of 3)
            out.append(tg.Instance(0, pol, cap, contracts=contracts, flags=flags, eps_q16=eps,
                                   s3_small_permille=int(rng.choice([0, 1, 100, 250, 500, 1000])),
                                   s3_move_threshold=int(rng.choice([0, 1, 2, 4]))))
    return out


@pytest.mark.parametrize("seed", range(60))
def test_random_tiny_traces(seed):
    rng = np.random.default_rng(seed)
    n_contracts = int(rng.integers(1, 4))
    kt = tg.random_key_trace(seed, n_req=int(rng.integers(1, 45)), max_blocks=int(rng.integers(1, 9)),
                             n_groups=int(rng.integers(1, 5)), n_prefix=8, n_contracts=n_contracts,
                             key_universe=int(rng.integers(4, 30)), with_ticks=bool(seed % 2))
    for inst in _instances(rng, n_contracts):
        _compare(kt, inst)


@pytest.mark.parametrize("cap,pol", itertools.product([16, 64, 200], POLICIES))
def test_tiny_workload_prefix_short(cap, pol):
    """Token-derived keys from the one-touch recipe (first 120 requests)."""
    tr = tg.onetouch_tiny(1000, 120)
    keys, off = oracle.hash_trace(tr)
    kt = tg.KeyTrace(keys, off, tr.group, tr.contract, tr.prefix, tr.n_groups, tr.n_prefix)
    for flags in ([0, 1, 2] if pol == tg.POLICY_PREFIXSHIELD else [0]):
        inst = tg.Instance(0, pol, cap, contracts=[(tg.Q16 // 2, 8 * tg.Q16)], flags=flags)
        _compare(kt, inst)


@pytest.mark.parametrize("seed", range(8))
def test_rate_ratio_at_the_q16_limit(seed):
    """Two contracts whose refill rates differ by exactly 2^16 (1/w of the
    fast one is 2^-16 in Q16, the smallest positive decrement of Eq. 8),
    both indebted by groups that share them, equal ticks so that no debt is
    refilled: the oracle agrees with the brute force on every counter and
    every request; one more unit of ratio is rejected by both."""
    rng = np.random.default_rng(900 + seed)
    kt = tg.random_key_trace(900 + seed, n_req=40, max_blocks=8, n_groups=3, n_prefix=6, n_contracts=2,
                             key_universe=30)
    kt.tick = np.zeros(kt.n_req, np.int64)
    slow = int(rng.choice([1, 5, 1 << 20]))
    for pol in POLICIES:
        inst = tg.Instance(0, pol, int(rng.integers(4, 14)), contracts=[(slow, 0), (slow << 16, 0)])
        _compare(kt, inst)
    bad = tg.Instance(0, tg.POLICY_PREFIXSHIELD, 8, contracts=[(slow, 0), ((slow << 16) + 1, 0)])
    with pytest.raises(ValueError):
        oracle.replay_key_trace(kt, bad)
    with pytest.raises(ValueError):
        brute_replay(kt.keys, kt.key_off, kt.group, kt.contract, kt.prefix, kt.n_groups, bad, tick=kt.tick)
