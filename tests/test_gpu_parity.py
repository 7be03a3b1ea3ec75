"""GPU parity: the HIP path (through the C ABI) against the oracle, bit-exact.

Keys: every key of every request.  Replay: every per-group and per-instance
counter, and the per-request (hits, new, evictions, orphans) quadruples.
Inputs are seeded synthetic traces (tracegen) or crafted key arrays."""
import numpy as np
import pytest

import oracle
from gpu_util import POLICIES, assert_same, gpu_hash, many_groups_batch, random_key_batch, replay_gpu, \
    run_key_traces, step_boundary_batch, workload_parity
from paper_2608_01657_amd import device as dv
from paper_2608_01657_amd import tracegen as tg

pytestmark = pytest.mark.gpu


def _edge_trace(seed=9):
    """Lengths around block boundaries, unaligned views, full int32 ids."""
    rng = np.random.default_rng(seed)
    lens = [0, 1, 15, 16, 17, 31, 32, 33, 63, 64, 65, 1023, 1024, 1025, 4096 + 7, 16384, 16384 + 15]
    lens += [int(x) for x in rng.integers(0, 3000, 60)]
    total = sum(lens) + 64
    toks = rng.integers(-2**31, 2**31, total, dtype=np.int64).astype(np.int32)
    offs, pos = [], 0
    for i, L in enumerate(lens):
        pos += i % 4          # every alignment of the view start
        offs.append(pos)
        pos += L
    toks = np.concatenate([toks, rng.integers(0, 32000, pos + 16, dtype=np.int64).astype(np.int32)])[:pos + 16]
    R = len(lens)
    return tg.Trace("edge", toks, np.array(offs, np.int64), np.array(lens, np.int32),
                    (np.arange(R) % 7).astype(np.uint8), np.zeros(R, np.uint8), np.arange(R, dtype=np.uint32),
                    7, R)


def _check_hash(trace):
    _, keys, off = gpu_hash(trace)
    okeys, ooff = oracle.hash_trace(trace)
    assert np.array_equal(off, ooff)
    assert keys.shape == okeys.shape
    bad = np.nonzero(keys != okeys)[0]
    assert bad.size == 0, f"{bad.size} keys differ, first at {bad[:5]}"


def test_hash_edge_cases():
    _check_hash(_edge_trace())


def test_hash_tail_of_buffer():
    """The last request ends exactly at the end of the token buffer."""
    rng = np.random.default_rng(3)
    for extra in range(4):
        L = 16 * 37 + extra
        toks = rng.integers(0, 32000, L + 3).astype(np.int32)
        tr = tg.Trace("tail", toks, np.array([3], np.int64), np.array([L], np.int32), np.zeros(1, np.uint8),
                      np.zeros(1, np.uint8), np.zeros(1, np.uint32), 1, 1)
        _check_hash(tr)


@pytest.mark.parametrize("name", ["tiny", "onetouch4096", "twopass", "chat"])
def test_hash_workloads(name):
    n = {"tiny": 4000, "onetouch4096": 3000, "twopass": 3000, "chat": 5000}[name]
    traces, _ = tg.workload(name, seeds=[0], n_requests=n)
    _check_hash(traces[0])


@pytest.mark.parametrize("chunk", range(4))
def test_replay_random_key_traces(chunk):
    """Crafted keys with frequent hits, orphans, duplicates and truncation;
    every policy and flag, 1-3 contracts, ticks, eps, S3 parameters."""
    run_key_traces(*random_key_batch(chunk))


def test_replay_many_groups():
    """64 accounting groups, several contracts with different refill rates
    (normalized debt, Eq. 5), ties in projected debt."""
    run_key_traces(*many_groups_batch())


def _workload_parity(name, seeds, n_requests, per_request=False, policies=tuple(POLICIES), **kw):
    return workload_parity(name, seeds, n_requests, per_request=per_request, policies=policies, **kw)


def test_replay_tiny_workload_full():
    _workload_parity("tiny", [0], None, per_request=True)


def test_replay_tiny_workload_variants():
    tr = tg.onetouch_tiny(1000, 4000)
    keys, off = oracle.hash_trace(tr)
    kt = tg.KeyTrace(keys, off, tr.group, tr.contract, tr.prefix, tr.n_groups, tr.n_prefix)
    per = [[tg.Instance(0, pol, cap, contracts=[(rho, 64 * tg.Q16)], flags=fl)
            for pol in POLICIES for cap in (16, 100, 256, 1000)
            for fl in ([0, 1, 2] if pol == tg.POLICY_PREFIXSHIELD else [0])
            for rho in (tg.Q16 // 8, 8 * tg.Q16)]]
    run_key_traces([kt], per)


def test_replay_onetouch4096_short():
    _workload_parity("onetouch4096", [0, 1], 4000, per_request=True)


def test_replay_twopass_short():
    _workload_parity("twopass", [0], 6000)


def test_replay_delayed_short():
    _workload_parity("delayed", [0], 8000)


def test_replay_chat_all_capacities():
    """Includes capacities whose state does not fit in LDS (workspace path)."""
    _workload_parity("chat", [0], 4000, per_request=True)


def test_replay_normalized_debt_tiers():
    """The Eq. 5 / Eq. 8 pins of the oracle (fast vs slow contract at equal
    raw debt, before and past the crossover) on the GPU."""
    from test_oracle_replay_pins import _tier_trace
    Q = tg.Q16
    kts, per = [], []
    for m, e in [(40, 20), (40, 36), (64, 47), (64, 60)]:
        kts.append(_tier_trace(m, e))
        per.append([tg.Instance(0, pol, 2 * m, contracts=[(4 * Q, 0), (Q, 0), (Q, 1 << 40)], flags=fl)
                    for pol in POLICIES for fl in ([0, 1, 2] if pol == tg.POLICY_PREFIXSHIELD else [0])])
    run_key_traces(kts, per)


@pytest.mark.parametrize("n", [0, 1, 1023, 1024, 1025, 50_000, 256 * 1024, 256 * 1024 + 1, (1 << 21) + 4097])
def test_block_offsets_sizes(n):
    """CSR block offsets at sizes around the chunking (1024 requests per
    chunk; the chunk-sum scan loops past 256 chunks), including negative
    lengths, which count as no blocks."""
    import torch
    rng = np.random.default_rng(n)
    lens = rng.integers(-20, 40000, n).astype(np.int32)
    d_len = torch.from_numpy(lens).to("cuda")
    d_off = torch.full((n + 1,), -7, dtype=torch.int64, device="cuda")
    dv.pc_block_offsets(d_len, d_off)
    torch.cuda.synchronize()
    assert np.array_equal(d_off.cpu().numpy(), oracle.block_offsets(lens))


def test_replay_last_request_displacements():
    """Table entries that find both buckets full are placed by the next
    request, or after the last one.  Traces whose final requests insert a
    full cache of fresh keys at the table's design load (C = 85: 16 buckets of
    8, load 2/3) leave such entries behind; every policy must still match the
    oracle with status 0."""
    kts, per = [], []
    for seed in range(16):
        rng = np.random.default_rng(500 + seed)
        C = 85
        reqs = [list(rng.integers(1, 2**63, C, dtype=np.int64)) for _ in range(4)]
        keys = np.array([k for r in reqs for k in r], dtype=np.int64).view(np.uint64)
        off = np.arange(0, C * len(reqs) + 1, C, dtype=np.int64)
        R = len(reqs)
        kts.append(tg.KeyTrace(keys, off, np.zeros(R, np.uint8), np.zeros(R, np.uint8),
                               np.arange(R, dtype=np.uint32), 1, R))
        per.append([tg.Instance(0, pol, C) for pol in POLICIES])
    run_key_traces(kts, per)


def _append_requests(kt, reqs, group=0):
    """KeyTrace `kt` followed by the requests `reqs` (lists of keys)."""
    keys = np.concatenate([kt.keys] + [np.asarray(r, np.uint64) for r in reqs])
    off = np.concatenate([kt.key_off, kt.key_off[-1] + np.cumsum([len(r) for r in reqs])]).astype(np.int64)
    R = len(reqs)
    return tg.KeyTrace(keys, off, np.concatenate([kt.group, np.full(R, group, np.uint8)]),
                       np.concatenate([kt.contract, np.zeros(R, np.uint8)]),
                       np.concatenate([kt.prefix, np.zeros(R, np.uint32)]), kt.n_groups, kt.n_prefix)


def test_replay_max_capacity():
    """C = PC_MAX_CAPACITY: the state lives in the workspace, the main table
    has 2^16 entries (every bit of the entry index kept in a slot's metadata
    word is used), the S3 ghost ring is at its 2^16 cap, and two final
    requests are longer than the cache (33,000 fresh keys, then the same
    keys again), so admission truncates."""
    from paper_2608_01657_amd import PC_MAX_CAPACITY
    C = PC_MAX_CAPACITY
    rng = np.random.default_rng(4242)
    kt = tg.random_key_trace(77, n_req=200, max_blocks=1500, n_groups=4, n_prefix=16, n_contracts=2,
                             key_universe=60000)
    long_req = list(rng.integers(1 << 40, 1 << 62, 33000, dtype=np.int64))
    kt = _append_requests(kt, [long_req, long_req], group=1)
    contracts = [(tg.Q16, 4 * tg.Q16), (tg.Q16 // 2, 0)]
    insts = [tg.Instance(0, tg.POLICY_LRU, C, contracts=contracts),
             tg.Instance(0, tg.POLICY_STATICQUOTA, C, contracts=contracts),
             tg.Instance(0, tg.POLICY_S3FIFO, C, contracts=contracts, s3_small_permille=100),
             tg.Instance(0, tg.POLICY_S3FIFO, C, contracts=contracts, s3_small_permille=500, s3_move_threshold=2)]
    insts += [tg.Instance(0, tg.POLICY_PREFIXSHIELD, C, contracts=contracts, flags=f, eps_q16=tg.Q16 // 2)
              for f in [0, 1, 2, 3]]
    res = run_key_traces([kt], [insts])
    for (groups, inst, _), spec in zip(res, insts):
        assert sum(g["truncated"] for g in groups) > 0, tg.POLICY_NAMES[spec.policy]
        assert inst["resident_max"] <= C


def test_replay_empty_and_blockless_traces():
    """A trace with no requests, and one whose requests hold no full block
    (zero keys each): every counter except the request counts stays zero,
    on both sides, for every policy."""
    empty = tg.KeyTrace(np.zeros(0, np.uint64), np.zeros(1, np.int64), np.zeros(0, np.uint8),
                        np.zeros(0, np.uint8), np.zeros(0, np.uint32), 1, 1)
    R = 9
    blockless = tg.KeyTrace(np.zeros(0, np.uint64), np.zeros(R + 1, np.int64), (np.arange(R) % 3).astype(np.uint8),
                            np.zeros(R, np.uint8), np.arange(R, dtype=np.uint32), 3, R)
    per = [[tg.Instance(0, pol, cap) for pol in POLICIES for cap in (1, 100)] for _ in range(2)]
    res = run_key_traces([empty, blockless], per)
    for groups, inst, _ in res:
        assert all(v == 0 for v in inst.values())
        assert all(v == 0 for g in groups for k, v in g.items() if k != "requests")


def test_hash_out_of_range_requests_are_skipped():
    """A request whose token range leaves the token buffer, whose length or
    offset is negative, or whose keys would pass n_keys, sets the status to
    PC_EINVAL and writes nothing; every other request still gets its keys."""
    import torch
    import paper_2608_01657_amd as P
    rng = np.random.default_rng(21)
    R = 40
    lens = rng.integers(0, 3000, R).astype(np.int32)
    toks = rng.integers(0, 32000, int(lens.sum()) + 64, dtype=np.int64).astype(np.int32)
    offs = np.concatenate([[0], np.cumsum(lens[:-1])]).astype(np.int64)
    lens[-1] = max(int(lens[-1]), 64)              # the last request has keys
    bad = {5: "tokens", 17: "length", 30: "offset", R - 1: "keys"}
    offs[5] = len(toks) - 10                       # runs past the token buffer
    lens[5] = 100
    lens[17] = -5
    offs[30] = -3
    key_off = oracle.block_offsets(lens)
    n_keys = int(key_off[-1]) - 1                  # the last request's keys do not fit
    ns = (np.arange(R) % 5).astype(np.int32)
    dev = torch.device("cuda")
    sentinel = 0x5A5A5A5A5A5A5A5A
    d_keys = torch.full((n_keys,), sentinel, dtype=torch.int64, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    P.pc_hash_blocks(torch.from_numpy(toks).to(dev), torch.from_numpy(offs).to(dev),
                     torch.from_numpy(lens).to(dev), torch.from_numpy(ns).to(dev),
                     torch.from_numpy(key_off).to(dev), d_keys, status, None)
    assert int(status.item()) == P.PC_EINVAL
    keys = d_keys.cpu().numpy()
    for r in range(R):
        a, b = int(key_off[r]), min(int(key_off[r + 1]), n_keys)
        if r in bad:
            assert np.all(keys[a:b] == sentinel), f"request {r} ({bad[r]}) wrote keys"
            continue
        want = oracle.hash_request(toks[offs[r]:offs[r] + lens[r]], int(ns[r])).view(np.int64)
        assert np.array_equal(keys[a:b], want), f"request {r}"


def _many_request_trace(n_req, seed, shared):
    """n_req requests: mostly blockless or one- and two-block requests, some
    of hundreds of tokens, a few of thousands, and a stretch of 300
    consecutive blockless requests.  shared: the requests read overlapping
    windows of one 2 M-token buffer at any int32 offset (token reuse: the
    4-wave key kernel); else each request has its own tokens, laid out back
    to back with gaps of 0-3 tokens (streaming: the 16-wave key kernel)."""
    rng = np.random.default_rng(seed)
    u = rng.random(n_req)
    lens = np.where(u < 0.90, rng.integers(0, 48, n_req),
                    np.where(u < 0.999, rng.integers(48, 400, n_req), rng.integers(400, 5000, n_req)))
    a = n_req // 3
    lens[a:a + 300] = rng.integers(0, 16, 300)
    lens = lens.astype(np.int32)
    if shared:
        n_tok = 2_000_000
        offs = (rng.random(n_req) * (n_tok - lens)).astype(np.int64)
    else:
        gaps = rng.integers(0, 4, n_req)
        offs = np.cumsum(gaps + lens) - lens
        n_tok = int(offs[-1] + lens[-1])
    toks = rng.integers(-2**31, 2**31, n_tok, dtype=np.int64).astype(np.int32)
    ns = rng.integers(0, 256, n_req).astype(np.uint8)
    blocks = int((lens // 16).sum())
    assert (blocks <= 2 * (n_tok // 16)) != shared, "the trace does not take the intended key kernel"
    return tg.Trace("many", toks, offs.astype(np.int64), lens, ns, np.zeros(n_req, np.uint8),
                    np.zeros(n_req, np.uint32), 256, n_req)


@pytest.mark.parametrize("n_req,shared", [(131_109, True), (1_507_339, False), (4_194_341, True)])
def test_hash_many_requests(n_req, shared):
    """Grids of 8 K to 1 M workgroups, with a ragged last workgroup, on both
    key kernels: every key of every request."""
    _check_hash(_many_request_trace(n_req, seed=n_req % 1000, shared=shared))


@pytest.mark.parametrize("n_req,shared", [(131_077, False), (4_194_309, True)])
def test_hash_bad_requests_among_many(n_req, shared):
    """Requests that fail the bounds check scattered through a large grid:
    the status is PC_EINVAL, they write nothing, and their neighbours in the
    same workgroup still get their keys."""
    import torch
    import paper_2608_01657_amd as P
    tr = _many_request_trace(n_req, seed=200 + n_req % 1000, shared=shared)
    okeys, ooff = oracle.hash_trace(tr)
    offs = tr.tok_off.copy()
    lens = tr.length
    withkeys = np.nonzero(lens >= 16)[0]
    rng = np.random.default_rng(7)
    bad = np.sort(rng.choice(withkeys, 12, replace=False))
    offs[bad[:6]] = -3                                  # negative offset
    offs[bad[6:]] = len(tr.tokens) - 5                  # runs past the token buffer
    dev = torch.device("cuda")
    sentinel = 0x5A5A5A5A5A5A5A5A
    n_keys = int(ooff[-1])
    d_keys = torch.full((n_keys,), sentinel, dtype=torch.int64, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    P.pc_hash_blocks(torch.from_numpy(tr.tokens).to(dev), torch.from_numpy(offs).to(dev),
                     torch.from_numpy(lens).to(dev), torch.from_numpy(tr.group.astype(np.int32)).to(dev),
                     torch.from_numpy(ooff).to(dev), d_keys, status, None)
    assert int(status.item()) == P.PC_EINVAL
    keys = d_keys.cpu().numpy().view(np.uint64)
    want = okeys.copy()
    for r in bad:
        want[ooff[r]:ooff[r + 1]] = np.uint64(sentinel)
    diff = np.nonzero(keys != want)[0]
    assert diff.size == 0, f"{diff.size} keys differ, first at {diff[:5]}"


def test_hash_request_length_limit():
    """A request of 2^30 tokens (4 GiB) or more is skipped with PC_EINVAL;
    one of 2^30 - 1 tokens, the longest allowed, gets all of its 2^26 - 1
    keys, equal to the oracle's."""
    import torch
    import paper_2608_01657_amd as P
    dev = torch.device("cuda")
    n_tok = (1 << 30) + 4096
    g = torch.Generator(device=dev).manual_seed(31)
    d_toks = torch.randint(-2**31, 2**31, (n_tok,), dtype=torch.int32, device=dev, generator=g)
    offs = np.array([0, 7, 123_456], np.int64)
    lens = np.array([1 << 30, (1 << 30) - 1, 5000], np.int32)
    ns = np.array([3, 4, 5], np.int32)
    key_off = oracle.block_offsets(lens)
    n_keys = int(key_off[-1])
    sentinel = 0x5A5A5A5A5A5A5A5A
    d_keys = torch.full((n_keys,), sentinel, dtype=torch.int64, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    P.pc_hash_blocks(d_toks, torch.from_numpy(offs).to(dev), torch.from_numpy(lens).to(dev),
                     torch.from_numpy(ns).to(dev), torch.from_numpy(key_off).to(dev), d_keys, status, None)
    assert int(status.item()) == P.PC_EINVAL
    keys = d_keys.cpu().numpy().view(np.uint64)
    del d_keys
    toks = d_toks.cpu().numpy()
    del d_toks
    assert np.all(keys[key_off[0]:key_off[1]] == np.uint64(sentinel)), "the 2^30-token request wrote keys"
    for r in (1, 2):
        want = oracle.hash_request(toks[offs[r]:offs[r] + lens[r]], int(ns[r]))
        got = keys[key_off[r]:key_off[r + 1]]
        bad = np.flatnonzero(got != want)
        assert bad.size == 0, f"request {r}: {bad.size} keys differ, first at {bad[:5]}"


def _prefix_trace(kt, k):
    """The first k requests of key trace kt."""
    return tg.KeyTrace(kt.keys[:int(kt.key_off[k])], kt.key_off[:k + 1].copy(), kt.group[:k].copy(),
                       kt.contract[:k].copy(), kt.prefix[:k].copy(), kt.n_groups, kt.n_prefix,
                       None if kt.tick is None else kt.tick[:k].copy())


def test_replay_malformed_request_stops_the_instance():
    """A request with a group, contract or prefix id out of range, or a tick
    below the previous one, stops its instance: status PC_EINVAL, every
    counter zero, the quadruples of the requests before it as the oracle
    gives them for that prefix of the trace; an instance of a well-formed
    trace in the same batch is unaffected."""
    import paper_2608_01657_amd as P
    base = tg.random_key_trace(4040, n_req=80, max_blocks=24, n_groups=3, n_prefix=9, n_contracts=2,
                               key_universe=60, with_ticks=True)
    k = 50
    kts, what = [base], ["well-formed"]
    for kind in ["group", "contract", "prefix", "tick"]:
        kt = tg.KeyTrace(base.keys.copy(), base.key_off.copy(), base.group.copy(), base.contract.copy(),
                         base.prefix.copy(), base.n_groups, base.n_prefix, base.tick.copy())
        if kind == "group":
            kt.group[k] = 3
        elif kind == "contract":
            kt.contract[k] = 2
        elif kind == "prefix":
            kt.prefix[k] = base.n_prefix
        else:
            kt.tick[k] = kt.tick[k - 1] - 1
        kts.append(kt)
        what.append(kind)
    contracts = [(tg.Q16, 8 * tg.Q16), (tg.Q16 // 3, 2 * tg.Q16)]
    dts = [dv.upload_keys(kt) for kt in kts]
    insts = [tg.Instance(ti, pol, 40, contracts=contracts) for ti in range(len(kts)) for pol in POLICIES]
    res, pr = replay_gpu(dts, insts, per_request=True)
    for j, inst in enumerate(insts):
        label = f"{what[inst.trace]} trace, {tg.POLICY_NAMES[inst.policy]}"
        groups, istats, status = res[j]
        if inst.trace == 0:
            o = oracle.replay_key_trace(kts[0], inst, per_request=True)
            assert_same(res[j], o, label)
            assert np.array_equal(pr[j], o.per_request), label
            continue
        assert status == P.PC_EINVAL, label
        assert all(v == 0 for v in istats.values()), label
        assert all(v == 0 for g in groups for v in g.values()), label
        o = oracle.replay_key_trace(_prefix_trace(kts[inst.trace], k), inst, per_request=True)
        assert np.array_equal(pr[j][:k], o.per_request), label


def test_hash_token_buffer_at_any_int32_offset():
    """The token buffer itself may start at any int32 (the kernel's token
    loads assume 4-byte alignment only): the same requests hashed from views
    that start 0..3 tokens into an allocation give the oracle's keys."""
    import torch
    import paper_2608_01657_amd as P
    rng = np.random.default_rng(77)
    lens = rng.integers(0, 2500, 30).astype(np.int32)
    toks = rng.integers(-2**31, 2**31, int(lens.sum()) + 8, dtype=np.int64).astype(np.int32)
    offs = np.concatenate([[0], np.cumsum(lens[:-1])]).astype(np.int64)
    ns = (np.arange(30) % 4).astype(np.int32)
    key_off = oracle.block_offsets(lens)
    want = np.concatenate([oracle.hash_request(toks[offs[r]:offs[r] + lens[r]], int(ns[r])) for r in range(30)])
    dev = torch.device("cuda")
    for shift in range(4):
        base = torch.zeros(len(toks) + 4, dtype=torch.int32, device=dev)
        view = base[shift:shift + len(toks)]
        view.copy_(torch.from_numpy(toks))
        assert view.data_ptr() % 16 == 4 * shift
        keys = torch.empty(max(int(key_off[-1]), 1), dtype=torch.int64, device=dev)
        status = torch.zeros(1, dtype=torch.int32, device=dev)
        P.pc_hash_blocks(view, torch.from_numpy(offs).to(dev), torch.from_numpy(lens).to(dev),
                         torch.from_numpy(ns).to(dev), torch.from_numpy(key_off).to(dev),
                         keys[:int(key_off[-1])], status, None)
        assert int(status.item()) == 0
        assert np.array_equal(keys[:int(key_off[-1])].cpu().numpy().view(np.uint64), want), f"shift {shift}"


def test_replay_step_boundary():
    """Requests of 255, 256, 257, 511, 512 and 513 blocks, on both sides of
    the 256-position lookup step (one-step requests keep their outcome in
    registers, longer ones go through the position arrays), with shared
    prefixes, duplicates within a request and keys reused across requests so
    that hits, orphans and duplicates all occur; every policy and
    PrefixShield flag at capacities below, at and above one step."""
    res = run_key_traces(*step_boundary_batch())
    # the crafted traces must actually produce duplicates and orphans
    assert sum(g["dups"] for groups, _, _ in res for g in groups) > 0
    assert sum(g["orphans"] for groups, _, _ in res for g in groups) > 0


def test_replay_extreme_debt_parameters():
    """Refill at the ABI's limits: rho up to 2^40 and beta, eps up to 2^50
    (Q16), tick gaps up to 2^40 and runs of equal ticks, so that rho * dt
    needs more than 64 bits and balances swing over most of the int64 range
    the accounting allows; every policy, PrefixShield with and without its
    debt gate."""
    kts, per = [], []
    for seed in range(8):
        rng = np.random.default_rng(7700 + seed)
        kt = tg.random_key_trace(7700 + seed, n_req=120, max_blocks=40, n_groups=4, n_prefix=16,
                                 n_contracts=3, key_universe=150, with_ticks=False)
        R = kt.n_req
        gaps = np.where(rng.random(R) < 0.3, 0, rng.integers(0, 1 << 40, R, dtype=np.int64))
        kt.tick = np.cumsum(gaps).astype(np.int64)
        insts = []
        for pol in POLICIES:
            for flags in ([0, 2] if pol == tg.POLICY_PREFIXSHIELD else [0]):
                # rates up to 2^40, at most a factor 2^16 apart (the Q16 limit of 1/w)
                base = int(rng.choice([1, 7, 1 << 20, 1 << 24]))
                contracts = [(min(1 << 40, base * int(rng.choice([1, 3, 1 << 10, 1 << 16]))),
                              int(rng.choice([0, 5, 1 << 50]))) for _ in range(3)]
                insts.append(tg.Instance(0, pol, int(rng.integers(20, 120)), contracts=contracts, flags=flags,
                                         eps_q16=int(rng.choice([0, 1 << 30, 1 << 50]))))
        kts.append(kt)
        per.append(insts)
    run_key_traces(kts, per)


def test_replay_rate_ratio_at_the_q16_limit():
    """Two contracts 2^16 apart in refill rate (the fast one's 1/w is one
    Q16 unit, the smallest positive decrement of Eq. 8), both indebted by
    groups that use both, with equal ticks so that no debt refills and
    PrefixShield's victim runs are long: every policy, PrefixShield with and
    without segmentation and its gate, per-request outputs too."""
    kts, per = [], []
    for seed in range(6):
        rng = np.random.default_rng(5150 + seed)
        kt = tg.random_key_trace(5150 + seed, n_req=200, max_blocks=30, n_groups=4, n_prefix=16,
                                 n_contracts=2, key_universe=120)
        kt.tick = np.zeros(kt.n_req, np.int64)
        slow = int(rng.choice([1, 1 << 24]))
        contracts = [(slow, 0), (slow << 16, 0)]
        insts = [tg.Instance(0, pol, int(rng.integers(16, 100)), contracts=contracts, flags=flags)
                 for pol in POLICIES for flags in ([0, 1, 2] if pol == tg.POLICY_PREFIXSHIELD else [0])]
        kts.append(kt)
        per.append(insts)
    res = run_key_traces(kts, per)
    assert sum(g["evicted_owned"] for groups, _, _ in res for g in groups) > 0


def test_replay_capacity_at_most_groups():
    """Capacities from 1 to a little above the number of groups: StaticQuota
    partitions of floor(C/G) = 0 (every probe truncated, nothing cached) and
    of one or two blocks, and the other policies at the same tiny sizes."""
    kts, per = [], []
    for seed in range(6):
        G = 5 + seed % 4
        kt = tg.random_key_trace(8800 + seed, n_req=150, max_blocks=12, n_groups=G, n_prefix=4 * G,
                                 n_contracts=2, key_universe=30, with_ticks=bool(seed % 2))
        insts = [tg.Instance(0, pol, cap, contracts=[(tg.Q16, 2 * tg.Q16), (tg.Q16 // 2, 0)])
                 for pol in POLICIES for cap in range(1, G + 4)]
        kts.append(kt)
        per.append(insts)
    res = run_key_traces(kts, per)
    # StaticQuota below one block per group caches nothing
    k = 0
    for kt, insts in zip(kts, per):
        for inst in insts:
            groups, istats, _ = res[k]
            k += 1
            if inst.policy == tg.POLICY_STATICQUOTA and inst.capacity < kt.n_groups:
                assert all(g["hits"] == 0 and g["charged"] == 0 for g in groups)
                assert istats["resident_max"] == 0


@pytest.mark.parametrize("dense", [False, True])
def test_replay_default_4096_layout(dense):
    """4096-block instances with default S3-FIFO settings, one contract,
    eps = 0 and no flags, on traces of at most 512 blocks per request, run
    the kernel's copy compiled for that layout; with other settings,
    contracts or capacities they run the general one.  Both against the
    oracle on crafted traces that overflow the cache (duplicates, orphans,
    requests past one lookup step), every policy.  dense: in a batch larger
    than the GPU holds at once, where the planner takes the hybrid layout
    (keys, prefix ids and ghost table in HBM; compile-time copies of that
    layout too)."""
    kts, per = [], []
    for seed in range(3):
        rng = np.random.default_rng(6100 + seed)
        G = 4
        reqs, groups, hist = [], [], []
        for r in range(90):
            n = int(rng.choice([40, 200, 256, 257, 400, 512]))
            ks = list(hist[int(rng.integers(0, len(hist)))][:int(rng.integers(0, 300))]) if hist and rng.random() < 0.5 else []
            while len(ks) < n:
                ks.append(int(rng.integers(1, 12000)))
            ks = ks[:n]
            hist.append(ks)
            reqs.append(ks)
            groups.append(int(rng.integers(0, G)))
        keys = np.array([k for r in reqs for k in r], dtype=np.uint64)
        off = np.concatenate([[0], np.cumsum([len(r) for r in reqs])]).astype(np.int64)
        R = len(reqs)
        ticks = np.cumsum(rng.integers(0, 3, R)).astype(np.int64)
        grp = np.array(groups, np.uint8)
        pfx = (np.array(groups) * 2 + np.arange(R) % 2).astype(np.uint32)
        one = [(tg.Q16 * 40 // 6, 192 * tg.Q16)]
        two = [(tg.Q16 * 40, 192 * tg.Q16), (tg.Q16 * 16, 128 * tg.Q16)]
        # one contract: the compile-time copy
        kts.append(tg.KeyTrace(keys, off, grp, np.zeros(R, np.uint8), pfx, G, 2 * G, ticks))
        per.append([tg.Instance(0, pol, 4096, contracts=one) for pol in POLICIES] +
                   [tg.Instance(0, tg.POLICY_PREFIXSHIELD, 4096, contracts=one, flags=f) for f in (1, 2)] +
                   [tg.Instance(0, tg.POLICY_PREFIXSHIELD, 4096, contracts=one, eps_q16=4 * tg.Q16),
                    tg.Instance(0, tg.POLICY_LRU, 4095, contracts=one)])
        # two contracts, other S3-FIFO settings: the general copy
        kts.append(tg.KeyTrace(keys, off, grp, (np.arange(R) % 2).astype(np.uint8), pfx, G, 2 * G, ticks))
        per.append([tg.Instance(0, pol, 4096, contracts=two) for pol in POLICIES] +
                   [tg.Instance(0, tg.POLICY_S3FIFO, 4096, contracts=two, s3_small_permille=250),
                    tg.Instance(0, tg.POLICY_S3FIFO, 4096, contracts=two, s3_move_threshold=2)])
    res = run_key_traces(kts, per, dense=dense)
    assert sum(inst["evictions"] for _, inst, _ in res) > 0

def test_replay_is_deterministic_and_order_free():
    """Instances are independent: launching the same batch twice gives
    identical records, and so does a shuffled instance order (the planner
    reorders instances by cost and by layout) once mapped back, per-request
    outputs included.  Mixed capacities put instances in both the LDS and
    the workspace layouts."""
    traces, insts = tg.workload("chat", seeds=[0, 1], n_requests=3000, policies=tuple(POLICIES))
    traces2, insts2 = tg.workload("onetouch4096", seeds=[0], n_requests=2000, policies=tuple(POLICIES))
    for i in insts2:
        i.trace += len(traces)
    traces += traces2
    insts += insts2
    dts = [gpu_hash(tr)[0] for tr in traces]
    b = dv.ReplayBatch(dts, insts, per_request=True)
    b.launch()
    r1, p1 = b.results(), b.per_request_arrays()
    b.launch()
    r2, p2 = b.results(), b.per_request_arrays()
    assert r1 == r2
    assert all(np.array_equal(a, c) for a, c in zip(p1, p2))
    perm = np.random.default_rng(11).permutation(len(insts))
    bs = dv.ReplayBatch(dts, [insts[k] for k in perm], per_request=True)
    bs.launch()
    rs, ps = bs.results(), bs.per_request_arrays()
    for j, k in enumerate(perm):
        assert rs[j] == r1[k], f"instance {k} ({insts[k].label}) differs when launched at position {j}"
        assert np.array_equal(ps[j], p1[k])
    assert all(st == 0 for _, _, st in r1)


@pytest.mark.parametrize("dense", [False, True])
def test_replay_large_capacities_both_layouts(dense):
    """Capacities of 1,500 to 9,000 blocks on crafted traces with hits,
    orphans, duplicates and requests past one lookup step, every policy and
    ablation, 1-3 contracts, S3-FIFO settings: alone, their state is whole in
    LDS (or in the workspace beyond its size); in a batch larger than the
    GPU holds at once, the planner takes the hybrid layout wherever it fits
    more instances per CU.  Per-request outputs too."""
    kts, per = [], []
    for seed in range(4):
        rng = np.random.default_rng(4400 + seed)
        nc = 1 + seed % 3
        kt = tg.random_key_trace(4400 + seed, n_req=160, max_blocks=700, n_groups=5, n_prefix=40, n_contracts=nc,
                                 key_universe=6000, with_ticks=bool(seed % 2))
        insts = []
        for pol in POLICIES:
            for flags in ([0, 1, 2] if pol == tg.POLICY_PREFIXSHIELD else [0]):
                contracts = [(int(rng.integers(tg.Q16 // 4, 4 * tg.Q16)), int(rng.integers(0, 64)) * tg.Q16)
                             for _ in range(nc)]
                insts.append(tg.Instance(0, pol, int(rng.choice([1500, 2048, 3000, 4096, 6000, 9000])),
                                         contracts=contracts, flags=flags,
                                         s3_small_permille=int(rng.choice([0, 100, 250, 1000])),
                                         s3_move_threshold=int(rng.choice([0, 1, 2]))))
        kts.append(kt)
        per.append(insts)
    res = run_key_traces(kts, per, dense=dense)
    assert sum(g["orphans"] for groups, _, _ in res for g in groups) > 0
    assert sum(i["evictions"] for _, i, _ in res) > 0


def test_trace_set_hashes_and_replays_like_separate_traces():
    """Traces hashed together (one block-offsets and one hash call over a
    shared token buffer, as bench.py does) give every trace's keys, and a
    replay over the set's per-trace views gives the oracle's records --
    traces with and without ticks, of different group counts, mixed."""
    traces = (tg.workload("tiny", seeds=[0], n_requests=900)[0] + tg.workload("chat_bursty", seeds=[1], n_requests=1500)[0]
              + tg.workload("onetouch4096", seeds=[2], n_requests=700)[0] + tg.workload("tiers", seeds=[0], n_requests=800)[0])
    ts = dv.TraceSet(traces).hash()
    assert int(ts.dt.status.item()) == 0
    okeys = [oracle.hash_trace(tr) for tr in traces]
    for j, (k, off) in enumerate(okeys):
        assert np.array_equal(ts.trace_keys(j), k), f"trace {j}: keys differ"
        assert np.array_equal(ts.trace_key_off(j), off), f"trace {j}: key offsets differ"
    insts = []
    for j, tr in enumerate(traces):
        for pol in POLICIES:
            insts.append(tg.Instance(j, pol, [256, 2048, 4096, 1024][j],
                                     contracts=list(tg.TIER_CONTRACTS) if j == 3 else [(tg.DEFAULT_RHO_Q16, tg.DEFAULT_BETA_Q16)]))
    res, pr = replay_gpu(ts.views, insts, per_request=True)
    for k, spec in enumerate(insts):
        o = oracle.replay_trace(traces[spec.trace], okeys[spec.trace][0], okeys[spec.trace][1], spec, per_request=True)
        assert_same(res[k], o, f"trace {spec.trace} {tg.POLICY_NAMES[spec.policy]}")
        assert np.array_equal(pr[k], o.per_request)
