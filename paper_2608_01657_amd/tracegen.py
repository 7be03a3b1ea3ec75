"""Seeded synthetic multi-tenant prefix-cache traces.

This module only draws inputs: token ids, request descriptors (accounting
group, service contract, logical prefix id) and replay-instance parameter
sets.  It holds none of the replay or hashing arithmetic, so both the CPU
oracle and the GPU path consume exactly the same inputs.

The workload shapes stand in for the paper's evaluation traces (Sec. V-A,
"Workloads": one-touch pollution, two-pass replay, delayed replay of the
debt-gate ablation in Sec. V-D, and ShareGPT-like benign conversations).
Neither the paper's traces nor ShareGPT are used; every token id is a
uniform draw from [0, 32000) by numpy's PCG64 generator.

A trace is a token stream plus per-request (offset, length) views into it.
Views may alias: a replayed prompt, and every turn of a conversation, point
back into tokens that are already in the stream.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

VOCAB = 32000
BLOCK_TOKENS = 16          # tokens per KV block (Sec. V-A: 16-token blocks)
Q16 = 1 << 16              # fixed-point scale: 2^16 represents one block

POLICY_LRU = 0
POLICY_S3FIFO = 1
POLICY_PREFIXSHIELD = 2
POLICY_STATICQUOTA = 3
POLICY_NAMES = {POLICY_LRU: "lru", POLICY_S3FIFO: "s3fifo", POLICY_PREFIXSHIELD: "prefixshield",
                POLICY_STATICQUOTA: "staticquota"}

FLAG_NO_SEGMENTATION = 1   # ablation of Sec. V-D, Fig. 3a
FLAG_NO_DEBT_GATE = 2      # ablation of Sec. V-D, Fig. 3b

# Standard contract tier of Sec. V-A (40 blocks/s refill, 192-block burst),
# with one request per tick at the paper's ~6 req/s operating point.
DEFAULT_RHO_Q16 = (40 * Q16 + 3) // 6   # 436907 = 40/6 blocks per tick, rounded
DEFAULT_BETA_Q16 = 192 * Q16


@dataclass
class Trace:
    name: str
    tokens: np.ndarray          # int32 [T]
    tok_off: np.ndarray         # int64 [R]
    length: np.ndarray          # int32 [R]
    group: np.ndarray           # uint8 [R]
    contract: np.ndarray        # uint8 [R]
    prefix: np.ndarray          # uint32 [R], dense per (group, logical prefix)
    n_groups: int
    n_prefix: int
    tick: Optional[np.ndarray] = None   # int64 [R] non-decreasing, or None
    roles: dict = field(default_factory=dict)  # group id -> "victim"/"polluter"/...

    @property
    def n_req(self) -> int:
        return int(self.length.shape[0])


@dataclass
class Instance:
    trace: int
    policy: int
    capacity: int
    contracts: List[Tuple[int, int]] = field(
        default_factory=lambda: [(DEFAULT_RHO_Q16, DEFAULT_BETA_Q16)])
    flags: int = 0
    eps_q16: int = 0
    s3_small_permille: int = 100
    s3_move_threshold: int = 1
    label: str = ""


@dataclass
class KeyTrace:
    """A replay input given directly as block keys (tests craft these)."""
    keys: np.ndarray            # uint64 [K]
    key_off: np.ndarray         # int64 [R+1]
    group: np.ndarray
    contract: np.ndarray
    prefix: np.ndarray
    n_groups: int
    n_prefix: int
    tick: Optional[np.ndarray] = None

    @property
    def n_req(self) -> int:
        return int(self.group.shape[0])


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def _zipf_choice(rng, s: float, n: int, size: int) -> np.ndarray:
    w = np.arange(1, n + 1, dtype=np.float64) ** (-s)
    return rng.choice(n, size=size, p=w / w.sum())


def _lognormal_len(rng, mu, sigma, size, lo=1, hi=None) -> np.ndarray:
    x = np.floor(np.exp(rng.normal(mu, sigma, size))).astype(np.int64)
    x = np.maximum(x, lo)
    if hi is not None:
        x = np.minimum(x, hi)
    return x


class _Stream:
    """Builds a token stream from request parts: each request is an optional
    prefix (an existing token array) followed by n fresh uniform tokens.
    The parts are only recorded; tokens() allocates the stream once and draws
    every fresh token in one call, in request order -- the same values as
    drawing each request's fresh tokens as it comes (bounded integer draws
    of a numpy Generator do not depend on how a run of them is split into
    calls), with one copy of the data instead of three."""

    def __init__(self, rng):
        self.rng = rng
        self.parts: List[tuple] = []   # (offset, prefix or None, n_fresh)
        self.pos = 0
        self.n_fresh = 0

    def add(self, prefix: Optional[np.ndarray], n_fresh: int) -> int:
        """Append a request of prefix + n_fresh fresh tokens; return its offset."""
        off = self.pos
        lp = 0 if prefix is None else len(prefix)
        self.parts.append((off, prefix, int(n_fresh)))
        self.pos += lp + int(n_fresh)
        self.n_fresh += int(n_fresh)
        return off

    def tokens(self) -> np.ndarray:
        out = np.empty(self.pos, np.int32)
        fresh = self.rng.integers(0, VOCAB, size=self.n_fresh, dtype=np.int32)
        fo = 0
        for off, prefix, nf in self.parts:
            lp = 0
            if prefix is not None:
                lp = len(prefix)
                out[off:off + lp] = prefix
            out[off + lp:off + lp + nf] = fresh[fo:fo + nf]
            fo += nf
        return out


def _finish(name, stream, offs, lens, groups, prefixes, n_groups, n_prefix, roles):
    R = len(offs)
    return Trace(name=name, tokens=stream.tokens(),
                 tok_off=np.asarray(offs, np.int64), length=np.asarray(lens, np.int32),
                 group=np.asarray(groups, np.uint8), contract=np.zeros(R, np.uint8),
                 prefix=np.asarray(prefixes, np.uint32), n_groups=n_groups,
                 n_prefix=n_prefix, roles=roles)


# --------------------------------------------------------------------------
# Workload recipes
# --------------------------------------------------------------------------

def onetouch_tiny(seed: int = 1000, n_requests: int = 4000) -> Trace:
    """2 groups; victim: one of 4 fixed 512-token hot prefixes (Zipf s=1.0)
    plus a 64-token fresh suffix; polluter: a fresh 512-token prompt.
    Requests alternate victim, polluter."""
    rng = _rng(seed)
    hot = rng.integers(0, VOCAB, size=(4, 512), dtype=np.int32)
    nv = (n_requests + 1) // 2
    z = _zipf_choice(rng, 1.0, 4, nv)
    st = _Stream(rng)
    offs, lens, groups, prefixes = [], [], [], []
    vi = pi = 0
    for r in range(n_requests):
        if r % 2 == 0:
            offs.append(st.add(hot[z[vi]], 64)); lens.append(512 + 64); groups.append(0)
            prefixes.append(int(z[vi])); vi += 1
        else:
            offs.append(st.add(None, 512)); lens.append(512); groups.append(1)
            prefixes.append(4 + pi); pi += 1
    return _finish(f"onetouch_tiny_s{seed}", st, offs, lens, groups, prefixes,
                   2, 4 + pi, {0: "victim", 1: "polluter"})


class _VictimSource:
    """32 hot prefixes of U{1024..4096} tokens, Zipf(0.9), + 128 fresh tokens."""

    def __init__(self, rng, n_hot=32, s=0.9, lo=1024, hi=4096, suffix=128, pid_base=0):
        self.rng = rng
        lens = rng.integers(lo, hi + 1, size=n_hot)
        self.hot = [rng.integers(0, VOCAB, size=int(L), dtype=np.int32) for L in lens]
        self.n_hot, self.s, self.suffix, self.pid_base = n_hot, s, suffix, pid_base

    def draw(self, count):
        return _zipf_choice(self.rng, self.s, self.n_hot, count)

    def emit(self, st: _Stream, z: int):
        return st.add(self.hot[z], self.suffix), len(self.hot[z]) + self.suffix, self.pid_base + int(z)


def _polluter_lengths(rng, n):
    return _lognormal_len(rng, 7.6, 0.5, n, lo=256, hi=8192)


def onetouch_4096(seed: int = 2000, n_requests: int = 50000) -> Trace:
    """Victim (group 0) vs polluter (group 1) at 1:3, pattern V,P,P,P."""
    rng = _rng(seed)
    vic = _VictimSource(rng)
    roles = np.array([0 if r % 4 == 0 else 1 for r in range(n_requests)])
    nv = int((roles == 0).sum()); npol = n_requests - nv
    z = vic.draw(nv)
    plen = _polluter_lengths(rng, npol)
    st = _Stream(rng)
    offs, lens, groups, prefixes = [], [], [], []
    vi = pi = 0
    for r in range(n_requests):
        if roles[r] == 0:
            o, L, pid = vic.emit(st, z[vi]); vi += 1; g = 0
        else:
            L = int(plen[pi]); o = st.add(None, L); pid = 32 + pi; pi += 1; g = 1
        offs.append(o); lens.append(L); groups.append(g); prefixes.append(pid)
    return _finish(f"onetouch_4096_s{seed}", st, offs, lens, groups, prefixes,
                   2, 32 + npol, {0: "victim", 1: "polluter"})


def two_pass(seed: int = 3000, n_requests: int = 80000) -> Trace:
    """Victim and polluter alternate; the polluter's n/4 unique prompts are
    replayed once more, in order and with the same prefix ids, right after
    the first pass."""
    rng = _rng(seed)
    vic = _VictimSource(rng)
    nv = (n_requests + 1) // 2
    npol = n_requests - nv
    n_unique = (npol + 1) // 2
    z = vic.draw(nv)
    plen = _polluter_lengths(rng, n_unique)
    st = _Stream(rng)
    offs, lens, groups, prefixes = [], [], [], []
    pol_views = []
    vi = pi = 0
    for r in range(n_requests):
        if r % 2 == 0:
            o, L, pid = vic.emit(st, z[vi]); vi += 1; g = 0
        else:
            if pi < n_unique:
                L = int(plen[pi]); o = st.add(None, L); pol_views.append((o, L))
                pid = 32 + pi
            else:
                k = pi - n_unique
                o, L = pol_views[k]; pid = 32 + k
            pi += 1; g = 1
        offs.append(o); lens.append(L); groups.append(g); prefixes.append(pid)
    return _finish(f"two_pass_s{seed}", st, offs, lens, groups, prefixes,
                   2, 32 + n_unique, {0: "victim", 1: "polluter"})


ATTACK_KINDS = ("none", "onetouch", "lowslow", "replay")


def attack_trace(kind: str, seed: int = 7000, n_requests: int = 4000) -> Trace:
    """The attack traces at the scale of the paper's setup: a victim group
    with four 1,536-token hot prefixes (96 blocks each, 384 in all; Zipf 1.0)
    plus 64 fresh tokens, and a polluter sending 1,536-token prompts.  The
    first tenth of the trace is victim-only (the victim's prefixes are warm
    and its creation debt has cleared when the attack starts); then:
      none      victim requests only (the no-attack control)
      onetouch  victim and a fresh polluter prompt alternate
      lowslow   one fresh polluter prompt every 8th request (the same kind of
                pressure, spread over time)
      replay    alternating; every polluter prompt is sent twice in a row
                (same prefix id), so its second request finds the blocks it
                created -- apparent reuse that the debt gate must not turn
                into protection"""
    if kind not in ATTACK_KINDS:
        raise ValueError(kind)
    rng = _rng(seed)
    hot = rng.integers(0, VOCAB, size=(4, 1536), dtype=np.int32)
    r_ = np.arange(n_requests)
    if kind == "none":
        pol = np.zeros(n_requests, bool)
    elif kind == "lowslow":
        pol = (r_ % 8) == 7
    else:
        pol = (r_ % 2) == 1
    pol &= r_ >= n_requests // 10
    nv = int((~pol).sum()); npol = int(pol.sum())
    z = _zipf_choice(rng, 1.0, 4, nv)
    n_unique = (npol + 1) // 2 if kind == "replay" else npol
    st = _Stream(rng)
    offs, lens, groups, prefixes = [], [], [], []
    views = []
    vi = pi = 0
    for r in range(n_requests):
        if not pol[r]:
            offs.append(st.add(hot[z[vi]], 64)); lens.append(1536 + 64); groups.append(0)
            prefixes.append(int(z[vi])); vi += 1
        else:
            if kind == "replay" and pi % 2 == 1:
                k = pi // 2
                o = views[k]; pid = 4 + k
            else:
                o = st.add(None, 1536); views.append(o); pid = 4 + len(views) - 1
            offs.append(o); lens.append(1536); groups.append(1); prefixes.append(pid); pi += 1
    return _finish(f"attack_{kind}_s{seed}", st, offs, lens, groups, prefixes,
                   2, 4 + max(n_unique, 1), {0: "victim", 1: "polluter"})


def selector_trace(n_groups: int, seed: int = 8000, n_requests: int = 20000) -> Trace:
    """Reclamation under contention from many groups: every request is a
    fresh prompt of lognormal(6.2, 0.5) tokens clipped to [128, 2048] (about
    31 blocks) from group g with probability proportional to g + 1, so every
    group is in debt by a different amount and, once the cache is full,
    every request needs a reclamation batch (the setting of the paper's
    selector-latency measurement, Sec. V-D)."""
    rng = _rng(seed)
    w = np.arange(1, n_groups + 1, dtype=np.float64)
    groups_ = rng.choice(n_groups, size=n_requests, p=w / w.sum())
    L_ = _lognormal_len(rng, 6.2, 0.5, n_requests, lo=128, hi=2048)
    st = _Stream(rng)
    offs, lens, groups, prefixes = [], [], [], []
    for r in range(n_requests):
        L = int(L_[r])
        offs.append(st.add(None, L)); lens.append(L); groups.append(int(groups_[r])); prefixes.append(r)
    return _finish(f"selector_g{n_groups}_s{seed}", st, offs, lens, groups, prefixes, n_groups, n_requests, {})


def delayed_replay(seed: int = 4000, n_requests: int = 200000) -> Trace:
    """8 groups: 6 benign (8 private 2048-token prefixes, Zipf 1.1, +128
    fresh tokens), a victim (as in the one-touch workload) and a polluter.
    Phases (fractions of the trace): [0, .2) every 4th request is a new
    polluter prompt; [.2, .45) no polluter (the delay); [.45, .65) every 4th
    request replays the polluter prompts in order; [.65, 1) no polluter."""
    rng = _rng(seed)
    benign_hot = [[rng.integers(0, VOCAB, size=2048, dtype=np.int32) for _ in range(8)]
                  for _ in range(6)]
    vic = _VictimSource(rng, pid_base=48)
    b1 = int(0.20 * n_requests); b2 = int(0.45 * n_requests)
    b3 = int(0.65 * n_requests)
    kinds = np.empty(n_requests, np.int64)   # 0..6 benign/victim group, 7 = polluter
    n_other = 0
    for r in range(n_requests):
        pol = (r < b1 or b2 <= r < b3) and (r % 4 == 3)
        kinds[r] = 7 if pol else -1
        n_other += (not pol)
    other_groups = rng.integers(0, 7, size=n_other)
    zb = _zipf_choice(rng, 1.1, 8, n_other)
    zv = vic.draw(n_other)
    n_unique = sum(1 for r in range(b1) if r % 4 == 3)
    plen = _polluter_lengths(rng, n_unique)
    st = _Stream(rng)
    offs, lens, groups, prefixes = [], [], [], []
    pol_views = []
    oi = pi = 0
    for r in range(n_requests):
        if kinds[r] == 7:
            if r < b1:
                L = int(plen[pi]); o = st.add(None, L); pol_views.append((o, L))
                pid = 80 + pi
            else:
                k = pi - n_unique
                if k >= n_unique:   # more replay slots than prompts: wrap
                    k %= n_unique
                o, L = pol_views[k]; pid = 80 + k
            pi += 1; g = 7
        else:
            g = int(other_groups[oi])
            if g < 6:
                zz = int(zb[oi])
                o = st.add(benign_hot[g][zz], 128); L = 2048 + 128; pid = 8 * g + zz
            else:
                o, L, pid = vic.emit(st, zv[oi])
            oi += 1
        offs.append(o); lens.append(L); groups.append(g); prefixes.append(pid)
    roles = {g: "benign" for g in range(6)}
    roles.update({6: "victim", 7: "polluter"})
    return _finish(f"delayed_replay_s{seed}", st, offs, lens, groups, prefixes,
                   8, 80 + n_unique, roles)


# The three service tiers of the paper's setup (premium, standard, basic:
# 64 / 40 / 16 blocks/s refill, bursts 256 / 192 / 128 blocks), converted to
# blocks per request at its ~6 req/s load, in Q16.
TIER_CONTRACTS = [((64 * Q16 + 3) // 6, 256 * Q16),
                  ((40 * Q16 + 3) // 6, 192 * Q16),
                  ((16 * Q16 + 3) // 6, 128 * Q16)]


def tiered_contracts(seed: int = 6000, n_requests: int = 50000) -> Trace:
    """Six tenants on three contract tiers (contract ids 0 premium, 1
    standard, 2 basic):
      g0 premium  victim-like hot prefixes (32, Zipf 0.9, +128 tokens)
      g1 standard 8 private 2048-token prefixes, Zipf 1.1, +128 tokens
      g2 basic    same shape as g1
      g3 two contracts: its prefixes 0-3 are billed to standard, 4-7 to basic
      g4 premium polluter (unique prompts, the one-touch length law)
      g5 basic polluter   (same)
    Each request picks its tenant with weights 20/15/15/15/15/20 %."""
    rng = _rng(seed)
    vic = _VictimSource(rng)
    hot = {g: [rng.integers(0, VOCAB, size=2048, dtype=np.int32) for _ in range(8)] for g in (1, 2, 3)}
    tenants = rng.choice(6, size=n_requests, p=[0.20, 0.15, 0.15, 0.15, 0.15, 0.20])
    zv = vic.draw(n_requests)
    zb = _zipf_choice(rng, 1.1, 8, n_requests)
    plen = _polluter_lengths(rng, n_requests)
    st = _Stream(rng)
    offs, lens, groups, prefixes, contracts = [], [], [], [], []
    n_unique = 0
    for r in range(n_requests):
        g = int(tenants[r])
        if g == 0:
            o, L, pid = vic.emit(st, zv[r]); c = 0
        elif g in (1, 2, 3):
            z = int(zb[r])
            o = st.add(hot[g][z], 128); L = 2048 + 128; pid = 32 + 8 * (g - 1) + z
            c = 1 if g == 1 else 2 if g == 2 else (1 if z < 4 else 2)
        else:
            L = int(plen[r]); o = st.add(None, L); pid = 56 + n_unique; n_unique += 1
            c = 0 if g == 4 else 2
        offs.append(o); lens.append(L); groups.append(g); prefixes.append(pid); contracts.append(c)
    tr = _finish(f"tiered_contracts_s{seed}", st, offs, lens, groups, prefixes, 6, 56 + n_unique,
                 {0: "premium victim", 1: "standard", 2: "basic", 3: "two contracts",
                  4: "premium polluter", 5: "basic polluter"})
    tr.contract = np.asarray(contracts, np.uint8)
    return tr


def conversations(seed: int = 5000, n_requests: int = 100000, n_groups: int = 16,
                  active_per_group: int = 4, max_tokens: int = 16384) -> Trace:
    """Benign multi-turn chats.  Each request picks a group uniformly, then
    one of its active conversations uniformly, and sends that conversation's
    next turn: all prior user+reply tokens plus new user tokens.  A
    conversation has U{2..10} turns; it ends early when its next prompt
    would exceed `max_tokens`, and is then replaced by a new one.  User
    turns ~ floor(exp(N(4.5, 1.0))), replies ~ floor(exp(N(5.5, 0.8))),
    both at least one token.  The logical prefix id is the conversation id.

    Every turn is a view into the conversation's own stream."""
    rng = _rng(seed)
    # a conversation stream is allocated with room for its longest prompt
    st_parts: List[np.ndarray] = []
    pos = 0
    convs = {}     # (g, slot) -> dict

    next_id = 0

    def new_conv():
        nonlocal next_id, pos
        turns = int(rng.integers(2, 11))
        users = _lognormal_len(rng, 4.5, 1.0, turns, lo=1)
        replies = _lognormal_len(rng, 5.5, 0.8, turns, lo=1)
        total = int(users.sum() + replies.sum())
        total = min(total, max_tokens + int(replies.max()) + 1)
        toks = rng.integers(0, VOCAB, size=total, dtype=np.int32)
        c = dict(id=next_id, turns=turns, done=0, users=users, replies=replies,
                 off=pos, ctx=0, cap=total)
        st_parts.append(toks); pos += total; next_id += 1
        return c

    gsel = rng.integers(0, n_groups, size=n_requests)
    ssel = rng.integers(0, active_per_group, size=n_requests)
    offs, lens, groups, prefixes = [], [], [], []
    for r in range(n_requests):
        g = int(gsel[r]); s = int(ssel[r])
        c = convs.get((g, s))
        while True:
            if c is None or c["done"] >= c["turns"]:
                c = new_conv(); convs[(g, s)] = c
            j = c["done"]
            plen = c["ctx"] + int(c["users"][j])
            if plen > max_tokens or plen > c["cap"]:
                c = None
                continue
            break
        offs.append(c["off"]); lens.append(plen); groups.append(g); prefixes.append(c["id"])
        c["ctx"] = plen + int(c["replies"][j])
        c["done"] = j + 1
    tokens = np.concatenate(st_parts) if st_parts else np.zeros(0, np.int32)
    roles = {g: "benign" for g in range(n_groups)}
    return Trace(name=f"conversations_s{seed}", tokens=tokens,
                 tok_off=np.asarray(offs, np.int64), length=np.asarray(lens, np.int32),
                 group=np.asarray(groups, np.uint8), contract=np.zeros(n_requests, np.uint8),
                 prefix=np.asarray(prefixes, np.uint32), n_groups=n_groups,
                 n_prefix=next_id, roles=roles)


# --------------------------------------------------------------------------
# Named workloads: traces x replay instances
# --------------------------------------------------------------------------

ALL_POLICIES = (POLICY_LRU, POLICY_S3FIFO, POLICY_PREFIXSHIELD)


def workload(name: str, seeds: Optional[Sequence[int]] = None,
             n_requests: Optional[int] = None, policies=ALL_POLICIES,
             capacities: Optional[Sequence[int]] = None):
    """Return (traces, instances) of a named workload.

    tiny          2 groups, C=256, 4,000 requests, 1 seed, 3 instances
    onetouch4096  2 groups, C=4096, 50,000 requests, 16 seeds, 48 instances
    twopass       2 groups, C=4096, 80,000 requests, 32 seeds, 96 instances
    delayed       8 groups, C=4096, 200,000 requests, 8 seeds,
                  refill in {1..128} blocks/tick -> 192 instances
    chat          16 groups, C in {1K..16K}, 100,000 requests, 64 seeds, 960
    scale1024     onetouch4096 traces x 64 variants (LRU, S3-FIFO and
                  PrefixShield at 62 refill rates k/4, k=1..62) = 1024
    tiers         6 groups on 3 contract tiers, C=4096, 50,000 requests,
                  8 seeds, 3 policies -> 24
    attack_<kind> the paper-scale attack traces (kind in ATTACK_KINDS),
                  C=511, 4,000 requests, 10 seeds x {LRU, S3-FIFO,
                  PrefixShield, PrefixShield without segmentation, without
                  the debt gate, StaticQuota} -> 60
    selector512x8, selector4096x32
                  one-touch contention from 8 / 32 groups at C = 512 / 4096
                  (the paper's selector measurement sizes), 20,000
                  requests, 4 seeds, 3 policies
    chat_bursty   chat traces whose requests arrive in bursts of 32 per tick
                  (the accounting clock of Eq. 1 advances 32 ticks between
                  bursts), C=4096, 3 policies
    `seeds` selects seed indices (0-based) and `n_requests` shortens traces.
    """
    traces: List[Trace] = []
    inst: List[Instance] = []
    if name == "tiny":
        idx = list(seeds) if seeds is not None else [0]
        for i in idx:
            traces.append(onetouch_tiny(1000 + i, n_requests or 4000))
            for pol in policies:
                inst.append(Instance(len(traces) - 1, pol, 256, label=f"{POLICY_NAMES[pol]}"))
    elif name in ("onetouch4096", "scale1024"):
        idx = list(seeds) if seeds is not None else list(range(16))
        for i in idx:
            traces.append(onetouch_4096(2000 + i, n_requests or 50000))
            t = len(traces) - 1
            if name == "onetouch4096":
                for pol in policies:
                    inst.append(Instance(t, pol, 4096, label=POLICY_NAMES[pol]))
            else:
                inst.append(Instance(t, POLICY_LRU, 4096, label="lru"))
                inst.append(Instance(t, POLICY_S3FIFO, 4096, label="s3fifo"))
                for k in range(1, 63):
                    inst.append(Instance(t, POLICY_PREFIXSHIELD, 4096,
                                         contracts=[(k * Q16 // 4, DEFAULT_BETA_Q16)],
                                         label=f"prefixshield_rho{k}/4"))
    elif name == "twopass":
        idx = list(seeds) if seeds is not None else list(range(32))
        for i in idx:
            traces.append(two_pass(3000 + i, n_requests or 80000))
            for pol in policies:
                inst.append(Instance(len(traces) - 1, pol, 4096, label=POLICY_NAMES[pol]))
    elif name == "delayed":
        idx = list(seeds) if seeds is not None else list(range(8))
        for i in idx:
            traces.append(delayed_replay(4000 + i, n_requests or 200000))
            for rho in (1, 2, 4, 8, 16, 32, 64, 128):
                for pol in policies:
                    inst.append(Instance(len(traces) - 1, pol, 4096,
                                         contracts=[(rho * Q16, DEFAULT_BETA_Q16)],
                                         label=f"{POLICY_NAMES[pol]}_rho{rho}"))
    elif name == "tiers":
        idx = list(seeds) if seeds is not None else list(range(8))
        for i in idx:
            traces.append(tiered_contracts(6000 + i, n_requests or 50000))
            for pol in policies:
                inst.append(Instance(len(traces) - 1, pol, 4096, contracts=list(TIER_CONTRACTS),
                                     label=POLICY_NAMES[pol]))
    elif name.startswith("attack_"):
        kind = name[len("attack_"):]
        idx = list(seeds) if seeds is not None else list(range(10))
        for i in idx:
            traces.append(attack_trace(kind, 7000 + i, n_requests or 4000))
            t = len(traces) - 1
            for pol in policies:
                inst.append(Instance(t, pol, 511, label=POLICY_NAMES[pol]))
            if POLICY_PREFIXSHIELD in policies:
                inst.append(Instance(t, POLICY_PREFIXSHIELD, 511, flags=FLAG_NO_SEGMENTATION,
                                     label="prefixshield_noseg"))
                inst.append(Instance(t, POLICY_PREFIXSHIELD, 511, flags=FLAG_NO_DEBT_GATE,
                                     label="prefixshield_nogate"))
            if POLICY_STATICQUOTA not in policies:   # the paper's partitioned baseline (Table I)
                inst.append(Instance(t, POLICY_STATICQUOTA, 511, label=POLICY_NAMES[POLICY_STATICQUOTA]))
    elif name in ("selector512x8", "selector4096x32"):
        C, G = (512, 8) if name == "selector512x8" else (4096, 32)
        idx = list(seeds) if seeds is not None else list(range(4))
        for i in idx:
            traces.append(selector_trace(G, 8000 + i, n_requests or 20000))
            for pol in policies:
                inst.append(Instance(len(traces) - 1, pol, C, label=POLICY_NAMES[pol]))
    elif name == "chat_bursty":
        idx = list(seeds) if seeds is not None else list(range(8))
        for i in idx:
            tr = conversations(5000 + i, n_requests or 100000)
            tr.tick = (np.arange(tr.n_req, dtype=np.int64) // 32) * 32
            traces.append(tr)
            for pol in policies:
                inst.append(Instance(len(traces) - 1, pol, 4096, label=POLICY_NAMES[pol]))
    elif name == "chat":
        idx = list(seeds) if seeds is not None else list(range(64))
        caps = list(capacities) if capacities is not None else [1024, 2048, 4096, 8192, 16384]
        for i in idx:
            traces.append(conversations(5000 + i, n_requests or 100000))
            for cap in caps:
                for pol in policies:
                    inst.append(Instance(len(traces) - 1, pol, cap,
                                         label=f"{POLICY_NAMES[pol]}_C{cap}"))
    else:
        raise ValueError(f"unknown workload {name!r}")
    return traces, inst


def random_key_trace(seed: int, n_req: int = 30, max_blocks: int = 8,
                     n_groups: int = 3, n_prefix: int = 6, n_contracts: int = 1,
                     key_universe: int = 24, p_share: float = 0.6,
                     with_ticks: bool = False) -> KeyTrace:
    """Tiny adversarial key traces: keys drawn from a small universe so that
    hits, orphans, duplicates and re-references are all frequent.  With
    probability `p_share` a request starts by copying the leading keys of an
    earlier request of the same group."""
    rng = _rng(seed)
    keys: List[int] = []
    off = [0]
    groups = rng.integers(0, n_groups, size=n_req)
    contracts = rng.integers(0, n_contracts, size=n_req)
    # prefix ids are dense per (group, logical prefix)
    per_group = max(1, n_prefix // n_groups)
    lp = rng.integers(0, per_group, size=n_req)
    prefixes = (groups * per_group + lp).astype(np.uint32)
    hist = {}
    for r in range(n_req):
        n = int(rng.integers(0, max_blocks + 1))
        g = int(groups[r])
        ks: List[int] = []
        if hist.get(g) and rng.random() < p_share:
            src = hist[g][int(rng.integers(0, len(hist[g])))]
            take = int(rng.integers(0, len(src) + 1))
            ks = list(src[:take])
        while len(ks) < n:
            ks.append(int(rng.integers(0, key_universe)) + 1000 * g * int(rng.random() < 0.8))
        ks = ks[:n]
        hist.setdefault(g, []).append(ks)
        keys.extend(ks)
        off.append(len(keys))
    tick = None
    if with_ticks:
        tick = np.cumsum(rng.integers(0, 4, size=n_req)).astype(np.int64)
    return KeyTrace(keys=np.asarray(keys, np.uint64), key_off=np.asarray(off, np.int64),
                    group=groups.astype(np.uint8), contract=contracts.astype(np.uint8),
                    prefix=prefixes, n_groups=n_groups, n_prefix=per_group * n_groups,
                    tick=tick)
