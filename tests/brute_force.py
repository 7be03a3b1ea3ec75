"""Scan-based brute-force replay for tiny traces (test-only).

Written independently of oracle/pc_oracle.c: no queues or indexes at all.
Every victim is found by scanning every cached block with an explicit sort
key, the way the paper's prototype selector scans reclaimable candidates in
software (Sec. IV, "Metadata and selector").  S3-FIFO keeps Python lists and
the ghost is the full insertion history with a window test.

Semantics (same reading as the oracle): per request -- OnRequest; lookup
(longest leading resident run, repeated keys are misses that do nothing
else); pin hits; drop resident blocks behind the first miss; OnTouch with
the pre-charge debt; reclaim max(0, new - free) victims; charge and classify
(Eqs. 1-2, Alg. 1); insert deepest-first; release deepest-first; account.
StaticQuota (Sec. V-A baseline): each group owns floor(C/G) blocks, a
request probes at most that many, and its victims are the requester's own
least recently released blocks.
"""
from __future__ import annotations

from typing import Dict, List

Q16 = 1 << 16
PROB, NORMAL, REUSE = 0, 1, 2

GROUP_FIELDS = ["requests", "probes", "hits", "misses", "charged", "evicted_owned",
                "evictions_caused", "promotions", "gated", "orphans", "dups", "truncated",
                "debt_end_q16", "debt_max_q16", "debt_sum_q16", "resident_end", "resident_max"]


def brute_replay(keys, key_off, group, contract, prefix, n_groups, inst, tick=None):
    C = inst.capacity
    pol = inst.policy                  # 0 LRU, 1 S3-FIFO, 2 PrefixShield, 3 StaticQuota
    quota = C // n_groups
    no_seg = bool(inst.flags & 1)
    no_gate = bool(inst.flags & 2)
    eps = inst.eps_q16
    rhos = [c[0] for c in inst.contracts]
    betas = [c[1] for c in inst.contracts]
    K = len(rhos)
    rmin = min(rhos)
    invw = [(rmin << 16) // r for r in rhos]
    if min(invw) < 1:
        raise ValueError("refill rates differ by more than a factor 2^16")
    s_cap = max(1, C * inst.s3_small_permille // 1000)
    g_cap = C - s_cap
    T = inst.s3_move_threshold

    bal = [[betas[c] for c in range(K)] for _ in range(n_groups)]
    last = [[0] * K for _ in range(n_groups)]
    blocks: Dict[int, dict] = {}
    referenced, admitted = set(), set()
    stamp = 0
    S: List[int] = []
    M: List[int] = []
    ghost: List[list] = []     # [key, seq, removed]
    gseq = 0
    st = [{f: 0 for f in GROUP_FIELDS} for _ in range(n_groups)]
    ist = {"evictions": 0, "s3_moves": 0, "s3_reinserts": 0, "s3_ghost_hits": 0,
           "s3_ghost_inserts": 0, "resident_end": 0, "resident_max": 0}
    per_req = []

    def eff(g, c, t):
        return min(betas[c], bal[g][c] + rhos[c] * (t - last[g][c]))

    def raw(g, t):
        return sum(max(0, -eff(g, c, t)) for c in range(K))

    def ndebt(g, t):
        return sum((max(0, -eff(g, c, t)) * invw[c]) >> 16 for c in range(K))

    def dec(g, t):
        ws = [invw[c] for c in range(K) if eff(g, c, t) < 0]
        return min(ws) if ws else 0

    def seg(b):
        return 0 if no_seg else b["cls"]

    def remove(key):
        b = blocks.pop(key)
        if b.get("q") == "S":
            S.remove(key)
        elif b.get("q") == "M":
            M.remove(key)
        return b

    def ghost_live(key):
        for e in ghost:
            if e[0] == key and not e[2] and e[1] >= gseq - g_cap:
                return e
        return None

    t = 0
    R = len(group)
    for r in range(R):
        g, c, p = int(group[r]), int(contract[r]), int(prefix[r])
        t = int(tick[r]) if tick is not None else r
        ks = [int(x) for x in keys[key_off[r]:key_off[r + 1]]]
        o = st[g]
        q1 = p in referenced
        referenced.add(p)
        o["requests"] += 1
        n = min(len(ks), quota if pol == 3 else C)
        o["truncated"] += len(ks) - n
        o["probes"] += n
        ks = ks[:n]

        seen = set()
        dup = [False] * n
        hits, new = [], []
        n_orph = 0
        run = True
        for j, key in enumerate(ks):
            if key in seen:
                dup[j] = True
                o["dups"] += 1
                continue
            seen.add(key)
            if run and key in blocks:
                blocks[key]["pinned"] = True
                hits.append(j)
                continue
            run = False
            if key in blocks:
                remove(key)
                o["orphans"] += 1
                n_orph += 1
            new.append(j)
        h, m = len(hits), len(new)
        o["hits"] += h
        o["misses"] += n - h

        # OnTouch
        if pol == 1:
            for j in hits:
                b = blocks[ks[j]]
                b["freq"] = min(b["freq"] + 1, 3)
        elif pol == 2:
            proven = q1 and (p in admitted)
            d = raw(g, t)
            for j in hits:
                b = blocks[ks[j]]
                if proven and b["owner"] == g and b["contract"] == c and b["prefix"] == p \
                        and b["cls"] != REUSE:
                    if d <= eps or no_gate:
                        b["cls"] = REUSE
                        o["promotions"] += 1
                    else:
                        o["gated"] += 1

        if pol == 3:
            e = max(0, m - (quota - sum(1 for b in blocks.values() if b["owner"] == g)))
        else:
            e = max(0, m - (C - len(blocks)))
        if pol == 2 and e:
            P = [ndebt(x, t) for x in range(n_groups)]
            D = [dec(x, t) for x in range(n_groups)]
        for _ in range(e):
            cands = [(k, b) for k, b in blocks.items() if not b["pinned"]]
            if pol == 0:
                vk = min(cands, key=lambda kb: kb[1]["stamp"])[0]
            elif pol == 3:
                vk = min(((k, b) for k, b in cands if b["owner"] == g), key=lambda kb: kb[1]["stamp"])[0]
            elif pol == 2:
                best = None
                for x in range(n_groups):
                    mine = [b for _, b in cands if b["owner"] == x]
                    if not mine or P[x] <= eps:
                        continue
                    s0 = min(seg(b) for b in mine)
                    hs = min(b["stamp"] for b in mine if seg(b) == s0)
                    keyx = (-P[x], s0, hs)
                    if best is None or keyx < best[0]:
                        best = (keyx, x, s0)
                if best is not None:
                    _, x, s0 = best
                    vk = min(((k, b) for k, b in cands if b["owner"] == x and seg(b) == s0),
                             key=lambda kb: kb[1]["stamp"])[0]
                    P[x] = max(0, P[x] - D[x])
                else:
                    vk = min(cands, key=lambda kb: (seg(kb[1]), kb[1]["stamp"]))[0]
            else:
                while True:
                    s_unp = [k for k in S if not blocks[k]["pinned"]]
                    m_unp = [k for k in M if not blocks[k]["pinned"]]
                    useS = (len(S) >= s_cap and s_unp) or not m_unp
                    if useS:
                        k0 = s_unp[0]
                        if blocks[k0]["freq"] >= T:
                            S.remove(k0)
                            blocks[k0]["freq"] = 0
                            blocks[k0]["q"] = "M"
                            M.append(k0)
                            ist["s3_moves"] += 1
                            continue
                        ghost.append([k0, gseq, False])
                        gseq += 1
                        ist["s3_ghost_inserts"] += 1
                        vk = k0
                        break
                    k0 = m_unp[0]
                    if blocks[k0]["freq"] > 0:
                        M.remove(k0)
                        blocks[k0]["freq"] -= 1
                        M.append(k0)
                        ist["s3_reinserts"] += 1
                        continue
                    vk = k0
                    break
            vb = remove(vk)
            st[vb["owner"]]["evicted_owned"] += 1
            o["evictions_caused"] += 1
            ist["evictions"] += 1

        cls = NORMAL
        if m > 0:
            B = eff(g, c, t) - m * Q16
            bal[g][c] = B
            last[g][c] = t
            o["charged"] += m
            cls = PROB if (B < -eps or p not in admitted) else NORMAL
            admitted.add(p)
        for j in reversed(new):
            key = ks[j]
            b = dict(owner=g, contract=c, prefix=p, cls=cls, freq=0, stamp=None,
                     pinned=True, q=None)
            blocks[key] = b
            if pol == 1:
                gl = ghost_live(key)
                if gl is not None:
                    gl[2] = True
                    b["q"] = "M"
                    M.append(key)
                    ist["s3_ghost_hits"] += 1
                else:
                    b["q"] = "S"
                    S.append(key)
        for j in range(n - 1, -1, -1):
            if dup[j]:
                continue
            b = blocks[ks[j]]
            b["pinned"] = False
            if pol != 1:
                stamp += 1
                b["stamp"] = stamp
        per_req.append((h, m, e, n_orph))
        for x in range(n_groups):
            d = raw(x, t)
            st[x]["debt_sum_q16"] += d
            st[x]["debt_max_q16"] = max(st[x]["debt_max_q16"], d)
            res = sum(1 for b in blocks.values() if b["owner"] == x)
            st[x]["resident_max"] = max(st[x]["resident_max"], res)
        ist["resident_max"] = max(ist["resident_max"], len(blocks))
    for x in range(n_groups):
        st[x]["debt_end_q16"] = raw(x, t) if R else 0
        st[x]["resident_end"] = sum(1 for b in blocks.values() if b["owner"] == x)
    ist["resident_end"] = len(blocks)
    return st, ist, per_req
