"""Host-side request metrics and the attack trace shapes."""
import numpy as np

from paper_2608_01657_amd import metrics
from paper_2608_01657_amd import tracegen as tg


def test_hit_ratio_arithmetic():
    pr = np.array([[2, 0, 0, 0], [0, 3, 1, 0], [6, 1, 0, 0], [0, 0, 0, 0]], np.int32)
    L = np.array([40, 48, 100, 0])
    r = metrics.hit_ratios(pr, L)
    assert np.allclose(r, [32 / 40, 0.0, 96 / 100, 0.0])

    class T:
        length = L
        group = np.array([0, 1, 0, 1])
    assert np.isclose(metrics.mean_hit_ratio(pr, T, group=0), (0.8 + 0.96) / 2)
    assert np.isclose(metrics.mean_hit_ratio(pr, T), (0.8 + 0.96) / 4)


def test_paired_bootstrap():
    a = [0.5, 0.6, 0.7, 0.8]
    m, lo, hi = metrics.paired_bootstrap(a, [x - 0.1 for x in a])
    assert np.isclose(m, 0.1) and np.isclose(lo, 0.1) and np.isclose(hi, 0.1)
    m, lo, hi = metrics.paired_bootstrap([1, 0, 1, 0, 1, 0], [0, 1, 0, 1, 0, 1], n_boot=2000)
    assert m == 0 and lo < 0 < hi


def test_attack_trace_shapes():
    n = 4000
    for kind in tg.ATTACK_KINDS:
        tr = tg.attack_trace(kind, 7000, n)
        assert tr.n_req == n
        pol = tr.group == 1
        assert not pol[: n // 10].any(), "warm-up is victim-only"
        v = ~pol
        assert (tr.length[v] == 1536 + 64).all() and (tr.length[pol] == 1536).all()
        assert set(np.unique(tr.prefix[v])) <= {0, 1, 2, 3}
        if kind == "none":
            assert not pol.any()
        elif kind == "lowslow":
            assert pol.sum() == sum(1 for r in range(n // 10, n) if r % 8 == 7)
        else:
            assert pol.sum() == sum(1 for r in range(n // 10, n) if r % 2 == 1)
        if kind == "replay":   # every polluter prompt twice in a row, same view and prefix id
            idx = np.nonzero(pol)[0]
            assert (tr.tok_off[idx[0::2]] == tr.tok_off[idx[1::2]]).all()
            assert (tr.prefix[idx[0::2]] == tr.prefix[idx[1::2]]).all()
            assert len(set(tr.prefix[idx[0::2]].tolist())) == len(idx) // 2
        elif kind in ("onetouch", "lowslow"):
            assert len(set(tr.prefix[pol].tolist())) == pol.sum()


def test_bursty_ticks():
    traces, insts = tg.workload("chat_bursty", seeds=[0], n_requests=1000)
    t = traces[0].tick
    assert t is not None and (np.diff(t) >= 0).all() and t[31] == 0 and t[32] == 32
