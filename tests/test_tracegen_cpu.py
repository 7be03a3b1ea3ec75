"""The seeded input generators: every workload's traces are a pure function
of the seed, and the lazily built token stream gives exactly the tokens that
drawing each request's fresh tokens in turn gives (so that its one bulk draw
changed no trace)."""
import hashlib

import numpy as np
import pytest

from paper_2608_01657_amd import tracegen as tg


def _fingerprint(tr):
    h = hashlib.sha256()
    for a in (tr.tokens, tr.tok_off, tr.length, tr.group, tr.contract, tr.prefix):
        h.update(np.ascontiguousarray(a).tobytes())
    h.update(str((tr.n_groups, tr.n_prefix, None if tr.tick is None else tr.tick.tobytes())).encode())
    return h.hexdigest()[:16]


# Short traces of every recipe, fingerprinted when the recipes were fixed.
RECIPES = {
    ("tiny", 0, None): "f99ac373c1f07305",
    ("twopass", 1, 999): "5be5bc1b20207b29",
    ("delayed", 2, 5001): "7cd856cfcbef25c6",
    ("attack_none", 0, None): "e1bf778987ea5bf7",
    ("attack_onetouch", 1, None): "2012184e1e9ef89b",
    ("attack_lowslow", 0, None): "cf3053bc382398f4",
    ("attack_replay", 0, None): "60606d1dfcf57227",
    ("selector512x8", 0, None): "4a0ece66bf032c0e",
    ("selector4096x32", 1, None): "983f74c6d75627a1",
    ("chat_bursty", 0, 3000): "577c32ca54205d15",
    ("onetouch4096", 1, 777): "5d3530adbcad3811",
}


@pytest.mark.parametrize("name,seed,n", sorted(RECIPES))
def test_recipes_unchanged(name, seed, n):
    traces, _ = tg.workload(name, seeds=[seed], n_requests=n)
    assert _fingerprint(traces[0]) == RECIPES[(name, seed, n)]


def test_lazy_stream_equals_per_request_draws():
    rng = np.random.default_rng(5)
    parts = [(None if i % 3 else rng.integers(0, 9, int(rng.integers(0, 40)), dtype=np.int32),
              int(rng.integers(0, 300))) for i in range(200)]
    st = tg._Stream(tg._rng(77))
    offs = [st.add(p, n) for p, n in parts]
    got = st.tokens()
    ref_rng = tg._rng(77)
    ref = []
    for p, n in parts:
        if p is not None:
            ref.append(p)
        ref.append(ref_rng.integers(0, tg.VOCAB, size=n, dtype=np.int32))
    ref = np.concatenate(ref)
    assert np.array_equal(got, ref)
    lens = [(0 if p is None else len(p)) + n for p, n in parts]
    assert offs == list(np.concatenate([[0], np.cumsum(lens)[:-1]]))
