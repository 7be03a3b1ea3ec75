"""Pins for the oracle's PCH64 block keys.

The paper does not define the block hash (it keeps the serving engine's
native content key, Sec. III-A and Sec. IV), so PCH64 is this build's own
definition.  These tests pin the oracle's implementation of it against
things other than itself:
  * the NH key constants re-derived here from their definition
    (fractional part of sqrt of the first 16 primes, Decimal arithmetic);
  * fmix64 against an inverse derived here from the MurmurHash3 finalizer's
    structure (xor-shift inverse, modular inverses of the multipliers);
  * closed forms of the NH digest (all factors 1 -> 8; a zero even factor
    cancels its partner);
  * the closed form of the affine chain, H_k = A^(k+1) H_-1 + sum A^(k-j) c_j,
    evaluated with Python integers;
  * structural properties: prefix extension, namespace separation,
    a token change affects exactly the keys from its block on.
"""
import os
from decimal import Decimal, getcontext

import numpy as np
import pytest

import oracle

M64 = (1 << 64) - 1
A = 0x9E3779B97F4A7C15
PRIMES = [2, 3, 5, 7, 11, 13, 17, 19, 23, 29, 31, 37, 41, 43, 47, 53]


def nh_keys():
    getcontext().prec = 60
    out = []
    for p in PRIMES:
        s = Decimal(p).sqrt()
        out.append(int((s - int(s)) * (1 << 31)) + 1)
    return out


def unxorshift(z, s):
    x = z
    for _ in range(64 // s + 1):
        x = z ^ (x >> s)
    return x & M64


def unfmix64(z):
    c1inv = pow(0xff51afd7ed558ccd, -1, 1 << 64)
    c2inv = pow(0xc4ceb9fe1a85ec53, -1, 1 << 64)
    z = unxorshift(z, 33)
    z = (z * c2inv) & M64
    z = unxorshift(z, 33)
    z = (z * c1inv) & M64
    z = unxorshift(z, 33)
    return z


def test_fmix64_is_the_murmur3_finalizer_bijection():
    rng = np.random.default_rng(1)
    assert oracle.fmix64(0) == 0
    for x in [1, 2, 3, M64, 1 << 63] + [int(v) for v in rng.integers(0, 2**63, 200, dtype=np.int64)]:
        y = oracle.fmix64(x)
        assert unfmix64(y) == x
    # avalanche sanity: flipping one input bit flips about half the output bits
    flips = [bin(oracle.fmix64(1 << b) ^ oracle.fmix64(0)).count("1") for b in range(64)]
    assert 20 < np.mean(flips) < 44


def _tok_for_factor(k, want):
    """token (int32) with (uint32(token) + k) mod 2^32 == want"""
    u = (want - k) % (1 << 32)
    return u - (1 << 32) if u >= (1 << 31) else u


def test_nh_digest_closed_forms():
    K = nh_keys()
    assert all(1 <= k <= 1 << 31 for k in K)
    ones = np.array([_tok_for_factor(K[i], 1) for i in range(16)], np.int32)
    assert oracle.block_digest(ones) == 8
    # factor values f_i chosen freely: digest = sum f_{2i} f_{2i+1} mod 2^64
    rng = np.random.default_rng(7)
    for _ in range(50):
        f = [int(x) for x in rng.integers(0, 2**32, 16, dtype=np.uint64)]
        toks = np.array([_tok_for_factor(K[i], f[i]) for i in range(16)], np.int32)
        want = sum(f[2 * i] * f[2 * i + 1] for i in range(8)) & M64
        assert oracle.block_digest(toks) == want
    # a zero even factor cancels its odd partner (the known NH weakness); the
    # cancelling token value is negative, outside any vocabulary id
    base = rng.integers(0, 32000, 16).astype(np.int32)
    for i in range(8):
        z = _tok_for_factor(K[2 * i], 0)
        assert z < 0
        a = base.copy(); a[2 * i] = z
        b = a.copy(); b[2 * i + 1] = (int(a[2 * i + 1]) + 17) % 32000
        assert oracle.block_digest(a) == oracle.block_digest(b)


def test_chain_closed_form():
    rng = np.random.default_rng(3)
    for ns in [0, 1, 5, 63]:
        L = int(rng.integers(16, 400))
        toks = rng.integers(0, 32000, L).astype(np.int32)
        keys = oracle.hash_request(toks, ns)
        nb = L // 16
        assert len(keys) == nb
        c = [oracle.fmix64(oracle.block_digest(toks[16 * j:16 * j + 16])) for j in range(nb)]
        h0 = oracle.fmix64(ns + 1)
        for k in range(nb):
            H = (pow(A, k + 1, 1 << 64) * h0 + sum(pow(A, k - j, 1 << 64) * c[j] for j in range(k + 1))) & M64
            assert int(keys[k]) == oracle.fmix64(H)


def test_prefix_extension_and_partial_tail():
    rng = np.random.default_rng(4)
    toks = rng.integers(0, 32000, 16 * 40 + 9).astype(np.int32)
    full = oracle.hash_request(toks, 1)
    assert len(full) == 40                   # the 9-token tail has no key
    for k in [0, 1, 7, 39]:
        assert np.array_equal(oracle.hash_request(toks[:16 * k + 15], 1), full[:k])
        assert np.array_equal(oracle.hash_request(toks[:16 * (k + 1)], 1), full[:k + 1])


def test_namespace_separation_and_locality():
    rng = np.random.default_rng(5)
    toks = rng.integers(0, 32000, 16 * 30).astype(np.int32)
    ks = [oracle.hash_request(toks, ns) for ns in range(8)]
    for a in range(8):
        for b in range(a + 1, 8):
            assert np.all(ks[a] != ks[b])     # different at every depth
    base = ks[0]
    for blk in [0, 3, 29]:
        for pos in [0, 5, 15]:
            t2 = toks.copy(); t2[16 * blk + pos] += 1
            k2 = oracle.hash_request(t2, 0)
            assert np.array_equal(k2[:blk], base[:blk])
            assert np.all(k2[blk:] != base[blk:])
    # swapping two different blocks changes the keys from the first of them on
    t3 = toks.copy(); t3[16 * 2:16 * 3], t3[16 * 5:16 * 6] = toks[16 * 5:16 * 6], toks[16 * 2:16 * 3]
    k3 = oracle.hash_request(t3, 0)
    assert np.array_equal(k3[:2], base[:2]) and np.all(k3[2:] != base[2:])


def test_golden_vectors():
    """Frozen known-answer vectors, written by tests/golden/make_golden.py
    (which calls only the oracle): guards the definition against drift."""
    path = os.path.join(os.path.dirname(__file__), "golden", "pch64_vectors.txt")
    with open(path) as f:
        lines = [l.split() for l in f if l.strip() and not l.startswith("#")]
    assert lines
    for row in lines:
        ns, seed, L = int(row[0]), int(row[1]), int(row[2])
        want = [int(x, 16) for x in row[3:]]
        toks = np.random.Generator(np.random.PCG64(seed)).integers(-2**31, 2**31, L, dtype=np.int64).astype(np.int32)
        got = [int(x) for x in oracle.hash_request(toks, ns)]
        assert got == want


def test_block_offsets_definition():
    """The plain offsets definition agrees with the C oracle's hash pass
    (which writes its own CSR offsets) and with a hand count: only full
    16-token blocks count, and a negative length counts as none."""
    from paper_2608_01657_amd import tracegen as tg
    traces, _ = tg.workload("tiny", seeds=[0], n_requests=300)
    tr = traces[0]
    _, off = oracle.hash_trace(tr)
    assert np.array_equal(oracle.block_offsets(tr.length), off)
    assert list(oracle.block_offsets([0, 15, 16, 17, 31, 32, -5, 1024 + 15])) == [0, 0, 0, 1, 2, 3, 5, 5, 69]
    assert list(oracle.block_offsets([])) == [0]
