"""CPU oracle for the PrefixShield replay hot path -- TEST INFRASTRUCTURE.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product path (the HIP library and its binding)
never loads it and shares no code with it.

`pc_oracle.c` holds the arithmetic (plain single-threaded C, integers only);
this module compiles it with gcc and exposes it through ctypes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import Dict, List, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pc_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

GROUP_FIELDS = ["requests", "probes", "hits", "misses", "charged", "evicted_owned",
                "evictions_caused", "promotions", "gated", "orphans", "dups", "truncated",
                "debt_end_q16", "debt_max_q16", "debt_sum_q16", "resident_end", "resident_max"]
INST_FIELDS = ["evictions", "s3_moves", "s3_reinserts", "s3_ghost_hits", "s3_ghost_inserts",
               "resident_end", "resident_max"]


def build(force: bool = True) -> str:
    """Compile the oracle into oracle/liboracle.so (gcc -O2)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared",
                               "-o", tmp, _SRC])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i64, i32 = ctypes.c_int64, ctypes.c_int32
        L.orc_fmix64.restype = ctypes.c_uint64
        L.orc_fmix64.argtypes = [ctypes.c_uint64]
        L.orc_block_digest.restype = ctypes.c_uint64
        L.orc_block_digest.argtypes = [P]
        L.orc_hash_request.restype = i64
        L.orc_hash_request.argtypes = [P, i64, ctypes.c_uint32, P]
        L.orc_hash_trace.restype = ctypes.c_int
        L.orc_hash_trace.argtypes = [P, P, P, P, i64, P, P]
        L.orc_replay.restype = ctypes.c_int
        L.orc_replay.argtypes = [P, P, P, P, P, P, i64, i32, i64, i32, i64, i32, i32,
                                 P, P, i64, i32, i32, P, P, P]
        L.orc_replay_timed.restype = ctypes.c_int
        L.orc_replay_timed.argtypes = [P, P, P, P, P, P, i64, i32, i64, i32, i64, i32, i32,
                                       P, P, i64, i32, i32, P, P, P, P]
        _lib = L
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def fmix64(x: int) -> int:
    return int(lib().orc_fmix64(ctypes.c_uint64(x & (2**64 - 1))))


def block_digest(tokens16: np.ndarray) -> int:
    t = np.ascontiguousarray(tokens16, dtype=np.int32)
    assert t.shape == (16,)
    return int(lib().orc_block_digest(_ptr(t)))


def hash_request(tokens: np.ndarray, ns: int) -> np.ndarray:
    t = np.ascontiguousarray(tokens, dtype=np.int32)
    out = np.zeros(len(t) // 16, np.uint64)
    n = lib().orc_hash_request(_ptr(t), len(t), ns, _ptr(out))
    assert n == len(out)
    return out


def block_offsets(req_len) -> np.ndarray:
    """CSR offsets of the full 16-token blocks (Sec. III-B: only full KV
    blocks count): off[r] = sum_{i<r} floor(max(len_i, 0) / 16), r = 0..R."""
    n = np.maximum(np.asarray(req_len, np.int64), 0) // 16
    return np.concatenate([np.zeros(1, np.int64), np.cumsum(n, dtype=np.int64)])


def hash_trace(trace):
    """Keys and CSR key offsets of every full block of every request."""
    R = trace.n_req
    total = int((trace.length.astype(np.int64) // 16).sum())
    keys = np.zeros(max(total, 1), np.uint64)
    off = np.zeros(R + 1, np.int64)
    rc = lib().orc_hash_trace(_ptr(np.ascontiguousarray(trace.tokens, np.int32)),
                              _ptr(np.ascontiguousarray(trace.tok_off, np.int64)),
                              _ptr(np.ascontiguousarray(trace.length, np.int32)),
                              _ptr(np.ascontiguousarray(trace.group, np.uint8)),
                              R, _ptr(keys), _ptr(off))
    if rc != 0:
        raise ValueError("oracle hash rejected the trace")
    return keys[:total], off


@dataclass
class ReplayResult:
    groups: List[Dict[str, int]]
    inst: Dict[str, int]
    per_request: Optional[np.ndarray]   # [R, 4]: hits, new blocks, evictions, orphans
    reclaim_ns: Optional[np.ndarray] = None   # [R]: wall-clock ns of each request's reclamation (0: none)


def replay(keys, key_off, group, contract, prefix, n_groups, n_prefix, inst,
           tick=None, per_request=False, time_reclaim=False) -> ReplayResult:
    """Replay one instance (`inst` has the attributes of tracegen.Instance).
    time_reclaim: also return each request's reclamation time (Alg. 2 as
    the oracle runs it: one victim selection at a time)."""
    keys = np.ascontiguousarray(keys, np.uint64)
    if keys.size == 0:
        keys = np.zeros(1, np.uint64)
    key_off = np.ascontiguousarray(key_off, np.int64)
    group = np.ascontiguousarray(group, np.uint8)
    contract = np.ascontiguousarray(contract, np.uint8)
    prefix = np.ascontiguousarray(prefix, np.uint32)
    tick = None if tick is None else np.ascontiguousarray(tick, np.int64)
    R = int(group.shape[0])
    K = len(inst.contracts)
    rho = np.array([c[0] for c in inst.contracts], np.int64)
    beta = np.array([c[1] for c in inst.contracts], np.int64)
    gs = np.zeros((n_groups, len(GROUP_FIELDS)), np.int64)
    st = np.zeros(len(INST_FIELDS), np.int64)
    pr = np.zeros((R, 4), np.int32) if per_request else None
    ns = np.zeros(max(R, 1), np.int64) if time_reclaim else None
    args = (_ptr(keys), _ptr(key_off), _ptr(group), _ptr(contract), _ptr(prefix),
            _ptr(tick), R, n_groups, n_prefix, inst.policy, inst.capacity,
            inst.flags, K, _ptr(rho), _ptr(beta), inst.eps_q16,
            inst.s3_small_permille, inst.s3_move_threshold,
            _ptr(gs), _ptr(st), _ptr(pr))
    rc = lib().orc_replay_timed(*args, _ptr(ns)) if time_reclaim else lib().orc_replay(*args)
    if rc != 0:
        raise ValueError(f"oracle replay rejected the input (rc={rc})")
    groups = [dict(zip(GROUP_FIELDS, map(int, row))) for row in gs]
    return ReplayResult(groups=groups, inst=dict(zip(INST_FIELDS, map(int, st))), per_request=pr,
                        reclaim_ns=None if ns is None else ns[:R])


def replay_key_trace(kt, inst, per_request=False) -> ReplayResult:
    return replay(kt.keys, kt.key_off, kt.group, kt.contract, kt.prefix, kt.n_groups,
                  kt.n_prefix, inst, tick=kt.tick, per_request=per_request)


def replay_trace(trace, keys, key_off, inst, per_request=False, time_reclaim=False) -> ReplayResult:
    return replay(keys, key_off, trace.group, trace.contract, trace.prefix, trace.n_groups,
                  trace.n_prefix, inst, tick=trace.tick, per_request=per_request, time_reclaim=time_reclaim)
