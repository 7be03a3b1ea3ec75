"""MI355X-native batched replay of a multi-tenant KV prefix cache (PrefixShield).

Thin ctypes binding over libpcreplay.so (C ABI in include/pc.h).  Every
function here only marshals arguments; block cutting, hashing and replay run
in the library's HIP kernels.  PyTorch provides device memory and streams.

The library is loaded from this package directory; if it is missing the
first call raises -- there is no CPU fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpcreplay.so")
# the same library with per-request-phase cycle counters (see phase_counters)
PHASES_LIB_PATH = os.path.join(_HERE, "libpcreplay_phases.so")
# the race-detection build: a pseudo-random per-wavefront delay after every
# replay barrier (results must not change)
JITTER_LIB_PATH = os.path.join(_HERE, "libpcreplay_jitter.so")
PHASE_NAMES = ["request_start", "lookup", "reclamation", "charge", "insert_release", "accounting"]
PHASE_EVENTS = ["evicting_requests", "log_compactions", "s3fifo_scan_batches", "prefixshield_queue_takes"]

PC_OK, PC_EINVAL, PC_ENOMEM, PC_EDEVICE, PC_EUNSUPPORTED, PC_EINTERNAL = 0, -1, -2, -3, -4, -5
PC_BLOCK_TOKENS = 16
PC_MAX_GROUPS, PC_MAX_CONTRACTS, PC_MAX_CAPACITY = 64, 4, 32767
PC_LRU, PC_S3FIFO, PC_PREFIXSHIELD, PC_STATICQUOTA = 0, 1, 2, 3
PC_FLAG_NO_SEGMENTATION, PC_FLAG_NO_DEBT_GATE = 1, 2
PC_STATS_RECORD_BYTES = 64 * 136 + 64
PC_LAYOUT_LDS, PC_LAYOUT_HYBRID, PC_LAYOUT_WS = 0, 1, 2
LAYOUT_NAMES = {PC_LAYOUT_LDS: "lds", PC_LAYOUT_HYBRID: "hybrid", PC_LAYOUT_WS: "workspace"}

GROUP_FIELDS = ["requests", "probes", "hits", "misses", "charged", "evicted_owned",
                "evictions_caused", "promotions", "gated", "orphans", "dups", "truncated",
                "debt_end_q16", "debt_max_q16", "debt_sum_q16", "resident_end", "resident_max"]
INST_FIELDS = ["evictions", "s3_moves", "s3_reinserts", "s3_ghost_hits", "s3_ghost_inserts",
               "resident_end", "resident_max"]


class PCError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"pc error {code}: {msg}")
        self.code = code


class pc_trace_desc(ctypes.Structure):
    _fields_ = [("d_keys", ctypes.c_void_p), ("d_key_off", ctypes.c_void_p),
                ("d_group", ctypes.c_void_p), ("d_contract", ctypes.c_void_p),
                ("d_prefix", ctypes.c_void_p), ("d_tick", ctypes.c_void_p),
                ("n_req", ctypes.c_int64), ("n_keys", ctypes.c_int64), ("n_prefix", ctypes.c_int64),
                ("n_groups", ctypes.c_int32), ("max_req_blocks", ctypes.c_int32)]


class pc_contract(ctypes.Structure):
    _fields_ = [("rho_q16", ctypes.c_int64), ("beta_q16", ctypes.c_int64)]


class pc_instance_desc(ctypes.Structure):
    _fields_ = [("trace", ctypes.c_int32), ("policy", ctypes.c_int32), ("capacity", ctypes.c_int32),
                ("flags", ctypes.c_int32), ("n_contracts", ctypes.c_int32),
                ("s3_small_permille", ctypes.c_int32), ("s3_move_threshold", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("eps_q16", ctypes.c_int64),
                ("contract", pc_contract * 4)]


class pc_group_stats(ctypes.Structure):
    _fields_ = [(f, ctypes.c_uint64) for f in GROUP_FIELDS[:12]] + \
               [(f, ctypes.c_int64) for f in GROUP_FIELDS[12:]]


class pc_instance_stats(ctypes.Structure):
    _fields_ = [(f, ctypes.c_uint64) for f in INST_FIELDS[:5]] + \
               [("resident_end", ctypes.c_int64), ("resident_max", ctypes.c_int64),
                ("status", ctypes.c_int32), ("reserved", ctypes.c_int32)]


EXPORTS = ["pc_last_error", "pc_block_offsets", "pc_hash_blocks", "pc_replay_workspace_bytes",
           "pc_replay_state_bytes", "pc_replay_batch", "pc_replay_batch_static", "pc_get_stats"]
PC_STATIC_WORKSPACE_BYTES = 64 << 20

_lib = None


def use_phase_counters(on: bool = True):
    """Select the phase-counter library (before the first call into the
    library).  Its stats record of group 63 holds the counters instead of
    group 63's own (instances must have at most 63 groups)."""
    global LIB_PATH
    if _lib is not None:
        raise RuntimeError("the library is already loaded")
    LIB_PATH = PHASES_LIB_PATH if on else os.path.join(_HERE, "libpcreplay.so")


def use_jitter_build():
    """Select the race-detection library (before the first call into the
    library): same entry points and results, with shifted wavefront timing
    inside every replay workgroup."""
    global LIB_PATH
    if _lib is not None:
        raise RuntimeError("the library is already loaded")
    LIB_PATH = JITTER_LIB_PATH


def phase_counters(groups) -> dict:
    """Decode the counters from an instance's group records (phase build)."""
    g = groups[63]
    vals = [g[f] for f in GROUP_FIELDS]
    out = {f"cycles_{n}": int(vals[i]) for i, n in enumerate(PHASE_NAMES)}
    out["span_cycles"] = int(vals[6])          # the instance's span on the shader clock
    out["span_ticks_100mhz"] = int(vals[7])    # and on the 100 MHz real-time clock
    out.update({n: int(vals[8 + i]) for i, n in enumerate(PHASE_EVENTS)})
    return out


def lib():
    """Load libpcreplay.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2608_01657_amd.build` (no CPU fallback exists)")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        L.pc_last_error.restype = ctypes.c_char_p
        L.pc_last_error.argtypes = []
        L.pc_block_offsets.restype = i32
        L.pc_block_offsets.argtypes = [P, i64, i32, P, P]
        L.pc_hash_blocks.restype = i32
        L.pc_hash_blocks.argtypes = [P, i64, P, P, P, P, i64, i32, P, i64, P, P]
        L.pc_replay_workspace_bytes.restype = i64
        L.pc_replay_workspace_bytes.argtypes = [ctypes.POINTER(pc_trace_desc), i32,
                                                ctypes.POINTER(pc_instance_desc), i32]
        L.pc_replay_state_bytes.restype = i32
        L.pc_replay_state_bytes.argtypes = [ctypes.POINTER(pc_trace_desc), i32, ctypes.POINTER(pc_instance_desc),
                                            i32, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int32)]
        L.pc_replay_batch.restype = i32
        L.pc_replay_batch.argtypes = [ctypes.POINTER(pc_trace_desc), i32, ctypes.POINTER(pc_instance_desc),
                                      i32, P, i64, P, P, P]
        L.pc_replay_batch_static.restype = i32
        L.pc_replay_batch_static.argtypes = [ctypes.POINTER(pc_trace_desc), i32, ctypes.POINTER(pc_instance_desc),
                                             i32, P, P, P]
        L.pc_get_stats.restype = i32
        L.pc_get_stats.argtypes = [P, i32, i32, ctypes.POINTER(pc_group_stats), i32,
                                   ctypes.POINTER(pc_instance_stats), P]
        _lib = L
    return _lib


def _check(rc: int):
    if rc != PC_OK:
        raise PCError(rc, lib().pc_last_error().decode())
    return rc


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


# --------------------------------------------------------------------------
# The C ABI, one function each
# --------------------------------------------------------------------------

def pc_last_error() -> str:
    return lib().pc_last_error().decode()


def pc_block_offsets(req_len, key_off, stream=None):
    """key_off[r] = sum_{i<r} floor(req_len[i]/16), r = 0..n_req (device tensors)."""
    n = int(req_len.numel())
    assert key_off.numel() == n + 1
    return _check(lib().pc_block_offsets(_ptr(req_len), n, PC_BLOCK_TOKENS, _ptr(key_off), _stream(stream)))


def pc_hash_blocks(tokens, req_tok_off, req_len, req_ns, key_off, keys, status, stream=None):
    """Chained 64-bit keys of every full 16-token block (device tensors)."""
    return _check(lib().pc_hash_blocks(_ptr(tokens), int(tokens.numel()), _ptr(req_tok_off), _ptr(req_len),
                                       _ptr(req_ns), _ptr(key_off), int(req_len.numel()), PC_BLOCK_TOKENS,
                                       _ptr(keys), int(keys.numel()), _ptr(status), _stream(stream)))


def _descs(traces: Sequence[pc_trace_desc], instances: Sequence[pc_instance_desc]):
    T = (pc_trace_desc * max(1, len(traces)))(*traces)
    I = (pc_instance_desc * max(1, len(instances)))(*instances)
    return T, I


def pc_replay_workspace_bytes(traces: Sequence[pc_trace_desc], instances: Sequence[pc_instance_desc]) -> int:
    T, I = _descs(traces, instances)
    v = lib().pc_replay_workspace_bytes(T, len(traces), I, len(instances))
    if v < 0:
        raise PCError(int(v), pc_last_error())
    return int(v)


def pc_replay_state_bytes(traces: Sequence[pc_trace_desc], instances: Sequence[pc_instance_desc]):
    """Per-instance state bytes and layout (PC_LAYOUT_LDS / _HYBRID / _WS)."""
    T, I = _descs(traces, instances)
    n = len(instances)
    b = (ctypes.c_int64 * max(n, 1))()
    f = (ctypes.c_int32 * max(n, 1))()
    _check(lib().pc_replay_state_bytes(T, len(traces), I, n, b, f))
    return [int(b[i]) for i in range(n)], [int(f[i]) for i in range(n)]


def pc_replay_batch(traces, instances, workspace, stats, per_request=None, stream=None):
    T, I = _descs(traces, instances)
    return _check(lib().pc_replay_batch(T, len(traces), I, len(instances), _ptr(workspace),
                                        int(workspace.numel() * workspace.element_size()), _ptr(stats),
                                        _ptr(per_request), _stream(stream)))


def pc_replay_batch_static(traces, instances, stats, per_request=None, stream=None):
    """pc_replay_batch on the library's static workspace (allocates nothing)."""
    T, I = _descs(traces, instances)
    return _check(lib().pc_replay_batch_static(T, len(traces), I, len(instances), _ptr(stats),
                                               _ptr(per_request), _stream(stream)))


def pc_get_stats(stats, n_inst: int, instance: int = -1, max_groups: int = 64, stream=None):
    """Returns (groups [count, max_groups] structs, instances [count] structs)."""
    count = n_inst if instance < 0 else 1
    G = (pc_group_stats * max(1, count * max_groups))()
    S = (pc_instance_stats * max(1, count))()
    _check(lib().pc_get_stats(_ptr(stats), n_inst, instance, G, max_groups, S, _stream(stream)))
    return G, S


# --------------------------------------------------------------------------
# Descriptor builders (host structs pointing at device tensors)
# --------------------------------------------------------------------------

def make_trace_desc(keys, key_off, group, contract, prefix, n_groups, n_prefix, max_req_blocks,
                    tick=None) -> pc_trace_desc:
    return pc_trace_desc(_ptr(keys), _ptr(key_off), _ptr(group), _ptr(contract), _ptr(prefix), _ptr(tick),
                         int(group.numel()), int(keys.numel()), int(n_prefix), int(n_groups),
                         int(max_req_blocks))


def make_instance_desc(inst) -> pc_instance_desc:
    """`inst` has the attributes of tracegen.Instance."""
    d = pc_instance_desc()
    d.trace, d.policy, d.capacity, d.flags = inst.trace, inst.policy, inst.capacity, inst.flags
    d.n_contracts = len(inst.contracts)
    d.s3_small_permille, d.s3_move_threshold, d.reserved = inst.s3_small_permille, inst.s3_move_threshold, 0
    d.eps_q16 = inst.eps_q16
    for i, (rho, beta) in enumerate(inst.contracts):
        d.contract[i].rho_q16, d.contract[i].beta_q16 = rho, beta
    return d


def stats_to_dicts(G, S, n_groups_per_inst: List[int], max_groups: int = 64):
    out = []
    for i, ng in enumerate(n_groups_per_inst):
        groups = []
        for g in range(ng):
            st = G[i * max_groups + g]
            groups.append({f: int(getattr(st, f)) for f in GROUP_FIELDS})
        s = S[i]
        out.append((groups, {f: int(getattr(s, f)) for f in INST_FIELDS}, int(s.status)))
    return out
