"""Device-side driver of the hot path: upload a trace, cut and hash it, replay
a batch of instances.  Only allocation and argument marshalling happen here;
all work runs in libpcreplay's kernels on the current HIP stream."""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np
import torch

from . import (make_instance_desc, phase_counters, make_trace_desc, pc_block_offsets, pc_get_stats, pc_hash_blocks,
               pc_replay_batch, pc_replay_workspace_bytes, stats_to_dicts, PC_STATS_RECORD_BYTES)


@dataclass
class DeviceTrace:
    tokens: torch.Tensor        # int32 [T]
    tok_off: torch.Tensor       # int64 [R]
    length: torch.Tensor        # int32 [R]
    ns: torch.Tensor            # int32 [R] namespace (= accounting group)
    group: torch.Tensor         # uint8 [R]
    contract: torch.Tensor      # uint8 [R]
    prefix: torch.Tensor        # int32 [R] (uint32 values)
    tick: Optional[torch.Tensor]
    n_groups: int
    n_prefix: int
    max_req_blocks: int
    key_off: Optional[torch.Tensor] = None   # int64 [R+1]
    keys: Optional[torch.Tensor] = None      # int64 [K] (uint64 bit patterns)
    status: Optional[torch.Tensor] = None
    n_keys: int = 0

    @property
    def n_req(self) -> int:
        return int(self.length.numel())

    @property
    def n_tokens(self) -> int:
        return int(self.tokens.numel())


def upload(trace, device="cuda") -> DeviceTrace:
    """Copy a tracegen.Trace to device memory."""
    dev = torch.device(device)
    tok = torch.from_numpy(np.ascontiguousarray(trace.tokens, np.int32))
    # allocations from torch's caching allocator are at least 256-byte aligned
    t = DeviceTrace(
        tokens=tok.to(dev),
        tok_off=torch.from_numpy(np.ascontiguousarray(trace.tok_off, np.int64)).to(dev),
        length=torch.from_numpy(np.ascontiguousarray(trace.length, np.int32)).to(dev),
        ns=torch.from_numpy(np.ascontiguousarray(trace.group, np.int32)).to(dev),
        group=torch.from_numpy(np.ascontiguousarray(trace.group, np.uint8)).to(dev),
        contract=torch.from_numpy(np.ascontiguousarray(trace.contract, np.uint8)).to(dev),
        prefix=torch.from_numpy(np.ascontiguousarray(trace.prefix, np.uint32).view(np.int32)).to(dev),
        tick=None if trace.tick is None else torch.from_numpy(np.ascontiguousarray(trace.tick, np.int64)).to(dev),
        n_groups=int(trace.n_groups), n_prefix=int(trace.n_prefix),
        max_req_blocks=int(trace.length.max() // 16) if trace.n_req else 0,
    )
    return t


def alloc_keys(t: DeviceTrace, stream=None):
    """Allocate key_off and keys (sizes come from the host-side lengths)."""
    dev = t.tokens.device
    t.key_off = torch.empty(t.n_req + 1, dtype=torch.int64, device=dev)
    t.status = torch.zeros(1, dtype=torch.int32, device=dev)
    return t


def cut_and_hash(t: DeviceTrace, n_keys: Optional[int] = None, stream=None) -> DeviceTrace:
    """Block offsets then chained keys, on the device."""
    if t.key_off is None:
        alloc_keys(t)
    pc_block_offsets(t.length, t.key_off, stream)
    if t.keys is None:
        if n_keys is None:
            n_keys = int(t.key_off[-1].item())      # one 8-byte read to size the key buffer
        t.n_keys = n_keys
        t.keys = torch.empty(max(n_keys, 1), dtype=torch.int64, device=t.tokens.device)
    t.status.zero_()
    pc_hash_blocks(t.tokens, t.tok_off, t.length, t.ns, t.key_off, t.keys[:t.n_keys] if t.n_keys else t.keys[:0],
                   t.status, stream)
    return t


@dataclass
class KeyDeviceTrace:
    """A replay input given directly as keys (tests craft these)."""
    keys: torch.Tensor
    key_off: torch.Tensor
    group: torch.Tensor
    contract: torch.Tensor
    prefix: torch.Tensor
    tick: Optional[torch.Tensor]
    n_groups: int
    n_prefix: int
    max_req_blocks: int
    n_keys: int


def upload_keys(kt, device="cuda") -> KeyDeviceTrace:
    dev = torch.device(device)
    keys = np.ascontiguousarray(kt.keys, np.uint64).view(np.int64)
    off = np.ascontiguousarray(kt.key_off, np.int64)
    mx = int(np.diff(off).max()) if len(off) > 1 else 0
    return KeyDeviceTrace(
        keys=torch.from_numpy(keys if keys.size else np.zeros(1, np.int64)).to(dev),
        key_off=torch.from_numpy(off).to(dev),
        group=torch.from_numpy(np.ascontiguousarray(kt.group, np.uint8)).to(dev),
        contract=torch.from_numpy(np.ascontiguousarray(kt.contract, np.uint8)).to(dev),
        prefix=torch.from_numpy(np.ascontiguousarray(kt.prefix, np.uint32).view(np.int32)).to(dev),
        tick=None if kt.tick is None else torch.from_numpy(np.ascontiguousarray(kt.tick, np.int64)).to(dev),
        n_groups=int(kt.n_groups), n_prefix=int(kt.n_prefix), max_req_blocks=mx, n_keys=int(keys.size))


def trace_desc(t):
    keys = t.keys[:t.n_keys] if t.n_keys else t.keys[:0]
    return make_trace_desc(keys, t.key_off, t.group, t.contract, t.prefix, t.n_groups, t.n_prefix,
                           t.max_req_blocks, t.tick)


class ReplayBatch:
    """Holds the descriptors, workspace and stats buffer of one batch so the
    same replay can be launched repeatedly (each launch starts from an empty
    cache)."""

    def __init__(self, dtraces: Sequence, instances: Sequence, per_request: bool = False):
        self.dtraces = list(dtraces)
        self.instances = list(instances)
        self.tdesc = [trace_desc(t) for t in self.dtraces]
        self.idesc = [make_instance_desc(i) for i in self.instances]
        dev = self.dtraces[0].key_off.device
        nbytes = pc_replay_workspace_bytes(self.tdesc, self.idesc)
        self.workspace = torch.empty((nbytes + 255) // 256 * 32, dtype=torch.int64, device=dev)
        self.stats = torch.zeros(len(self.instances) * PC_STATS_RECORD_BYTES // 8, dtype=torch.int64, device=dev)
        self.per_request = None
        if per_request:
            n = sum(4 * int(self.dtraces[i.trace].key_off.numel() - 1) for i in self.instances)
            self.per_request = torch.zeros(max(n, 1), dtype=torch.int32, device=dev)

    def launch(self, stream=None):
        pc_replay_batch(self.tdesc, self.idesc, self.workspace, self.stats, self.per_request, stream)

    def results(self, stream=None):
        G, S = pc_get_stats(self.stats, len(self.instances), -1, 64, stream)
        ng = [self.dtraces[i.trace].n_groups for i in self.instances]
        return stats_to_dicts(G, S, ng)

    def phase_counters(self, stream=None) -> List[dict]:
        """Per-instance phase cycles and event counts (phase-counter library
        only; see paper_2608_01657_amd.use_phase_counters)."""
        G, S = pc_get_stats(self.stats, len(self.instances), -1, 64, stream)
        full = stats_to_dicts(G, S, [64] * len(self.instances))
        return [phase_counters(groups) for groups, _, _ in full]

    def per_request_arrays(self) -> List[np.ndarray]:
        assert self.per_request is not None
        host = self.per_request.cpu().numpy()
        out, off = [], 0
        for i in self.instances:
            n = int(self.dtraces[i.trace].key_off.numel() - 1)
            out.append(host[off:off + 4 * n].reshape(n, 4))
            off += 4 * n
        return out


@dataclass
class TraceView:
    """One trace of a TraceSet as the replay reads it: its requests' rows of
    the set's arrays, with key offsets into the set's whole key buffer."""
    keys: torch.Tensor
    key_off: torch.Tensor
    group: torch.Tensor
    contract: torch.Tensor
    prefix: torch.Tensor
    tick: Optional[torch.Tensor]
    n_groups: int
    n_prefix: int
    max_req_blocks: int
    n_keys: int


class TraceSet:
    """Several traces in one set of device buffers, so that block offsets and
    keys of all of them take one pc_block_offsets and one pc_hash_blocks
    call.  Requests keep their own trace's namespace (group) and token view;
    `views` are what ReplayBatch takes, one per trace."""

    def __init__(self, traces: Sequence, device="cuda"):
        dev = torch.device(device)
        tok_base = np.cumsum([0] + [int(tr.tokens.size) for tr in traces[:-1]], dtype=np.int64)
        self.req_base = np.cumsum([0] + [tr.n_req for tr in traces], dtype=np.int64)
        cat = lambda xs, dt: torch.from_numpy(np.ascontiguousarray(np.concatenate(xs), dt)).to(dev)
        any_tick = any(tr.tick is not None for tr in traces)
        self.dt = DeviceTrace(
            tokens=cat([tr.tokens for tr in traces], np.int32),
            tok_off=cat([np.asarray(tr.tok_off, np.int64) + b for tr, b in zip(traces, tok_base)], np.int64),
            length=cat([tr.length for tr in traces], np.int32),
            ns=cat([tr.group for tr in traces], np.int32),
            group=cat([tr.group for tr in traces], np.uint8),
            contract=cat([tr.contract for tr in traces], np.uint8),
            prefix=cat([np.asarray(tr.prefix, np.uint32).view(np.int32) for tr in traces], np.int32),
            # a trace without ticks counts time in requests (tick = request index)
            tick=cat([tr.tick if tr.tick is not None else np.arange(tr.n_req, dtype=np.int64) for tr in traces],
                     np.int64) if any_tick else None,
            n_groups=max(int(tr.n_groups) for tr in traces), n_prefix=max(int(tr.n_prefix) for tr in traces),
            max_req_blocks=max(int(tr.length.max() // 16) if tr.n_req else 0 for tr in traces))
        self.meta = [(int(tr.n_groups), int(tr.n_prefix), int(tr.length.max() // 16) if tr.n_req else 0)
                     for tr in traces]
        self.views: List[TraceView] = []

    def hash(self, stream=None):
        """Offsets and keys of every trace (one call each); views are made on
        the first call."""
        t = self.dt
        cut_and_hash(t, n_keys=t.n_keys if t.keys is not None else None, stream=stream)
        if not self.views:
            for j, (ng, npfx, mx) in enumerate(self.meta):
                r0, r1 = int(self.req_base[j]), int(self.req_base[j + 1])
                self.views.append(TraceView(
                    keys=t.keys[:t.n_keys] if t.n_keys else t.keys[:0], key_off=t.key_off[r0:r1 + 1],
                    group=t.group[r0:r1], contract=t.contract[r0:r1], prefix=t.prefix[r0:r1],
                    tick=None if t.tick is None else t.tick[r0:r1], n_groups=ng, n_prefix=npfx, max_req_blocks=mx,
                    n_keys=t.n_keys))
        return self

    def trace_keys(self, j) -> np.ndarray:
        """Keys of trace j (host copy)."""
        k0, k1 = int(self.dt.key_off[int(self.req_base[j])].item()), int(self.dt.key_off[int(self.req_base[j + 1])].item())
        return self.dt.keys[k0:k1].cpu().numpy().view(np.uint64)

    def trace_key_off(self, j) -> np.ndarray:
        """Key offsets of trace j relative to its own first key (host copy)."""
        o = self.dt.key_off[int(self.req_base[j]):int(self.req_base[j + 1]) + 1].cpu().numpy()
        return o - o[0]
