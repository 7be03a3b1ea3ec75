"""The C ABI without a GPU: the library loads, exports every function that
include/pc.h declares, and rejects malformed calls on the host (before any
device work) with the documented error codes.  No compute call is made."""
import ctypes
import os
import re

import pytest

import paper_2608_01657_amd as P
from paper_2608_01657_amd import tracegen as tg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x10000   # a non-null device address; host validation never dereferences it


def _declared():
    src = open(os.path.join(ROOT, "include", "pc.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^[A-Za-z_][\w \t\*]*?\b(pc_\w+)\s*\(", src, flags=re.M)))


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("pc_hash_blocks", "pc_replay_batch", "pc_get_stats", "pc_block_offsets",
              "pc_replay_workspace_bytes", "pc_last_error"):
        assert n in names


@pytest.mark.parametrize("path", [P.LIB_PATH, P.PHASES_LIB_PATH, P.JITTER_LIB_PATH],
                         ids=["product", "phase_counters", "race_detection"])
def test_library_exports_every_declared_symbol(path):
    """The product library and both test builds of the same sources (phase
    counters, race detection) load and export the whole boundary."""
    lib = ctypes.CDLL(path)
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing
    assert sorted(P.EXPORTS) == sorted(_declared()), "binding and header disagree"


def test_struct_sizes_match_header():
    assert ctypes.sizeof(P.pc_group_stats) == 136
    assert ctypes.sizeof(P.pc_instance_stats) == 64
    assert P.PC_STATS_RECORD_BYTES == 64 * 136 + 64


def _trace(**kw):
    t = P.pc_trace_desc()
    t.d_keys = t.d_key_off = t.d_group = t.d_contract = t.d_prefix = FAKE
    t.n_req, t.n_keys, t.n_prefix, t.n_groups, t.max_req_blocks = 10, 100, 4, 2, 20
    for k, v in kw.items():
        setattr(t, k, v)
    return t


def _inst(**kw):
    i = P.make_instance_desc(tg.Instance(0, tg.POLICY_PREFIXSHIELD, 64))
    for k, v in kw.items():
        setattr(i, k, v)
    return i


def _ws(t, i):
    lib = P.lib()
    return lib.pc_replay_workspace_bytes((P.pc_trace_desc * 1)(t), 1, (P.pc_instance_desc * 1)(i), 1)


def test_workspace_size_of_a_valid_batch():
    assert _ws(_trace(), _inst()) > 0


@pytest.mark.parametrize("field,value,needle", [
    ("capacity", 0, "capacity"),
    ("capacity", P.PC_MAX_CAPACITY + 1, "capacity"),
    ("policy", 4, "policy"),
    ("flags", 4, "flags"),
    ("n_contracts", 0, "n_contracts"),
    ("n_contracts", 5, "n_contracts"),
    ("reserved", 1, "reserved"),
    ("eps_q16", -1, "eps"),
    ("trace", 1, "trace"),
])
def test_instance_validation(field, value, needle):
    assert _ws(_trace(), _inst(**{field: value})) == P.PC_EINVAL
    assert needle in P.pc_last_error()


def test_contract_validation():
    i = _inst()
    i.contract[0].rho_q16 = 0
    assert _ws(_trace(), i) == P.PC_EINVAL and "rho" in P.pc_last_error()
    i = _inst()
    i.contract[0].beta_q16 = -1
    assert _ws(_trace(), i) == P.PC_EINVAL and "beta" in P.pc_last_error()


def test_contract_rate_ratio_limit():
    """Eq. 8 needs a positive decrement 1/W_g; in Q16, 1/w_c = rho_min/rho_c
    is representable down to 2^-16, so rates of one instance may differ by a
    factor 2^16 at most."""
    for slow, fast, ok in [(1, 1 << 16, True), (1, (1 << 16) + 1, False), (1 << 24, 1 << 40, True),
                           (3, 3 << 16, True), (3, (3 << 16) + 3, False)]:
        i = _inst(n_contracts=2)
        i.contract[0].rho_q16, i.contract[1].rho_q16 = slow, fast
        rc = _ws(_trace(), i)
        if ok:
            assert rc > 0, P.pc_last_error()
        else:
            assert rc == P.PC_EINVAL and "2^16" in P.pc_last_error()


@pytest.mark.parametrize("field,value", [
    ("n_groups", 0), ("n_groups", 65), ("n_req", -1), ("d_keys", 0), ("d_key_off", 0),
])
def test_trace_validation(field, value):
    assert _ws(_trace(**{field: value}), _inst()) == P.PC_EINVAL


def test_replay_rejects_small_or_misaligned_workspace():
    lib = P.lib()
    T = (P.pc_trace_desc * 1)(_trace())
    I = (P.pc_instance_desc * 1)(_inst())
    need = lib.pc_replay_workspace_bytes(T, 1, I, 1)
    assert need > 0
    assert lib.pc_replay_batch(T, 1, I, 1, FAKE, need - 1, FAKE, None, None) == P.PC_ENOMEM
    assert lib.pc_replay_batch(T, 1, I, 1, FAKE + 4, need, FAKE, None, None) == P.PC_EINVAL
    assert lib.pc_replay_batch(T, 1, I, 1, None, need, FAKE, None, None) == P.PC_EINVAL


def test_hash_rejects_before_launch():
    lib = P.lib()
    st = ctypes.c_void_p(FAKE)
    # only 16-token blocks are implemented
    assert lib.pc_hash_blocks(FAKE, 64, FAKE, FAKE, FAKE, FAKE, 1, 32, FAKE, 4, st, None) == P.PC_EUNSUPPORTED
    assert lib.pc_hash_blocks(FAKE, 64, FAKE, FAKE, FAKE, FAKE, 1, 16, FAKE, 4, None, None) == P.PC_EINVAL
    # tokens are int32: a buffer off 4-byte alignment is refused
    assert lib.pc_hash_blocks(FAKE + 2, 64, FAKE, FAKE, FAKE, FAKE, 1, 16, FAKE, 4, st, None) == P.PC_EINVAL
    assert lib.pc_hash_blocks(FAKE, -1, FAKE, FAKE, FAKE, FAKE, 1, 16, FAKE, 4, st, None) == P.PC_EINVAL
    assert lib.pc_block_offsets(FAKE, 4, 8, FAKE, None) == P.PC_EUNSUPPORTED


def test_get_stats_rejects_bad_instance_index():
    lib = P.lib()
    G = (P.pc_group_stats * 64)()
    S = (P.pc_instance_stats * 1)()
    assert lib.pc_get_stats(FAKE, 2, 5, G, 64, S, None) == P.PC_EINVAL
    assert lib.pc_get_stats(None, 2, 0, G, 64, S, None) == P.PC_EINVAL


def test_product_path_has_no_fallback(monkeypatch):
    """Without the built library the binding raises; it never computes on
    the host."""
    monkeypatch.setattr(P, "LIB_PATH", os.path.join(ROOT, "no_such_library.so"))
    monkeypatch.setattr(P, "_lib", None)
    with pytest.raises(RuntimeError, match="no CPU fallback"):
        P.pc_last_error()


def test_state_bytes_on_the_host():
    """Per-instance state size: grows with capacity, the S3-FIFO ghost table
    and PrefixShield's per-block prefix ids add to it, and C = 16384 does not
    fit LDS at all (gfx950: 160 KiB per CU)."""
    T = [_trace()]
    I = [_inst(policy=0, capacity=512), _inst(policy=0, capacity=4096), _inst(policy=1, capacity=4096),
         _inst(policy=2, capacity=4096), _inst(policy=2, capacity=16384)]
    b, lay = P.pc_replay_state_bytes(T, I)
    assert b[0] < b[1] < b[3] and b[1] < b[2]
    assert b[1] >= 4096 * (8 + 2 + 4)          # key, stamp, meta per block at least
    assert b[3] - b[1] >= 4096 * 4             # prefix id per block
    assert lay[4] == P.PC_LAYOUT_WS
    lib = P.lib()
    bad = (P.pc_instance_desc * 1)(_inst(capacity=0))
    out_b = (ctypes.c_int64 * 1)()
    out_f = (ctypes.c_int32 * 1)()
    assert lib.pc_replay_state_bytes((P.pc_trace_desc * 1)(_trace()), 1, bad, 1, out_b, out_f) == P.PC_EINVAL


LDS_CU, STATIC_RESERVE = 160 * 1024, 5120


def _lds_part(b, pol, C=4096, ghost_bytes=32 << 10):
    """LDS bytes of a hybrid instance: its block keys (PrefixShield: 16-byte
    key and prefix-id records) and S3-FIFO's ghost table are in the
    workspace."""
    return b - (16 * C if pol == 2 else 8 * C) - (ghost_bytes if pol == 1 else 0)


def test_layout_lets_two_4096_block_instances_share_a_cu():
    """In a batch too large to run at once, the planner keeps a 4096-block
    LRU, S3-FIFO or PrefixShield instance's block keys (and prefix ids,
    ghost table) in the workspace -- the hybrid layout -- which brings its LDS
    state to half of a CU's 160 KiB, so two share a CU; StaticQuota (free-slot
    stack) stays whole in LDS, one per CU.  When the batch fits the 256 CUs
    at once, every instance keeps its whole state in LDS.  Small capacities
    stay in LDS, 16,384 blocks go to the workspace."""
    t = _trace(max_req_blocks=512)
    b, lay = P.pc_replay_state_bytes([t], [_inst(policy=p, capacity=4096) for p in range(4)] * 150)
    assert lay[:4] == [P.PC_LAYOUT_HYBRID, P.PC_LAYOUT_HYBRID, P.PC_LAYOUT_HYBRID, P.PC_LAYOUT_LDS]
    for pol in range(3):
        x = _lds_part(b[pol], pol)
        assert 2 * (((x + STATIC_RESERVE + 511) // 512) * 512) <= LDS_CU, (pol, x)
    assert b[3] + STATIC_RESERVE <= LDS_CU < 2 * (b[3] + STATIC_RESERVE)
    b, lay = P.pc_replay_state_bytes([t], [_inst(policy=p, capacity=4096) for p in range(4)] * 12)
    assert lay == [P.PC_LAYOUT_LDS] * 48
    b, lay = P.pc_replay_state_bytes([_trace(max_req_blocks=1024)], [_inst(policy=p, capacity=1024) for p in range(4)])
    assert lay == [P.PC_LAYOUT_LDS] * 4
    b, lay = P.pc_replay_state_bytes([_trace(max_req_blocks=1024)], [_inst(policy=p, capacity=16384) for p in range(4)])
    assert lay == [P.PC_LAYOUT_WS] * 4


def test_default_4096_layout_is_sized_for_512_block_requests():
    """A 4096-block instance with default S3-FIFO settings is a candidate for
    the kernel's compile-time copy, so the planner lays it out for requests
    of 512 blocks whatever its trace's longest request (the buffers that
    depend on it only grow); other settings keep the trace's own sizing.
    The sizes are those of the layouts' allocation order with the table at
    load 1/2 (all in LDS: 117,504 bytes for LRU, 150,272 for S3-FIFO,
    135,440 for PrefixShield), or at the largest size that keeps two
    instances per CU (hybrid: 109,568 / 142,336 / 142,288 bytes, of which
    76,800 / 76,800 / 76,752 in LDS)."""
    short = _trace(max_req_blocks=100)
    full = _trace(max_req_blocks=512)
    for pol, want in ((0, 117504), (1, 150272), (2, 135440)):
        b, lay = P.pc_replay_state_bytes([short, full], [_inst(policy=pol, capacity=4096, trace=0),
                                                         _inst(policy=pol, capacity=4096, trace=1)])
        assert list(b) == [want, want] and lay == [P.PC_LAYOUT_LDS] * 2
    for pol, want, lds in ((0, 109568, 76800), (1, 142336, 76800), (2, 142288, 76752)):
        b, lay = P.pc_replay_state_bytes([short, full], [_inst(policy=pol, capacity=4096, trace=k % 2)
                                                         for k in range(600)])
        assert set(b) == {want} and set(lay) == {P.PC_LAYOUT_HYBRID} and _lds_part(want, pol) == lds
    # a non-default small queue, or another capacity, keeps the short sizing
    b, _ = P.pc_replay_state_bytes([short, full], [_inst(policy=1, capacity=4096, trace=0, s3_small_permille=250),
                                                   _inst(policy=1, capacity=4096, trace=1, s3_small_permille=250),
                                                   _inst(policy=0, capacity=4095, trace=0),
                                                   _inst(policy=0, capacity=4095, trace=1)])
    assert b[0] < b[1] and b[2] < b[3]


def test_static_entry_rejects_batches_beyond_its_array():
    """The entry point that allocates nothing refuses, on the host, a batch
    whose workspace exceeds the static array (PC_ENOMEM), and a null stats
    pointer (PC_EINVAL)."""
    lib = P.lib()
    t = _trace(n_prefix=1 << 31)            # prefix bitmaps alone need 512 MiB
    T = (P.pc_trace_desc * 1)(t)
    I = (P.pc_instance_desc * 1)(_inst())
    need = lib.pc_replay_workspace_bytes(T, 1, I, 1)
    assert need > P.PC_STATIC_WORKSPACE_BYTES
    assert lib.pc_replay_batch_static(T, 1, I, 1, FAKE, None, None) == P.PC_ENOMEM
    assert "static workspace" in P.pc_last_error()
    T = (P.pc_trace_desc * 1)(_trace())
    assert lib.pc_replay_batch_static(T, 1, I, 1, None, None, None) == P.PC_EINVAL


def test_static_workspace_size_matches_header():
    src = open(os.path.join(ROOT, "include", "pc.h")).read()
    m = re.search(r"#define PC_STATIC_WORKSPACE_BYTES \((\d+)LL << (\d+)\)", src)
    assert m and (int(m.group(1)) << int(m.group(2))) == P.PC_STATIC_WORKSPACE_BYTES
