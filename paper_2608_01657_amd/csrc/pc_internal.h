// pc_internal.h -- shapes shared between the host ABI layer and the gfx950
// kernels of libpcreplay.  Not part of the public ABI (include/pc.h is).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pcr {

// ---- per-slot metadata word (uint32) -------------------------------------
//  bits 0-5  owner group        bits 6-7  contract
//  bits 8-9  retention class    bits 10-11 S3-FIFO frequency (0..3)
//  bit 12    S3-FIFO main queue bit 13 resident (cached or being created)
//  bit 14    pinned by the running request
//  bit 15    has a live entry in the free-queue log (stamp valid)
//  bits 16-31  index of the block's entry in the main table (resident
//              blocks; kept through cuckoo displacement)
constexpr uint32_t kOwnerMask = 0x3Fu;
constexpr int kContractShift = 6;
constexpr int kClsShift = 8;
constexpr int kFreqShift = 10;
constexpr uint32_t kQMain = 1u << 12;
constexpr uint32_t kRes = 1u << 13;
constexpr uint32_t kPin = 1u << 14;
constexpr uint32_t kInLog = 1u << 15;
constexpr int kTposShift = 16;
constexpr uint32_t kLowMeta = 0xFFFFu;

constexpr int kProb = 0, kNormal = 1, kReuse = 2;   // Sec. III-A retention classes
constexpr int kLRU = 0, kS3 = 1, kPS = 2, kSQ = 3;
constexpr int kFlagNoSeg = 1, kFlagNoGate = 2;

constexpr uint32_t kEmpty = 0xFFFFFFFFu;   // empty table entry

// Where an instance's state lives.
//   kLayLds     every state array in LDS
//   kLayHybrid  the block keys, the prefix ids of PrefixShield, the request's
//               own keys and S3-FIFO's ghost table in the workspace (HBM);
//               the arrays every probe and every queue scan reads
//               (metadata, stamps, block table, free-queue log, per-request
//               sets, queue counters) in LDS.  A 4096-block instance then
//               needs under 80 KiB of LDS, so two share a CU.
//   kLayWs      every state array in the workspace
constexpr int kLayLds = 0, kLayHybrid = 1, kLayWs = 2;

// LDS that each workgroup of the LDS kernels keeps beside its state: the
// kernel's static exchange area (asserted in the kernel), rounded up so that
// both library builds plan alike.
constexpr int64_t kStaticLdsReserve = 5120;
// Workgroups of the LDS kernels that fit one CU by registers (each asks for
// two waves per SIMD).
constexpr int kMaxWgPerCu = 2;
// LDS of one gfx950 CU (the most one workgroup may take).
constexpr int64_t kGfx950LdsPerCu = 160 * 1024;

constexpr int ceil_log2c(int64_t v) {
    int b = 0;
    while (((int64_t)1 << b) < v) ++b;
    return b;
}

// State-region offsets (bytes from the instance's state base) of a layout,
// in allocation order, 16-byte aligned regions.  Arrays that a layout keeps
// in the workspace (o_key, o_pfx, o_rkeys, o_gtable under kLayHybrid) get
// offset -1; the state of kLayWs is this same region, placed in the
// workspace.  Stamps are 16-bit in LDS layouts (the log ring then has at
// most 2^16 positions) and 32-bit in the workspace layout.
struct StateOffsets {
    int32_t o_key, o_stamp, o_meta, o_table, o_log, o_rkeys, o_rset, o_posslot, o_vlist, o_rcnt, o_res;
    int32_t o_pfx, o_cnt, o_cur, o_fstack, o_gtable;
    int64_t end;
};
constexpr StateOffsets state_offsets(int layout, int policy, int64_t C, int64_t maxn, int32_t nb, int32_t log_log2,
                                     int32_t rs_log2, int32_t gnb_log2, bool ghost) {
    StateOffsets f{-1, -1, -1, -1, -1, -1, -1, -1, -1, -1, -1, -1, -1, -1, -1, -1, 0};
    int64_t so = 0;
    auto take = [&so](int64_t bytes) { const int64_t o = so; so = (so + bytes + 15) / 16 * 16; return (int32_t)o; };
    const bool hyb = layout == kLayHybrid;
    const int64_t mx = maxn < 1 ? 1 : maxn;
    if (!hyb) f.o_key = take(8 * C);
    f.o_stamp = take((layout == kLayWs ? 4 : 2) * C);
    f.o_meta = take(4 * C);
    f.o_table = take(32 * (int64_t)nb);
    f.o_log = take((int64_t)2 << log_log2);
    if (!hyb) f.o_rkeys = take(8 * mx);
    f.o_rset = take((int64_t)4 << rs_log2);
    f.o_posslot = take(2 * mx);
    f.o_vlist = take(2 * mx);
    f.o_rcnt = take((int64_t)4 << (rs_log2 - 3));
    f.o_res = take(4 * 64);
    if (policy == 2 && !hyb) f.o_pfx = take(4 * C);
    if (policy == 2 || policy == 3) {   // per-(group, segment) queues
        f.o_cnt = take(4 * 192);
        f.o_cur = take(4 * 196);
    }
    if (policy == 3) f.o_fstack = take(2 * C);   // StaticQuota: free-slot stack
    if (policy == 1 && ghost && !hyb) f.o_gtable = take((int64_t)32 << gnb_log2);
    f.end = so;
    return f;
}

// Workgroups of the LDS kernels that fit one CU when each holds `state`
// bytes of LDS state (LDS is allocated in 512-byte granules), at most
// kMaxWgPerCu; 0 if none fits.
constexpr int wg_per_cu(int64_t state, int64_t lds_cu) {
    const int64_t per = (state + kStaticLdsReserve + 511) / 512 * 512;
    const int64_t n = per > lds_cu ? 0 : lds_cu / per;
    return (int)(n < kMaxWgPerCu ? n : kMaxWgPerCu);
}

// The state of one instance in one layout.  The main table has an even
// number of 8-entry buckets, between load 2/3 and load 1/2: the largest that
// keeps the most workgroups per CU (more room means fewer cuckoo
// displacements).  The request's duplicate set is at most half full and
// also holds one claim counter per table bucket.  per_cu = 0: the layout
// does not fit a CU (LDS layouts) or is kLayWs.
struct StatePlan {
    int per_cu;
    int32_t nb, rs_log2;
    StateOffsets f;
};
constexpr StatePlan plan_state(int layout, int policy, int64_t C, int64_t maxn, int32_t log_log2, int32_t gnb_log2,
                               bool ghost, int64_t lds_cu) {
    const int64_t mx = maxn < 1 ? 1 : maxn;
    int32_t nb_lo = (int32_t)((C * 3 + 15) / 16);
    nb_lo = nb_lo < 2 ? 2 : nb_lo + (nb_lo & 1);
    int32_t nb_hi = (int32_t)(C / 4);
    nb_hi += nb_hi & 1;
    if (nb_hi < nb_lo) nb_hi = nb_lo;
    auto rs_of = [&](int32_t nb) {
        int r = 6;
        const int a = ceil_log2c(2 * mx), b = ceil_log2c(nb);
        r = a > r ? a : r;
        r = b > r ? b : r;
        return gnb_log2 > r ? gnb_log2 : r;
    };
    StatePlan p{0, nb_lo, rs_of(nb_lo), state_offsets(layout, policy, C, maxn, nb_lo, log_log2, rs_of(nb_lo),
                                                      gnb_log2, ghost)};
    if (layout == kLayWs || log_log2 > 16) return p;
    p.per_cu = wg_per_cu(p.f.end, lds_cu);
    if (p.per_cu == 0) return p;
    for (int32_t nb = nb_hi; nb > nb_lo; nb -= 2) {
        const int32_t rs = rs_of(nb);
        const StateOffsets f = state_offsets(layout, policy, C, maxn, nb, log_log2, rs, gnb_log2, ghost);
        if (wg_per_cu(f.end, lds_cu) == p.per_cu) {
            p.nb = nb;
            p.rs_log2 = rs;
            p.f = f;
            break;
        }
    }
    return p;
}

// The default layout of a 4096-block instance (S3-FIFO small queue 10 %, move
// threshold 1, one contract, eps = 0, no ablation flags) on traces whose
// requests hold at most 512 blocks: every such trace gives the same sizes.
// The host marks an instance with DevInst::fixc = kFixC when its derived
// parameters and offsets equal these exactly (in either LDS layout), and the
// replay kernel then runs a copy compiled with them as constants.
constexpr int32_t kFixC = 4096;
constexpr int32_t kFixLogLog2 = 13;
constexpr int32_t kFixGnbLog2S3 = 10, kFixGrLog2S3 = 14;    // S3-FIFO; other policies: 0, 0
constexpr int32_t kFixScap = 409, kFixGcap = 3687, kFixMoveThr = 1;
constexpr int32_t kFixMaxn = 512;   // the host lays such instances out for requests of 512 blocks
constexpr StatePlan fix_plan(int layout, int policy) {
    return plan_state(layout, policy, kFixC, kFixMaxn, kFixLogLog2, policy == 1 ? kFixGnbLog2S3 : 0, policy == 1,
                      kGfx950LdsPerCu);
}
constexpr uint16_t kNoSlot = 0xFFFF;

// Stats record offsets (int64 words): 64 groups x 17, then instance x 8.
constexpr int kGroupFields = 17;
constexpr int kInstOffset = 64 * kGroupFields;
constexpr int kRecordWords = 64 * kGroupFields + 8;

// Per-instance plan computed on the host.  State offsets are byte offsets
// from the instance's state base: dynamic LDS for kLayLds and kLayHybrid,
// else the workspace region at ws_state.  The ghost ring and the prefix
// bitmaps always live in the workspace, and so do the block keys and prefix
// ids of a hybrid instance (ws_key, ws_pfx).  A hybrid PrefixShield instance
// keeps a slot's key and prefix id together, in one 16-byte record per slot
// (key at byte 0, prefix id at byte 8), so that a lookup reads both, and an
// insert writes both, in one cache line.
struct DevInst {
    int32_t trace, policy, capacity, flags;
    int32_t n_contracts, s_cap, g_cap, move_thr;
    int64_t eps;
    int64_t rho[4], beta[4], invw[4];
    int32_t maxn;          // max probes in one request (<= capacity)
    int32_t nb;            // main table buckets (8 entries each; even)
    int32_t log_log2;      // free-queue log ring entries
    int32_t rs_log2;       // per-request duplicate-detection set entries
    int32_t gnb_log2;      // S3 ghost table buckets
    int32_t gr_log2;       // S3 ghost ring entries
    int32_t layout;        // kLayLds / kLayHybrid / kLayWs
    int32_t state_bytes;   // size of the state region
    int32_t n_prefix_words;
    // state-region offsets (bytes)
    int32_t o_key, o_stamp, o_meta, o_table, o_log, o_posslot, o_rset, o_rkeys, o_vlist;
    int32_t o_pfx, o_gtable, o_rcnt, o_res, o_cnt, o_cur, o_fstack;
    int32_t fixc;          // kFixC: the kernel takes the parameters below as constants
    int32_t pad;
    // workspace offsets (bytes from workspace base)
    int64_t ws_state;      // state region when layout == kLayWs
    int64_t ws_key;        // uint64 [C] block keys (kLayHybrid; PrefixShield: the 16-byte records)
    int64_t ws_pfx;        // PrefixShield's prefix id of slot 0 (kLayHybrid): ws_key + 8, stride 16
    int64_t ws_gtable;     // uint32 [8 << gnb_log2] ghost table (kLayHybrid, S3-FIFO)
    int64_t ws_bits;       // uint32 [2 * n_prefix_words]: referenced, admitted
    int64_t ws_gring;      // uint64 [1 << gr_log2] (S3)
    int64_t per_req_off;   // int32 element offset into the per-request output, or -1
};

struct DevTrace {
    const uint64_t *keys;
    const int64_t *key_off;
    const uint8_t *group;
    const uint8_t *contract;
    const uint32_t *prefix;
    const int64_t *tick;
    int64_t n_req, n_keys, n_prefix;
    int32_t n_groups, max_req_blocks;
};

// Launchers (defined in the .hip files; host-callable).
hipError_t launch_block_offsets(const int32_t *len, int64_t n_req, int64_t *key_off,
                                hipStream_t s);
hipError_t launch_hash(const int32_t *tokens, int64_t n_tokens, const int64_t *tok_off,
                       const int32_t *len, const int32_t *ns, const int64_t *key_off,
                       int64_t n_req, uint64_t *keys, int64_t n_keys, int32_t *status,
                       hipStream_t s);
int32_t replay_static_lds_bytes();
// Raise the dynamic-LDS limit of the LDS-state kernels to lds_bytes (once
// per batch, before its launches).
hipError_t replay_set_lds_limit(int32_t lds_bytes);
// One launch of n_launch instances d_order[0..n_launch) of one layout,
// planned for per_cu instances per CU.
hipError_t launch_replay(const DevInst *d_inst, const DevTrace *d_traces, const int32_t *d_order,
                         int32_t n_launch, int32_t lds_bytes, int layout, int per_cu, uint8_t *ws,
                         int64_t *stats, int32_t *per_req, hipStream_t s);
// the translation unit of the kernels with state in global memory
// (pc_replay_global.hip: hybrid and workspace layouts)
hipError_t replay_hybrid_set_lds_limit(int32_t lds_bytes);
hipError_t launch_replay_global(const DevInst *d_inst, const DevTrace *d_traces, const int32_t *d_order,
                                int32_t n_launch, int32_t lds_bytes, int layout, uint8_t *ws, int64_t *stats,
                                int32_t *per_req, hipStream_t s);

}  // namespace pcr
