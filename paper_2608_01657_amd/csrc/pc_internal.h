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

// The default layout of a 4096-block instance (S3-FIFO small queue 10 %, move
// threshold 1, one contract, eps = 0, no ablation flags) on traces whose
// requests hold at most 512 blocks: every such trace gives these sizes, and
// its state fits LDS.  The host marks an
// instance with DevInst::fixc = kFixC when its derived parameters equal these
// exactly, and the replay kernel then runs a copy compiled with them as
// constants.
constexpr int32_t kFixC = 4096;
constexpr int32_t kFixNbLog2 = 10, kFixRsLog2 = 10, kFixLogLog2 = 13;
constexpr int32_t kFixGnbLog2S3 = 10, kFixGrLog2S3 = 14;    // S3-FIFO; other policies: 0, 0
constexpr int32_t kFixScap = 409, kFixGcap = 3687, kFixMoveThr = 1;
constexpr int32_t kFixMaxn = 512;   // the host lays such instances out for requests of 512 blocks

// State-region offsets of that layout, in the order the host allocates them
// (16-byte aligned regions): equal to the host's for every marked instance.
struct FixOffsets {
    int32_t o_key, o_stamp, o_meta, o_table, o_log, o_rkeys, o_rset, o_posslot, o_vlist, o_rcnt, o_res;
    int32_t o_pfx, o_cnt, o_cur, o_fstack, o_gtable, end;
};
constexpr FixOffsets fix_offsets(int policy) {
    FixOffsets f{};
    int32_t so = 0;
    auto take = [&so](int32_t bytes) { const int32_t o = so; so = (so + bytes + 15) / 16 * 16; return o; };
    const int32_t C = kFixC, mx = kFixMaxn;
    f.o_key = take(8 * C);
    f.o_stamp = take(4 * C);
    f.o_meta = take(4 * C);
    f.o_table = take(32 << kFixNbLog2);
    f.o_log = take(2 << kFixLogLog2);
    f.o_rkeys = take(8 * mx);
    f.o_rset = take(4 << kFixRsLog2);
    f.o_posslot = take(2 * mx);
    f.o_vlist = take(2 * mx);
    f.o_rcnt = take(4 << (kFixRsLog2 - 3));
    f.o_res = take(4 * 64);
    if (policy == kPS) f.o_pfx = take(4 * C);
    if (policy == kPS || policy == kSQ) {
        f.o_cnt = take(4 * 192);
        f.o_cur = take(4 * 196);
    }
    if (policy == kSQ) f.o_fstack = take(2 * C);
    if (policy == kS3) f.o_gtable = take(32 << kFixGnbLog2S3);
    f.end = so;
    return f;
}
constexpr uint16_t kNoSlot = 0xFFFF;

// Stats record offsets (int64 words): 64 groups x 17, then instance x 8.
constexpr int kGroupFields = 17;
constexpr int kInstOffset = 64 * kGroupFields;
constexpr int kRecordWords = 64 * kGroupFields + 8;

// Per-instance plan computed on the host.  State offsets are byte offsets
// from the instance's state base: dynamic LDS when in_lds, else the
// workspace region at ws_state.  The ghost ring and the prefix bitmaps always
// live in the workspace.
struct DevInst {
    int32_t trace, policy, capacity, flags;
    int32_t n_contracts, s_cap, g_cap, move_thr;
    int64_t eps;
    int64_t rho[4], beta[4], invw[4];
    int32_t maxn;          // max probes in one request (<= capacity)
    int32_t nb_log2;       // main table buckets (8 entries each)
    int32_t log_log2;      // free-queue log ring entries
    int32_t rs_log2;       // per-request duplicate-detection set entries
    int32_t gnb_log2;      // S3 ghost table buckets
    int32_t gr_log2;       // S3 ghost ring entries
    int32_t in_lds;        // 1: state in dynamic LDS
    int32_t state_bytes;   // size of the state region
    int32_t n_prefix_words;
    // state-region offsets (bytes)
    int32_t o_key, o_stamp, o_meta, o_table, o_log, o_posslot, o_rset, o_rkeys, o_vlist;
    int32_t o_pfx, o_gtable, o_rcnt, o_res, o_cnt, o_cur, o_fstack;
    int32_t fixc;          // kFixC: the kernel takes the parameters below as constants
    // workspace offsets (bytes from workspace base)
    int64_t ws_state;      // state region when !in_lds
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
hipError_t launch_replay(const DevInst *d_inst, const DevTrace *d_traces, const int32_t *d_order,
                         int32_t n_launch, int32_t lds_bytes, bool in_lds, uint8_t *ws,
                         int64_t *stats, int32_t *per_req, hipStream_t s);

}  // namespace pcr
