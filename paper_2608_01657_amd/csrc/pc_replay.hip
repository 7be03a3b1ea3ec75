// pc_replay.hip -- batched replay of multi-tenant prefix-cache instances on
// gfx950: one workgroup of 4 wavefronts (one per SIMD) per instance.
//
// Per request (Alg. 1 hooks and Alg. 2 reclamation of the paper):
//   OnRequest           prior-reference bit of (g,p), recorded
//   lookup              longest leading run of resident blocks; later
//                       repeats of a key inside the request are misses
//   pin + OnTouch       S3-FIFO frequency, or the debt-gated promotion of
//                       Eq. 4 using the debt before this request's charge
//   reclamation         truly free slots first, then e victims: LRU order,
//                       S3-FIFO small/main/ghost, PrefixShield's
//                       projected-debt argmax (Eqs. 5-8) with the
//                       reuse-segmented order inside the group (Eq. 9), or
//                       StaticQuota's own partition of floor(C/G) blocks
//   OnCacheFullBlocks   charge n_r (Eqs. 1-2), initial class, admission
//   insert + release    new blocks take the victims' slots; every block of
//                       the request returns to the free queue deepest first
//   accounting          raw debt D_g (Eq. 3) and occupancy of every group
//
// Work split: per-block work (keys, log entries, new blocks) is spread over
// the 256 threads; everything that is one value per instance (queue
// pointers, counters) or one value per accounting group (balances, debts,
// the argmax of Eq. 7: lane x = group x) is computed redundantly by all four
// wavefronts from the same inputs, so it never has to be exchanged.  The only
// exchange is a block-wide ballot (each wave's 64-bit ballot through LDS and
// one barrier), which gives every thread block-wide counts and ranks.
//
// State of one instance (capacity C, largest request n_max):
//   key[C] u64, stamp[C], meta[C] u32      -- one slot per cached block
//   table[8*NB] u32  2-choice bucketized hash, entry = tag16 | slot16
//   log[R] u16       free-queue log: the slot of each appended entry; an
//                    entry at absolute position q is live iff its slot has
//                    the in-log bit and stamp == q (stamps are 16-bit when
//                    the state is in LDS: R <= 2^16, and every position a
//                    scan compares lies in the live window of R)
//   rkeys, rset, posslot, vlist   per-request keys, duplicate set,
//                    position -> slot, victims' slots
//   pfx[C] (PrefixShield), ghost table (S3-FIFO), per-group counters
// Three layouts, the same code instantiated for each: everything in
// dynamic LDS; the hybrid one, with the block keys, prefix ids and request
// keys in the workspace (HBM) and the rest in LDS, so that two 4096-block
// instances share a CU; or everything in the workspace.  The ghost ring
// (keys of S3-FIFO's ghost entries) and the prefix bitmaps stay in HBM.
//
// Victims of one request are chosen in bulk: LRU takes the first e live log
// entries, 256 per step; PrefixShield turns the per-victim argmax of Eq. 7
// into runs (the winner keeps winning while its projected debt stays above
// every other candidate's) and drains each run from the group's per-segment
// cursor; S3-FIFO processes queue heads 256 at a time and cuts each batch
// where the one-at-a-time rule would switch queues.  Each shortcut
// reproduces the one-victim-at-a-time definition exactly.
#include <cstddef>
#include <type_traits>

#include "pc_internal.h"

namespace pcr {
namespace {

#define DEV __device__ __forceinline__

constexpr int kW = 4;              // wavefronts per instance
constexpr int kB = 64 * kW;        // threads per instance
constexpr int64_t kScale = 65536;
constexpr uint16_t kNewMark = 0xFFFE;      // posslot: new block, slot not yet assigned
constexpr int32_t kErrInternal = -5;

DEV uint64_t ballot(bool p) { return __ballot(p); }
DEV int popc(uint64_t m) { return __popcll(m); }
DEV int mbcnt(uint64_t m) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}
DEV int first_bit(uint64_t m) { return __ffsll((unsigned long long)m) - 1; }   // m != 0
DEV uint32_t rfl(uint32_t v) { return (uint32_t)__builtin_amdgcn_readfirstlane((int)v); }
DEV uint64_t rfl64(uint64_t v) { return ((uint64_t)rfl((uint32_t)(v >> 32)) << 32) | rfl((uint32_t)v); }
DEV uint32_t bcast32(uint32_t v, int l) { return (uint32_t)__builtin_amdgcn_readlane((int)v, l); }
DEV int64_t bcast64(int64_t v, int l) {
    uint32_t lo = bcast32((uint32_t)(uint64_t)v, l);
    uint32_t hi = bcast32((uint32_t)((uint64_t)v >> 32), l);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}
// Wavefront reductions in DPP steps (no LDS): an inclusive scan under the
// operation -- within each row of 16 lanes (row_shr 1, 2, 4, 8), then rows 1
// and 3 take the last lane of the row before them (row_bcast:15), then rows 2
// and 3 take lane 31 (row_bcast:31) -- leaves the result in lane 63.  A lane
// with no source lane keeps `old`.  Called with every lane active.
template <int kCtrl, int kRowMask>
DEV uint32_t dpp32(uint32_t old, uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, kCtrl, kRowMask, 0xF, false);
}
template <int kCtrl, int kRowMask>
DEV int64_t dpp64(int64_t old, int64_t v) {
    const uint32_t lo = dpp32<kCtrl, kRowMask>((uint32_t)(uint64_t)old, (uint32_t)(uint64_t)v);
    const uint32_t hi = dpp32<kCtrl, kRowMask>((uint32_t)((uint64_t)old >> 32), (uint32_t)((uint64_t)v >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}
#define PC_WAVE_SCAN(v, OP, DPP, IDENT)                   \
    do {                                                  \
        v = OP(v, DPP<0x111, 0xF>(IDENT, v));             \
        v = OP(v, DPP<0x112, 0xF>(IDENT, v));             \
        v = OP(v, DPP<0x114, 0xF>(IDENT, v));             \
        v = OP(v, DPP<0x118, 0xF>(IDENT, v));             \
        v = OP(v, DPP<0x142, 0xA>(IDENT, v));             \
        v = OP(v, DPP<0x143, 0xC>(IDENT, v));             \
    } while (0)
DEV int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }
DEV uint32_t min32(uint32_t a, uint32_t b) { return a < b ? a : b; }
DEV uint32_t add32(uint32_t a, uint32_t b) { return a + b; }
DEV int64_t wave_max64(int64_t v) {
    const int64_t own = v;
    PC_WAVE_SCAN(v, max64, dpp64, own);
    return bcast64(v, 63);
}
DEV uint32_t wave_min32(uint32_t v) {
    const uint32_t own = v;
    PC_WAVE_SCAN(v, min32, dpp32, own);
    return bcast32(v, 63);
}
DEV uint32_t wave_sum32(uint32_t v) {
    PC_WAVE_SCAN(v, add32, dpp32, 0u);
    return bcast32(v, 63);
}
// position of the k-th (0-based) set bit of m (k < popc(m)), in one
// wavefront step: lane l holds bit l, and the answer is the lane whose bit is
// set with exactly k set bits below it.  Called with every lane active, with
// m and k the same in every lane.
DEV int nth_bit(uint64_t m, int k) {
    const bool hit = ((m >> __lane_id()) & 1ull) != 0 && mbcnt(m) == k;
    return first_bit(ballot(hit));
}
// floor(a / b) for 0 < b < 2^63: below 2^53 a double-precision estimate and
// an exact integer correction (the estimate is off by at most one or two);
// above, plain shift-and-subtract.  b = 0 returns 0 (callers never pass it).
DEV uint64_t udiv64(uint64_t a, uint64_t b) {
    if (a < b || b == 0) return 0;
    if (a >> 53) {
        uint64_t q = 0, r = 0;
        for (int i = 63; i >= 0; --i) {
            r = (r << 1) | ((a >> i) & 1u);
            if (r >= b) { r -= b; q |= 1ull << i; }
        }
        return q;
    }
    uint64_t q = (uint64_t)((double)a / (double)b);
    int64_t r = (int64_t)(a - q * b);
    while (r < 0) { --q; r += (int64_t)b; }
    while ((uint64_t)r >= b) { ++q; r -= (int64_t)b; }
    return q;
}
// Keep a wave-uniform value in a VGPR (it is only used in per-lane
// arithmetic) so it does not occupy scalar registers.
template <typename T>
DEV T in_vgpr(T x) {
    asm volatile("" : "+v"(x));
    return x;
}

// Global-memory pointers.  Trace arrays reach the kernel through a
// descriptor, so without the address space the compiler would use flat loads,
// which also count against the LDS wait counter: every LDS wait would then
// wait for the in-flight HBM prefetches.
#define GLOBAL __attribute__((address_space(1)))
template <typename T>
DEV const GLOBAL T *gptr(const T *p) { return (const GLOBAL T *)p; }
template <typename T>
DEV GLOBAL T *gptr_rw(T *p) { return (GLOBAL T *)p; }
// Hybrid PrefixShield's per-slot record of block key and prefix id.
struct alignas(16) KeyRec {
    uint64_t key;
    uint32_t pfx, pad;
};
// One field of every record of a global array of records, read and written
// as an array: element i is p[i * kStride] (in units of T).
template <typename T, int kStride>
struct StridedGlobal {
    GLOBAL T *p;
    DEV GLOBAL T &operator[](uint32_t i) const { return p[(uint64_t)i * kStride]; }
};

// Block-wide ballot result: one 64-bit mask per wavefront.
struct BMask {
    uint64_t w[kW];
    DEV int count() const {
        int c = 0;
#pragma unroll
        for (int i = 0; i < kW; ++i) c += popc(w[i]);
        return c;
    }
    // set bits before thread (wid, lane)
    DEV int rank(int wid) const {
        int c = 0;
#pragma unroll
        for (int i = 0; i < kW; ++i) c += i < wid ? popc(w[i]) : 0;
        uint64_t mine = 0;
#pragma unroll
        for (int i = 0; i < kW; ++i) mine = i == wid ? w[i] : mine;
        return c + mbcnt(mine);
    }
    DEV bool any() const {
        uint64_t a = 0;
#pragma unroll
        for (int i = 0; i < kW; ++i) a |= w[i];
        return a != 0;
    }
    // thread index (wid*64+lane) of the first set bit, or kB.  Selects, not
    // branches: the masks are wave-uniform, and a branch per word costs more
    // than the word's find-first-set.
    DEV int first() const {
        int r = kB;
#pragma unroll
        for (int i = kW - 1; i >= 0; --i) r = w[i] ? 64 * i + first_bit(w[i]) : r;
        return r;
    }
    // thread index of the k-th set bit (k < count()), or kB: the word that
    // holds it is picked by running popcounts, then one lane-parallel step
    // finds the bit.  Called with every lane active.
    DEV int nth(int k) const {
        uint64_t sel = 0;
        int off = kB;
        bool done = false;
#pragma unroll
        for (int i = 0; i < kW; ++i) {
            const int c = popc(w[i]);
            const bool take = !done && k < c;
            sel = take ? w[i] : sel;
            off = take ? 64 * i : off;
            k = (!done && !take) ? k - c : k;
            done = done || take;
        }
        const int b = nth_bit(sel, k);
        return done ? off + b : kB;
    }
    // keep only bits of threads below index t
    DEV BMask below(int t) const {
        BMask r;
#pragma unroll
        for (int i = 0; i < kW; ++i) {
            const int lo = t - 64 * i;
            r.w[i] = lo >= 64 ? w[i] : (lo <= 0 ? 0ull : (w[i] & ((1ull << lo) - 1)));
        }
        return r;
    }
    // keep only bits of threads at index t or above
    DEV BMask from(int t) const {
        BMask r;
#pragma unroll
        for (int i = 0; i < kW; ++i) {
            const int lo = t - 64 * i;
            r.w[i] = lo <= 0 ? w[i] : (lo >= 64 ? 0ull : (w[i] & ~((1ull << lo) - 1)));
        }
        return r;
    }
    DEV BMask andnot(const BMask &o) const {
        BMask r;
#pragma unroll
        for (int i = 0; i < kW; ++i) r.w[i] = w[i] & ~o.w[i];
        return r;
    }
    DEV BMask operator|(const BMask &o) const {
        BMask r;
#pragma unroll
        for (int i = 0; i < kW; ++i) r.w[i] = w[i] | o.w[i];
        return r;
    }
};

// Per-workgroup exchange area (static LDS, both variants).
struct Coll {
    unsigned long long m[2][8][kW];   // block ballots, double-buffered
    uint32_t novf;                    // pending cuckoo displacements
    uint32_t qf;                      // prior-reference / admitted bits of the request (read with novf)
    uint32_t nghost;                  // ghost hits among the request's new blocks
    int32_t kerr;                     // displacement failure
    uint32_t pad;
    uint64_t kkey[kB];                // displacement scratch: keys
    uint32_t kval[kB];                // displacement scratch: entries
    uint32_t kmain[kB];               // 1 = main table, 0 = ghost table
#ifdef PC_PROFILE
    uint64_t prof[8];                 // cycles per request phase (thread 0)
    uint64_t prof_last;
    uint64_t prof_t0, prof_rt0;       // shader clock and 100 MHz real-time clock at the instance's start
    uint64_t pcnt[8];                 // event counts (thread 0)
#endif
};
static_assert(offsetof(Coll, qf) == offsetof(Coll, novf) + 4 && offsetof(Coll, novf) % 8 == 0,
              "novf and qf are read together as one 64-bit word");
static_assert(sizeof(Coll) <= kStaticLdsReserve, "the host plans LDS with this much static LDS per workgroup");

// Key -> two table buckets out of nb (even, any size: the bucket is the
// high word of a 32x32-bit product), a 16-bit tag from the other half of
// the first mix (never 0xFFFF, so empty entries never match a tag), two
// duplicate-set buckets.  Keys are usually hash outputs already, but the
// ABI accepts any uint64, so mix with 32-bit ops.
struct TH {
    uint32_t b1, b2, tag, r1, r2;
};
DEV TH thash(uint64_t k, uint32_t nb, uint32_t rbmask) {
    const uint32_t lo = (uint32_t)k, hi = (uint32_t)(k >> 32);
    uint32_t x = lo * 0x85EBCA6Bu ^ hi;
    x ^= x >> 15;
    x *= 0x2C1B3C6Du;
    x ^= x >> 13;
    uint32_t y = (hi * 0xC2B2AE35u) ^ (lo + 0x27D4EB2Fu);
    y ^= y >> 16;
    y *= 0x9E3779B1u;
    y ^= x >> 7;
    TH h;
    h.b1 = __umulhi(x, nb);
    h.b2 = __umulhi(y, nb);
    if (h.b2 == h.b1) h.b2 = h.b1 ^ 1u;
    const uint32_t t = x & 0xFFFFu;
    h.tag = t == 0xFFFFu ? 0xFFFEu : t;
    h.r1 = y & rbmask;
    h.r2 = (y >> 13) & rbmask;
    if (h.r2 == h.r1) h.r2 = h.r1 ^ 1u;
    return h;
}

DEV uint32_t owner_of(uint32_t mt) { return mt & kOwnerMask; }
DEV uint32_t contract_of(uint32_t mt) { return (mt >> kContractShift) & 3u; }
DEV uint32_t cls_of(uint32_t mt) { return (mt >> kClsShift) & 3u; }
DEV uint32_t freq_of(uint32_t mt) { return (mt >> kFreqShift) & 3u; }

// Optional per-phase cycle accounting (the phase-counter build, -DPC_PROFILE).
// Thread 0 reads the shader clock at each phase boundary of a request:
//   0 request start (descriptor checks, OnRequest)   1 lookup (+ prefetch)
//   2 reclamation   3 charge   4 insert + release   5 accounting
// and counts: 0 requests that evicted, 1 log compactions, 2 S3-FIFO scan
// batches, 3 PrefixShield queue takes.  The instance's whole span is also
// taken on the shader clock and on the 100 MHz real-time clock, which gives
// the shader clock's rate.  The totals replace the record of group 63 in the
// stats.  The counters cost a few percent; nothing of the
// replay itself is skipped or changed.
// PROF_MARK(i) adds the cycles since the previous mark to counter i.
#ifdef PC_PROFILE
#define PROF_MARK(i)                                              \
    do {                                                          \
        const uint64_t prof_now = __builtin_amdgcn_s_memtime();   \
        if (tid == 0) {                                           \
            X.prof[i] += prof_now - X.prof_last;                  \
            X.prof_last = prof_now;                               \
        }                                                         \
    } while (0)
#define PROF_COUNT(i, v) do { if (tid == 0) X.pcnt[i] += (uint64_t)(v); } while (0)
#else
#define PROF_MARK(i) do { } while (0)
#define PROF_COUNT(i, v) do { } while (0)
#endif

// Descriptor of one request (loaded one request ahead).
// Fields are kept as loaded (no arithmetic on them until the request runs,
// so that issuing the loads never waits for them).
struct Req {
    uint8_t g, c;
    uint32_t p;
    int64_t t, ko, kend;
    DEV int64_t nfull() const { return kend - ko; }
};

// Parameters derived from an instance's capacity and S3-FIFO settings.
// kFix = 0: read from its descriptor.  kFix = kFixC: the default 4096-block
// layout in layout kLay, by the host's own planning function evaluated at
// compile time, so that they fold into the instructions instead of holding
// scalar registers.
template <int kLay, int kPol, int kFix>
struct Params {
    int C;
    uint32_t nb, rsmask, rbmask, lmask, R, gnb, gnbmask, grmask;
    int32_t s_cap, g_cap, move_thr;
    uint32_t gne, gspan;      // ghost table entries; sweep span (ring - g_cap - 256)
    uint64_t gsrate;          // ceil(gne * 2^16 / gspan): entries swept per insertion, Q16
    int flags, K, nseg;
    int64_t eps;
    DEV void set_params(const DevInst &I) {
        flags = I.flags;
        K = I.n_contracts;
        nseg = (kPol == kPS && !(flags & kFlagNoSeg)) ? 3 : 1;
        eps = I.eps;
        C = I.capacity;
        nb = (uint32_t)I.nb;
        rsmask = (1u << I.rs_log2) - 1u;
        rbmask = rsmask >> 3;
        R = 1u << I.log_log2;
        lmask = R - 1u;
        gnb = 1u << I.gnb_log2;
        gnbmask = gnb - 1u;
        grmask = (1u << I.gr_log2) - 1u;
        gne = 8u << I.gnb_log2;
        gspan = (grmask + 1u) - (uint32_t)I.g_cap - (uint32_t)kB;
        gsrate = I.g_cap > 0 ? (((uint64_t)gne << 16) + gspan - 1) / gspan : 0;
        s_cap = I.s_cap;
        g_cap = I.g_cap;
        move_thr = I.move_thr;
    }
};
template <int kLay, int kPol>
struct Params<kLay, kPol, kFixC> {
    static constexpr int32_t kGnb = kPol == kS3 ? kFixGnbLog2S3 : 0, kGr = kPol == kS3 ? kFixGrLog2S3 : 0;
    static constexpr StatePlan kPlan = fix_plan(kLay, kPol);
    static constexpr int C = kFixC;
    static constexpr uint32_t nb = (uint32_t)kPlan.nb, rsmask = (1u << kPlan.rs_log2) - 1u;
    static constexpr uint32_t rbmask = rsmask >> 3, R = 1u << kFixLogLog2, lmask = R - 1u;
    static constexpr uint32_t gnb = 1u << kGnb, gnbmask = gnb - 1u, grmask = (1u << kGr) - 1u;
    static constexpr int32_t s_cap = kFixScap, g_cap = kFixGcap, move_thr = kFixMoveThr;
    static constexpr uint32_t gne = 8u << kGnb, gspan = (grmask + 1u) - (uint32_t)g_cap - (uint32_t)kB;
    static constexpr uint64_t gsrate = g_cap > 0 ? (((uint64_t)gne << 16) + gspan - 1) / gspan : 0;
    // one contract, eps = 0, no ablation flags
    static constexpr int flags = 0, K = 1, nseg = kPol == kPS ? 3 : 1;
    static constexpr int64_t eps = 0;
    DEV void set_params(const DevInst &) {}
};

// kPol is the instance's policy: each policy gets its own specialized copy
// of the request loop (no runtime policy tests, fewer live registers).
// kLay is where the state lives (kLayLds, kLayHybrid, kLayWs).
template <int kLay, int kPol, int kFix = 0>
struct Replayer : Params<kLay, kPol, kFix> {
    using Pm = Params<kLay, kPol, kFix>;
    // barriers fence LDS only while the state (all but the hybrid layout's
    // keys and prefix ids) is in LDS
    static constexpr bool kLds = kLay != kLayWs;
    static constexpr bool kHyb = kLay == kLayHybrid;
    // hybrid PrefixShield: a slot's key and prefix id share one 16-byte
    // record in global memory (key at byte 0, prefix id at byte 8)
    static constexpr bool kPack = kHyb && kPol == kPS;
    using KeyPtr = typename std::conditional<
        kPack, StridedGlobal<uint64_t, 2>,
        typename std::conditional<kHyb, GLOBAL uint64_t *, uint64_t *>::type>::type;
    using PfxPtr = typename std::conditional<
        kPack, StridedGlobal<uint32_t, 4>,
        typename std::conditional<kHyb, GLOBAL uint32_t *, uint32_t *>::type>::type;
    using GtPtr = typename std::conditional<kHyb, GLOBAL uint32_t *, uint32_t *>::type;   // S3-FIFO ghost table
    using StampT = typename std::conditional<kLay == kLayWs, uint32_t, uint16_t>::type;
    using Pm::C;
    using Pm::nb;
    using Pm::rsmask;
    using Pm::rbmask;
    using Pm::lmask;
    using Pm::R;
    using Pm::gnb;
    using Pm::gnbmask;
    using Pm::grmask;
    using Pm::s_cap;
    using Pm::g_cap;
    using Pm::move_thr;
    using Pm::gne;
    using Pm::gspan;
    using Pm::gsrate;
    using Pm::flags;
    using Pm::K;
    using Pm::nseg;
    using Pm::eps;
    static constexpr int policy = kPol;
    // per-(group, segment) free queues: live counts and log cursors
    static constexpr bool kQueues = kPol == kPS || kPol == kSQ;
    Coll &X;
    const int tid, wid, lane;
    int cb;                   // ballot buffer in use
    // ---------------- configuration (uniform)
    const DevInst &I;
    const DevTrace &T;
    int G;
    int room;                 // most blocks one request may hold: C, or the StaticQuota partition
    int64_t rho[4], beta[4], invw[4];   // kept in VGPRs
    // ---------------- arrays
    KeyPtr key;
    PfxPtr pfx;
    const GLOBAL KeyRec *krec;   // the 16-byte records themselves (kPack)
    uint64_t *rkeys;          // (not in the hybrid layout: the trace's keys are read instead)
    StampT *stamp;
    uint32_t *meta, *table, *rset, *rcnt, *cnt, *cur, *res;
    GtPtr gtable;
    uint16_t *log, *posslot, *vlist, *fstack;
    GLOBAL uint32_t *bits;
    GLOBAL uint64_t *gring;
    const GLOBAL uint64_t *tkeys;
    const GLOBAL int64_t *tkoff, *ttick;
    const GLOBAL uint8_t *tgroup, *tcontract;
    const GLOBAL uint32_t *tprefix;
    int64_t n_req, n_keys, n_prefix;   // trace sizes, read once
    int64_t max_rb;
    int32_t npw;              // prefix bitmap words
    bool has_tick;
    // ---------------- uniform state (identical in every wavefront)
    uint32_t head, tail;      // live log window [head, tail)
    int32_t hwm;              // slots [hwm, C) have never been used
    int32_t ftop;             // StaticQuota: free slots on the slot stack
    int32_t nvict;            // victims of the current request
    int32_t resident;         // resident blocks (excludes blocks being created)
    int32_t s_size, s_unp, m_unp;
    uint32_t gseq, curS, curM;
    uint32_t gseq0;           // gseq when this request's reclamation began
    uint32_t gsw;             // ghost sweep cursor
    int32_t rmax;
    int32_t err;
    // ---------------- statistics and group state (lane x = group x, VGPRs)
    uint64_t ev_total, s3_moves, s3_reins, s3_ghits, s3_gins;
    uint64_t evw;             // evictions of group `lane` seen by this wavefront
    int64_t bal[4], last[4];
    uint64_t c_req, c_probe, c_hit, c_miss, c_charged, c_evc, c_promo, c_gated, c_orph, c_dup, c_trunc;
    int64_t d_max, d_sum;
    int32_t r_max;
    int last_h, last_m, last_e, last_o;
    int32_t *preq;            // per-request quadruples of this instance, or null
    int64_t pr_next;          // first request whose quadruple is not written yet

    DEV Replayer(Coll &coll, const DevInst &inst, const DevTrace &tr, uint8_t *sbase, uint8_t *ws)
        : X(coll), tid((int)threadIdx.x), wid((int)rfl(threadIdx.x >> 6)), lane((int)__lane_id()), cb(0),
          I(inst), T(tr) {
        this->set_params(I);
        G = T.n_groups;
        room = policy == kSQ ? C / G : C;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            rho[c] = in_vgpr(I.rho[c]);
            beta[c] = in_vgpr(I.beta[c]);
            invw[c] = in_vgpr(I.invw[c]);
        }
        // the default-layout copy takes its array offsets as constants (the
        // host marks an instance for it only when they equal its own)
        constexpr bool fx = kFix == kFixC;
        constexpr StateOffsets F = fix_plan(kLay, kPol).f;
        if constexpr (kHyb) {
            if constexpr (kPack) {
                key = KeyPtr{gptr_rw(reinterpret_cast<uint64_t *>(ws + I.ws_key))};
                pfx = PfxPtr{gptr_rw(reinterpret_cast<uint32_t *>(ws + I.ws_key)) + 2};
                krec = gptr(reinterpret_cast<const KeyRec *>(ws + I.ws_key));
            } else {
                key = gptr_rw(reinterpret_cast<uint64_t *>(ws + I.ws_key));
                pfx = gptr_rw(reinterpret_cast<uint32_t *>(ws + I.ws_pfx));
                krec = nullptr;
            }
            gtable = gptr_rw(reinterpret_cast<uint32_t *>(ws + I.ws_gtable));
            rkeys = nullptr;
        } else {
            key = reinterpret_cast<uint64_t *>(sbase + (fx ? F.o_key : I.o_key));
            pfx = reinterpret_cast<uint32_t *>(sbase + (fx ? F.o_pfx : I.o_pfx));
            gtable = reinterpret_cast<uint32_t *>(sbase + (fx ? F.o_gtable : I.o_gtable));
            rkeys = reinterpret_cast<uint64_t *>(sbase + (fx ? F.o_rkeys : I.o_rkeys));
            krec = nullptr;
        }
        stamp = reinterpret_cast<StampT *>(sbase + (fx ? F.o_stamp : I.o_stamp));
        meta = reinterpret_cast<uint32_t *>(sbase + (fx ? F.o_meta : I.o_meta));
        table = reinterpret_cast<uint32_t *>(sbase + (fx ? F.o_table : I.o_table));
        rset = reinterpret_cast<uint32_t *>(sbase + (fx ? F.o_rset : I.o_rset));
        cnt = reinterpret_cast<uint32_t *>(sbase + (fx ? F.o_cnt : I.o_cnt));
        cur = reinterpret_cast<uint32_t *>(sbase + (fx ? F.o_cur : I.o_cur));
        res = reinterpret_cast<uint32_t *>(sbase + (fx ? F.o_res : I.o_res));
        log = reinterpret_cast<uint16_t *>(sbase + (fx ? F.o_log : I.o_log));
        posslot = reinterpret_cast<uint16_t *>(sbase + (fx ? F.o_posslot : I.o_posslot));
        vlist = reinterpret_cast<uint16_t *>(sbase + (fx ? F.o_vlist : I.o_vlist));
        fstack = reinterpret_cast<uint16_t *>(sbase + (fx ? F.o_fstack : I.o_fstack));
        rcnt = reinterpret_cast<uint32_t *>(sbase + (fx ? F.o_rcnt : I.o_rcnt));
        bits = gptr_rw(reinterpret_cast<uint32_t *>(ws + I.ws_bits));
        gring = gptr_rw(reinterpret_cast<uint64_t *>(ws + I.ws_gring));
        n_req = T.n_req;
        n_keys = T.n_keys;
        n_prefix = T.n_prefix;
        max_rb = T.max_req_blocks;
        has_tick = T.tick != nullptr;
        npw = I.n_prefix_words;
        tkeys = gptr(T.keys);
        tkoff = gptr(T.key_off);
        ttick = gptr(T.tick);
        tgroup = gptr(T.group);
        tcontract = gptr(T.contract);
        tprefix = gptr(T.prefix);
    }

    // ============================================================ sync
#ifdef PC_JITTER
    // Race-detection build: after every barrier each wavefront waits a
    // pseudo-random time (from the shader clock, the workgroup and the
    // wavefront): 0-7 x 128 cycles, or after one barrier in eight 0-63 x 128
    // cycles, longer than most barrier intervals.  The wavefronts of a
    // workgroup so enter each interval in shifted order, and a result that
    // depends on which one gets somewhere first (shared state read in the
    // interval in which another wavefront writes it) shows up as a parity
    // difference.
    DEV void jitter() const {
        uint64_t t = __builtin_amdgcn_s_memtime();
        t ^= (uint64_t)(blockIdx.x * 0x9E3779B9u) ^ ((uint64_t)wid << 17);
        t *= 0xff51afd7ed558ccdull;
        t ^= t >> 33;
        const uint32_t r = (uint32_t)(t >> 5);
        const uint32_t d = __builtin_amdgcn_readfirstlane(((r >> 3) & 7u) == 0u ? (r >> 6) & 63u : r & 7u);
        for (uint32_t i = 0; i < d; ++i) __builtin_amdgcn_s_sleep(2);
    }
#else
    DEV void jitter() const {}
#endif
    // Barrier making state-memory writes visible to the workgroup.  With the
    // state in LDS, only LDS is fenced, so global prefetches stay in flight.
    DEV void bsync() {
        if constexpr (kLds) {
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
        } else {
            __syncthreads();
        }
        jitter();
    }
    // Barrier for global memory too (ghost ring, prefix bitmaps).
    DEV void gsync() {
        __syncthreads();
        jitter();
    }

    template <int M>
    DEV void bballot(const bool (&p)[M], BMask (&out)[M]) {
        uint64_t b[M];
#pragma unroll
        for (int i = 0; i < M; ++i) b[i] = ballot(p[i]);
        if (lane == 0) {
#pragma unroll
            for (int i = 0; i < M; ++i) X.m[cb][i][wid] = b[i];
        }
        bsync();
#pragma unroll
        for (int i = 0; i < M; ++i)
#pragma unroll
            for (int ww = 0; ww < kW; ++ww) out[i].w[ww] = rfl64(X.m[cb][i][ww]);
        cb ^= 1;
    }
    DEV BMask bballot1(bool p) {
        bool a[1] = {p};
        BMask o[1];
        bballot<1>(a, o);
        return o[0];
    }

    // ============================================================ debt (lane x)
    // Eq. 1, exactly: min(beta, B + rho*dt) with the product in 128 bits.
    DEV int64_t eff(int c, int64_t t) const {
        const int64_t dt = t - last[c];
        const uint64_t gap = (uint64_t)(beta[c] - bal[c]);
        const uint64_t lo = (uint64_t)rho[c] * (uint64_t)dt;
        const uint64_t hi = __umul64hi((uint64_t)rho[c], (uint64_t)dt);
        if (hi != 0 || lo >= gap) return beta[c];
        return bal[c] + (int64_t)lo;
    }
    DEV int64_t raw_debt(int64_t t) const {   // Eq. 3
        if (K == 1) { const int64_t b = eff(0, t); return b < 0 ? -b : 0; }
        int64_t d = 0;
#pragma unroll
        for (int c = 0; c < 4; ++c)
            if (c < K) { int64_t b = eff(c, t); if (b < 0) d -= b; }
        return d;
    }
    DEV int64_t norm_debt(int64_t t) const {  // Eq. 5, 1/w_c in Q16
        if (K == 1) { const int64_t b = eff(0, t); return b < 0 ? -b : 0; }   // w = 1
        int64_t d = 0;
#pragma unroll
        for (int c = 0; c < 4; ++c)
            if (c < K) {
                int64_t b = eff(c, t);
                if (b < 0) {
                    uint64_t a = (uint64_t)(-b), w = (uint64_t)invw[c];
                    uint64_t lo = a * w, hi = __umul64hi(a, w);
                    d += (int64_t)((hi << 48) | (lo >> 16));
                }
            }
        return d;
    }
    // Eq. 8: 1/W_g, the smallest decrement among indebted contracts, or 0
    // when none is indebted (the host keeps every invw at 1 or more)
    DEV int64_t decrement(int64_t t) const {
        if (K == 1) return eff(0, t) < 0 ? kScale : 0;
        int64_t m = -1;
#pragma unroll
        for (int c = 0; c < 4; ++c)
            if (c < K && eff(c, t) < 0 && (m < 0 || invw[c] < m)) m = invw[c];
        return m < 0 ? 0 : m;
    }

    // ============================================================ tables
    // both buckets of h (two 16-byte loads each), from LDS or global memory
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    template <typename P4>
    DEV static void unpack_buckets(P4 t4, const TH &h, uint32_t e[16]) {
        const u32x4 a0 = t4[2 * h.b1], a1 = t4[2 * h.b1 + 1], c0 = t4[2 * h.b2], c1 = t4[2 * h.b2 + 1];
        e[0] = a0.x; e[1] = a0.y; e[2] = a0.z; e[3] = a0.w; e[4] = a1.x; e[5] = a1.y; e[6] = a1.z; e[7] = a1.w;
        e[8] = c0.x; e[9] = c0.y; e[10] = c0.z; e[11] = c0.w; e[12] = c1.x; e[13] = c1.y; e[14] = c1.z; e[15] = c1.w;
    }
    DEV void load_buckets(const uint32_t *tb, const TH &h, uint32_t e[16]) const {
        unpack_buckets(reinterpret_cast<const u32x4 *>(tb), h, e);
    }
    DEV void load_buckets(const GLOBAL uint32_t *tb, const TH &h, uint32_t e[16]) const {
        unpack_buckets(reinterpret_cast<const GLOBAL u32x4 *>(tb), h, e);
    }
    DEV uint32_t epos(const TH &h, int i) const { return i < 8 ? 8 * h.b1 + i : 8 * h.b2 + (i - 8); }
    // Probe both buckets of k.  Returns the number of tag matches; `cand` is
    // the slot of the last one.  With one match the caller confirms the key
    // (together with its other loads); with several, tfind_slow decides.
    // `fm` receives the free-entry mask of the two buckets (bits 0-7 b1,
    // 8-15 b2): the lookup's snapshot of the table, which a one-step
    // request inserts with (the table does not change between the lookup
    // and the insertion except for reclamation's clears, which only free
    // entries).
    DEV int tprobe(const TH &h, uint32_t &cand, uint32_t &fm) const {
        uint32_t e[16];
        load_buckets(table, h, e);
        return tscan(h, e, cand, fm);
    }
    // tprobe on buckets already loaded
    DEV int tscan(const TH &h, const uint32_t (&e)[16], uint32_t &cand, uint32_t &fm) const {
        int nm = 0;
        uint32_t cv = 0, f = 0;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const bool mt = (e[i] >> 16) == h.tag;
            nm += mt;
            cv = mt ? e[i] : cv;
            f |= (e[i] == kEmpty ? 1u : 0u) << i;
        }
        cand = cv & 0xFFFFu;
        fm = f;
        return nm;
    }
    DEV int tfind_slow(uint64_t k, const TH &h) const {
        uint32_t e[16];
        load_buckets(table, h, e);
        for (int i = 0; i < 16; ++i)
            if ((e[i] >> 16) == h.tag && key[e[i] & 0xFFFFu] == k) return (int)(e[i] & 0xFFFFu);
        return -1;
    }
    // Free-entry mask of both buckets of a snapshot (bits 0-7 bucket b1,
    // bits 8-15 bucket b2).  In the ghost table an entry that left the
    // window counts as free (see glive).
    DEV uint32_t free_mask(const uint32_t (&e)[16], bool ghost, uint32_t gref) const {
        uint32_t m = 0;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const bool f = ghost ? !glive(e[i], gref) : e[i] == kEmpty;
            m |= (f ? 1u : 0u) << i;
        }
        return m;
    }
    // Parallel insert without compare-and-swap.  Every inserter of a step
    // reads its two buckets (the snapshot) before a barrier that no table
    // write crosses; after it, a claim counter per bucket (ctr[b], kEmpty
    // meaning zero) hands out distinct ranks, and rank r takes the r-th free
    // entry of the snapshot -- the emptier bucket first.  `touched` records
    // the counters used, which tclaim_reset puts back to kEmpty after the
    // next barrier.  Returns the entry's index, or kEmpty when both buckets
    // are full.
    template <typename TP>
    DEV uint32_t tclaim(TP tb, uint32_t *ctr, uint32_t val, const TH &h, const uint32_t (&e)[16],
                        uint32_t &touched, bool ghost = false, uint32_t gref = 0) {
        return tclaim_m(tb, ctr, val, h, free_mask(e, ghost, gref), touched);
    }
    template <typename TP>
    DEV uint32_t tclaim_m(TP tb, uint32_t *ctr, uint32_t val, const TH &h, uint32_t fm, uint32_t &touched) {
        const uint32_t m1 = fm & 0xFFu, m2 = fm >> 8;
        const bool sec = __builtin_popcount(m2) > __builtin_popcount(m1);
        touched = 0;
        for (int pass = 0; pass < 2; ++pass) {
            const bool use2 = (pass == 0) == sec;
            const uint32_t b = use2 ? h.b2 : h.b1;
            uint32_t msk = use2 ? m2 : m1;
            touched |= use2 ? 2u : 1u;
            uint32_t r = atomicAdd(&ctr[b], 1u) + 1u;
            if (r < (uint32_t)__builtin_popcount(msk)) {
                while (r--) msk &= msk - 1u;
                const uint32_t at = 8 * b + (uint32_t)__builtin_ctz(msk);
                tb[at] = val;
                return at;
            }
        }
        return kEmpty;
    }
    DEV void tclaim_reset(uint32_t *ctr, const TH &h, uint32_t touched) {
        if (touched & 1u) ctr[h.b1] = kEmpty;
        if (touched & 2u) ctr[h.b2] = kEmpty;
    }
    // Record an entry that found both buckets full; kick_pending() places it.
    DEV void defer_kick(uint32_t val, uint64_t k, bool main) {
        const uint32_t i = atomicAdd(&X.novf, 1u);
        X.kval[i] = val;
        X.kkey[i] = k;
        X.kmain[i] = main ? 1u : 0u;
    }
    // the main-table entry of slot s is now at index p
    DEV void set_tpos(uint32_t s, uint32_t p) { meta[s] = (meta[s] & kLowMeta) | (p << kTposShift); }
    // Serial cuckoo displacement, one thread.  gref: ghost sequence that
    // decides which ghost entries are still live.
    template <typename TP>
    DEV bool kick(TP tb, bool main, uint32_t val, uint64_t k, uint32_t gref) {
        const uint32_t nbk = main ? nb : gnb;
        uint32_t cv = val;
        uint64_t ck = k;
        uint32_t from = 0xFFFFFFFFu;
        for (int it = 0; it < 512; ++it) {
            const TH h = thash(ck, nbk, rbmask);
            for (int i = 0; i < 16; ++i) {
                const uint32_t p = epos(h, i);
                if (main ? tb[p] == kEmpty : !glive(tb[p], gref)) {
                    tb[p] = cv;
                    if (main) set_tpos(cv & 0xFFFFu, p);
                    return true;
                }
            }
            uint32_t b = (h.b1 == from) ? h.b2 : h.b1;
            if (from == 0xFFFFFFFFu && (it & 1)) b = h.b2;
            const uint32_t w = (uint32_t)(it * 5 + (uint32_t)(ck >> 7)) & 7u;
            const uint32_t victim = tb[8 * b + w];
            tb[8 * b + w] = cv;
            if (main) set_tpos(cv & 0xFFFFu, 8 * b + w);
            cv = victim;
            ck = main ? key[victim & 0xFFFFu] : gring[victim & grmask];
            from = b;
        }
        return false;
    }
    // Called by all threads after a barrier that follows defer_kick calls.
    DEV void kick_pending(uint32_t gref = 0) {
        const uint32_t nk = rfl(X.novf);
        if (nk == 0) return;
        // every wavefront reads the count before thread 0 clears it (one
        // that read it after would skip the barriers below); the walk reads
        // the keys of table entries, which this request may just have
        // written (hybrid layout: in global memory)
        if constexpr (kHyb) gsync();
        else bsync();
        if (tid == 0) {
            for (uint32_t i = 0; i < nk; ++i) {
                const bool main = X.kmain[i] != 0;
                const bool placed = main ? kick(table, true, X.kval[i], X.kkey[i], gref)
                                         : kick(gtable, false, X.kval[i], X.kkey[i], gref);
                if (!placed) X.kerr = kErrInternal;
            }
            X.novf = 0;
        }
        gsync();
        if (rfl((uint32_t)X.kerr)) err = kErrInternal;
    }

    // ============================================================ per-group counters
    // LDS atomics on a few shared counters serialize lane by lane, so the
    // lanes of a wavefront are grouped by index first: one atomic per
    // distinct index.  Called by every lane of the wavefront.
    DEV void wave_add(uint32_t *arr, uint32_t idx, bool active, int d) {
        uint64_t act = ballot(active);
        while (act) {
            const int l = first_bit(act);
            const uint32_t x = __builtin_amdgcn_readlane(idx, l);
            const uint64_t m = ballot(active && idx == x);
            if (lane == l) atomicAdd(&arr[x], (uint32_t)(d * popc(m)));
            act &= ~m;
        }
    }

    // ============================================================ eviction core
    // A resident block's metadata carries the index of its main-table entry
    // (set where the entry is claimed or displaced), so a victim's entry is
    // known from the metadata the scan reads anyway.
    DEV static uint32_t victim_entry(bool maybe, uint32_t mt) { return maybe ? (mt >> kTposShift) : kEmpty; }
    // Slot named by log position pos, or slot 0 past the tail.  The load is
    // unconditional (the masked position is always inside the log) and the
    // entry is used only when valid, since the log past the tail may never
    // have been written; so every slot index is below C, and a scan can load
    // the slot's metadata, stamp and key together without a branch.
    DEV uint32_t slot_at(uint32_t pos, bool valid) const {
        const uint32_t e = log[pos & lmask];
        return valid ? e : 0u;
    }
    // Victims of one step: thread with v holds victim slot s with metadata mt
    // (vrank = its rank among the step's victims) and its table entry loc.
    // Every thread calls this.
    DEV void evict_elems(bool v, uint32_t s, uint32_t mt, int vrank, uint32_t loc) {
        const uint32_t o = owner_of(mt);
        // per distinct owner among the victims: evictions counted in lane
        // `owner`, and one atomic on the owner's resident count
        uint64_t act = ballot(v);
        while (act) {
            const int l = first_bit(act);
            const uint32_t x = __builtin_amdgcn_readlane(o, l);
            const uint64_t m = ballot(v && o == x);
            const int c = popc(m);
            if ((uint32_t)lane == x) evw += (uint64_t)c;
            if (lane == l) atomicAdd(&res[x], (uint32_t)(-c));
            act &= ~m;
        }
        if (v) {
            if (loc != kEmpty) table[loc] = kEmpty;
            meta[s] = 0;
            vlist[nvict + vrank] = (uint16_t)s;
        }
    }
    DEV void evicted(int nv) {
        nvict += nv;
        resident -= nv;
        ev_total += (uint64_t)nv;
    }

    // Compaction of the free-queue log: live entries keep their order and
    // are renumbered from `head`; all cursors restart at `head`.  One
    // barrier per 256-position step (its ballot): a step writes log
    // positions below the next step's reads (nw <= p0, and fewer than R
    // positions apart, so no two alias in the ring), metadata is not
    // written at all, and a slot's stamp, which a step rewrites for its live
    // entries, decides nothing in the next step whichever value that step
    // reads -- a later position of the same slot is a stale copy, and
    // neither the old nor the new stamp equals it.
    DEV void compact() {
        PROF_COUNT(1, 1);
        bsync();
        uint32_t nw = head;
        for (uint32_t p0 = head; p0 < tail; p0 += kB) {
            const uint32_t pos = p0 + tid;
            const bool valid = pos < tail;
            const uint32_t s = slot_at(pos, valid);
            const uint32_t mt = meta[s];
            const StampT st = stamp[s];
            const bool live = valid && (mt & kInLog) && st == (StampT)pos;
            const BMask lm = bballot1(live);   // every read of this step is done
            if (live) {
                const uint32_t np = nw + (uint32_t)lm.rank(wid);
                log[np & lmask] = (uint16_t)s;
                stamp[s] = (StampT)np;
            }
            nw += (uint32_t)lm.count();
        }
        tail = nw;
        if constexpr (kQueues)
            for (int i = tid; i < 196; i += kB) cur[i] = head;
        curS = curM = head;
        bsync();
    }
    DEV void ensure_room(uint32_t k) {
        if (tail + k - head <= R) return;
        if constexpr (kQueues) {   // lowest cursor of a non-empty queue bounds every live entry
            // Every wavefront reads every queue count and keeps its own copy
            // of head, so all must read the same counts: a barrier before the
            // reads (a request that evicted nothing reaches here with none
            // after its lookup's count updates) and one after them (the
            // insert that follows changes counts).  head, tail and k are
            // uniform, so all wavefronts take this branch together.
            bsync();
            uint32_t m = tail;
            for (int i = lane; i < 192; i += 64)
                if (cnt[i] > 0 && cur[i] < m) m = cur[i];
            m = wave_min32(m);
            bsync();
            if (m > head) head = m;
        } else if constexpr (policy == kS3) {
            const uint32_t m = curS < curM ? curS : curM;
            if (m > head) head = m;
        }
        if (tail + k - head > R) compact();
    }

    // ---------------------------------------------------------------- LRU
    DEV void evict_lru(int e) {
        int rem = e;
        while (rem > 0 && err == 0) {
            const uint32_t pos = head + tid;
            const bool valid = pos < tail;
            const uint32_t s = slot_at(pos, valid);
            const uint32_t mt = meta[s];
            const StampT st = stamp[s];
            const bool live = valid && (mt & kInLog) && st == (StampT)pos;
            const uint32_t loc = victim_entry(live, mt);
            const BMask lm = bballot1(live);
            const int rk = lm.rank(wid);
            const int tot = lm.count();
            const int nv = tot < rem ? tot : rem;
            evict_elems(live && rk < rem, s, mt, rk, loc);
            evicted(nv);
            if (nv == rem) head = head + (uint32_t)lm.nth(rem - 1) + 1;
            else head = (head + kB < tail) ? head + kB : tail;
            rem -= nv;
            if (nv == 0 && head >= tail) err = kErrInternal;
            bsync();
        }
    }

    // ---------------------------------------------------------------- PrefixShield
    // Take k victims from queue ci in free-queue order.  x < 0: any owner;
    // s < 0: any class (no segmentation).
    DEV void ps_take(int x, int s, int ci, int k) {
        PROF_COUNT(3, 1);
        // every live entry sits at or above head; a cursor left behind by an
        // idle queue skips the dead stretch below it
        uint32_t c = rfl(cur[ci]);
        if (c < head) c = head;
        int rem = k;
        while (rem > 0 && err == 0) {
            const uint32_t pos = c + tid;
            const bool valid = pos < tail;
            const uint32_t sl = slot_at(pos, valid);
            const uint32_t mt = meta[sl];
            const StampT st = stamp[sl];
            const bool live = valid && (mt & kInLog) && st == (StampT)pos;
            const bool match = live && (x < 0 || (int)owner_of(mt) == x) && (s < 0 || (int)cls_of(mt) == s);
            const uint32_t loc = victim_entry(match, mt);
            const BMask mm = bballot1(match);
            const int rk = mm.rank(wid);
            const int tot = mm.count();
            const int nv = tot < rem ? tot : rem;
            const bool vic = match && rk < rem;
            wave_add(cnt, 3 * owner_of(mt) + (s < 0 ? 0u : (uint32_t)s), vic, -1);
            evict_elems(vic, sl, mt, rk, loc);
            evicted(nv);
            if (nv == rem) c = c + (uint32_t)mm.nth(rem - 1) + 1;
            else c = (c + kB < tail) ? c + kB : tail;
            rem -= nv;
            if (nv == 0 && c >= tail) err = kErrInternal;
            bsync();
        }
        // every wavefront stores the (same) cursor, so each one's next read
        // of it follows its own store; the loop's barriers already order
        // every read of this call before these stores
        if (lane == 0) cur[ci] = c;
    }
    // Oldest live entry of queue (x, s); advances that queue's cursor to it.
    DEV uint32_t ps_headpos(int x, int s) {
        const int ci = 3 * x + (s < 0 ? 0 : s);
        uint32_t c = rfl(cur[ci]);
        if (c < head) c = head;
        uint32_t found = 0xFFFFFFFFu;
        while (c < tail) {
            const uint32_t pos = c + tid;
            const bool valid = pos < tail;
            const uint32_t sl = slot_at(pos, valid);
            const uint32_t mt = meta[sl];
            const StampT st = stamp[sl];
            const bool live = valid && (mt & kInLog) && st == (StampT)pos;
            const bool match = live && (int)owner_of(mt) == x && (s < 0 || (int)cls_of(mt) == s);
            const BMask mm = bballot1(match);
            if (mm.any()) { found = c + (uint32_t)mm.first(); c = found; break; }
            c = (c + kB < tail) ? c + kB : tail;
        }
        bsync();
        if (tid == 0) cur[ci] = c;
        bsync();
        return found;
    }
    DEV void evict_ps(int e, int64_t t) {
        const bool grp = lane < G;
        int64_t P = 0, D = 0;
        uint32_t avail = 0;
        if (grp) {
            P = norm_debt(t);
            D = decrement(t);
            avail = cnt[3 * lane] + cnt[3 * lane + 1] + cnt[3 * lane + 2];
        }
        int rem = e;
        while (rem > 0 && err == 0) {
            const bool inE = grp && avail > 0 && P > eps;      // Eq. 6
            const uint64_t Em = ballot(inE);
            if (!Em) break;
            const int64_t pm = wave_max64(inE ? P : -1);       // Eq. 7
            uint64_t tied = ballot(inE && P == pm);
            int gs = first_bit(tied);
            if (popc(tied) > 1) {   // ties: lowest non-empty segment, then oldest head entry
                uint32_t seg = 3;
                if (grp)
                    for (int s = nseg - 1; s >= 0; --s)
                        if (cnt[3 * lane + s] > 0) seg = (uint32_t)s;
                const int mseg = (int)wave_min32(((tied >> lane) & 1) ? seg : 3u);
                tied &= ballot(seg == (uint32_t)mseg);
                gs = first_bit(tied);
                if (popc(tied) > 1) {
                    uint32_t best = 0xFFFFFFFFu;
                    for (uint64_t tm = tied; tm; tm &= tm - 1) {
                        const int x = first_bit(tm);
                        const uint32_t hp = ps_headpos(x, nseg == 1 ? -1 : mseg);
                        if (hp < best) { best = hp; gs = x; }
                    }
                }
            }
            const int64_t Pg = bcast64(P, gs), Dg = bcast64(D, gs);
            if (Dg <= 0) { err = kErrInternal; break; }   // an indebted group has a positive decrement
            const int ag = (int)bcast32(avail, gs);
            const int64_t p2 = wave_max64((inE && lane != gs) ? P : -1);
            const int64_t thr = p2 > eps ? p2 : eps;
            // g* keeps winning strictly while P - i*D > max(second, eps); with
            // one contract the decrement is exactly one block (a shift)
            int64_t k1 = 0;
            if (Pg > thr) {
                const uint64_t num = (uint64_t)(Pg - thr) + (uint64_t)Dg - 1;
                k1 = K == 1 ? (int64_t)(num >> 16) : (int64_t)udiv64(num, (uint64_t)Dg);
            }
            int64_t k = k1 > 1 ? k1 : 1;
            if (k > rem) k = rem;
            if (k > ag) k = ag;
            if (nseg == 1) {
                ps_take(gs, -1, 3 * gs, (int)k);
            } else {
                int kk = (int)k;
                for (int s = 0; s < 3 && kk > 0; ++s) {
                    const int cs = (int)rfl(cnt[3 * gs + s]);
                    const int tk = cs < kk ? cs : kk;
                    if (tk > 0) ps_take(gs, s, 3 * gs + s, tk);
                    kk -= tk;
                }
            }
            if (lane == gs) {
                P -= k * Dg;
                if (P < 0) P = 0;
                avail -= (uint32_t)k;
            }
            rem -= (int)k;
        }
        // no indebted candidate owner: global segment order (Eq. 9 fallback)
        for (int s = 0; s < nseg && rem > 0 && err == 0; ++s) {
            uint32_t cs = 0;
            if (grp) cs = cnt[3 * lane + (nseg == 1 ? 0 : s)];
            const int tot = (int)wave_sum32(cs);
            const int tk = tot < rem ? tot : rem;
            if (tk > 0) ps_take(-1, nseg == 1 ? -1 : s, 192 + s, tk);
            rem -= tk;
        }
        if (rem > 0) err = kErrInternal;
    }

    // ---------------------------------------------------------------- S3-FIFO
    // The ghost remembers the last g_cap insertions.  Entries hold (tag, ring
    // position = sequence mod 2^gr); an entry is live while its age
    // gref - 1 - sequence is below g_cap, so leaving the window needs no work
    // at all.  A sweep clears dead entries before their age could wrap the
    // ring: each batch (nv <= 256 insertions) sweeps at least
    // ceil(nv * entries / span) entries at its start, span = 2^gr - g_cap - 256.
    // Between two visits of an entry fewer than 256 + span insertions happen,
    // so an entry seen live at one visit (age < g_cap) has age below
    // g_cap + 256 + span = 2^gr when it is seen next, and is cleared then if
    // dead.  Any 2^gr of at least 2 g_cap + 256 works (span >= g_cap); the
    // host takes min(2^16, next power of two >= 4 g_cap + 256), so span is
    // at least 3 g_cap and the sweep proportionally lighter.
    DEV bool glive(uint32_t e, uint32_t gref) const {
        return e != kEmpty && ((gref - 1u - (e & 0xFFFFu)) & grmask) < (uint32_t)g_cap;
    }
    // ghost hit for key k: remove it and report true.  Entries written by
    // this request's own reclamation hold its victims' keys, never the key
    // of one of its new blocks, and are skipped without reading the ring.
    DEV bool ghost_take(uint64_t k) {
        const TH h = thash(k, gnb, rbmask);
        uint32_t e[16];
        load_buckets(gtable, h, e);
        // entries with the key's tag first (branch-free): a match is rare,
        // and only a lane with one checks liveness and reads the ring
        uint32_t tm = 0;
#pragma unroll
        for (int i = 0; i < 16; ++i) tm |= ((e[i] >> 16) == h.tag ? 1u : 0u) << i;
        int at = -1;
        if (tm != 0u) {
            const uint32_t nown = gseq - gseq0;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const uint32_t pos = e[i] & 0xFFFFu;
                if (at < 0 && ((tm >> i) & 1u) && glive(e[i], gseq) && ((gseq - 1u - pos) & grmask) >= nown &&
                    gring[pos & grmask] == k)
                    at = i;
            }
        }
        if (at >= 0) gtable[epos(h, at)] = kEmpty;
        return at >= 0;
    }
    // Sweep of the ghost table for a batch of at most kB insertions (see
    // the ghost's description above); runs before the batch's barrier.
    DEV void ghost_sweep() {
        uint32_t ns = (uint32_t)(((uint64_t)kB * gsrate + 0xFFFFu) >> 16);
        if (ns > gne) ns = gne;
        // every read of the first kRounds rounds is issued before any clear
        // (the host's sizing keeps ns below 700, within 3 rounds of kB; the
        // loop after them only guards that bound)
        constexpr int kRounds = 3;
        uint32_t ev[kRounds];
#pragma unroll
        for (int q = 0; q < kRounds; ++q) {
            const uint32_t i = (uint32_t)(q * kB + tid);
            ev[q] = i < ns ? gtable[(gsw + i) & (gne - 1u)] : kEmpty;
        }
#pragma unroll
        for (int q = 0; q < kRounds; ++q) {
            const uint32_t i = (uint32_t)(q * kB + tid);
            if (ev[q] != kEmpty && !glive(ev[q], gseq)) gtable[(gsw + i) & (gne - 1u)] = kEmpty;
        }
        for (uint32_t i = (uint32_t)(kRounds * kB + tid); i < ns; i += kB) {
            const uint32_t ix = (gsw + i) & (gne - 1u);
            const uint32_t e = gtable[ix];
            if (e != kEmpty && !glive(e, gseq)) gtable[ix] = kEmpty;
        }
        gsw += ns;
    }
    // First position of the batch's cut: the first candidate whose counts of
    // candidates (cr), moves (mr) and evictions (er) before it fail the
    // batch's conditions -- small queue: (cr >= la and (munp or mr >= 1)) or
    // er >= lim; main queue: er >= lim -- or kB.  Lane l evaluates thread
    // positions 64 w + l of every word w with running counts, so the cut
    // takes one ballot per word instead of serial scans of the masks.
    // Called with every lane active.
    DEV static int s3_stop(const BMask &candm, const BMask &mvm, const BMask &evm, bool small, int la, bool munp,
                           int lim) {
        uint64_t fm[kW];
        int pc = 0, pm = 0, pe = 0;
#pragma unroll
        for (int w = 0; w < kW; ++w) {
            const uint64_t cw = candm.w[w], mw = mvm.w[w], ew = evm.w[w];
            const int cr = pc + mbcnt(cw), mr = pm + mbcnt(mw), er = pe + mbcnt(ew);
            const bool f = small ? ((cr >= la && (munp || mr >= 1)) || er >= lim) : er >= lim;
            fm[w] = ballot(f) & cw;
            pc += popc(cw);
            pm += popc(mw);
            pe += popc(ew);
        }
        int stop = kB;
#pragma unroll
        for (int w = kW - 1; w >= 0; --w) stop = fm[w] ? 64 * w + first_bit(fm[w]) : stop;
        return stop;
    }
    // One scan step per batch: the queue in use (S or M, Z18) is scanned from
    // its cursor; candidates are its live unpinned entries.  Everything a
    // victim needs that does not depend on which candidates end up as
    // victims (its table entry, its ghost buckets, the ghost sweep) is done
    // before the step's only ballot.
    DEV void evict_s3(int e) {
        int rem = e;
        uint32_t spS = curS, spM = curM;
        uint32_t keptS = 0xFFFFFFFFu, keptM = 0xFFFFFFFFu;
        while (rem > 0 && err == 0) {
            if (tail + kB - head > R) {
                ensure_room(kB);
                spS = curS; spM = curM;
                keptS = keptM = 0xFFFFFFFFu;
            }
            // the queue sizes are wave-uniform; saying so keeps the batch
            // cut below in scalar code instead of exec-masked vector code
            rem = (int)rfl((uint32_t)rem);
            s_size = (int)rfl((uint32_t)s_size);
            s_unp = (int)rfl((uint32_t)s_unp);
            m_unp = (int)rfl((uint32_t)m_unp);
            const bool useS = (s_size >= s_cap && s_unp > 0) || (m_unp == 0);
            PROF_COUNT(2, 1);
            const uint32_t sp = useS ? spS : spM;
            const uint32_t lim = tail;
            if (sp >= lim) { err = kErrInternal; break; }
            const uint32_t pos = sp + tid;
            const bool valid = pos < lim;
            const uint32_t sl = slot_at(pos, valid);
            // a small-queue victim is remembered by the ghost: its key is
            // read with the metadata and stamp, in the same round trip
            const bool gho = useS && g_cap > 0;
            const uint32_t mt = meta[sl];
            const StampT st = stamp[sl];
            const uint64_t kv = gho ? key[sl] : 0ull;
            const bool live = valid && (mt & kInLog) && st == (StampT)pos;
            const bool inQ = live && (useS ? !(mt & kQMain) : (mt & kQMain) != 0);
            const bool cand = inQ && !(mt & kPin);
            const uint32_t f = freq_of(mt);
            // small queue: move (accessed) or evict into the ghost;
            // main queue: reinsert (freq > 0) or evict
            const bool mv = cand && (useS ? (int)f >= move_thr : f > 0);
            const bool maybe_ev = cand && !mv;
            const uint32_t loc = victim_entry(maybe_ev, mt);
            const uint64_t vk = maybe_ev ? kv : 0ull;
            TH hg = {};
            uint32_t gfree = 0;
            if (gho) {
                if (maybe_ev) {
                    hg = thash(vk, gnb, rbmask);
                    uint32_t eg[16];
                    load_buckets(gtable, hg, eg);
                    gfree = free_mask(eg, true, gseq);
                }
                ghost_sweep();
            }
            bool p3[3] = {cand, mv, inQ};
            BMask m3[3];
            bballot<3>(p3, m3);
            const BMask &candm = m3[0], &mvm = m3[1], &inQm = m3[2];
            const BMask evm = candm.andnot(mvm);
            // The batch is the longest prefix of candidates that may all be
            // processed: each condition below holds on a prefix of them, so
            // `stop` (first candidate not processed, kB if none) is the
            // earliest position where one of them starts to fail.
            // Small queue: a candidate may be processed while |S| less the
            // candidates before it is still >= S_cap with unpinned S left
            // (rank < la), or while M has no unpinned block and nothing moved
            // there before it; main queue: while fewer than min(rem, unpinned
            // M) evictions precede it; both: while fewer than `rem`.  Each
            // condition fails from some candidate on, so `stop` is the first
            // candidate where the combination fails (kB if none).
            const int stop = useS ? s3_stop(candm, mvm, evm, true, min(s_size - s_cap + 1, s_unp), m_unp > 0, rem)
                                  : s3_stop(candm, mvm, evm, false, 0, false, min(rem, m_unp));
            const bool proc = cand && tid < stop;
            const BMask pmm = mvm.below(stop), pem = evm.below(stop);
            const int nmv = pmm.count(), nev = pem.count();
            // live entries of this queue that stay behind the scan point
            const BMask kept = inQm.andnot(candm).below(stop);
            const int kf = stop < kB ? (kept.any() ? (kept.first() < stop ? kept.first() : stop) : stop)
                                     : (kept.any() ? kept.first() : -1);
            if (kf >= 0) {
                const uint32_t kp = sp + (uint32_t)kf;
                if (useS) { if (kp < keptS) keptS = kp; } else { if (kp < keptM) keptM = kp; }
            }
            // moves / reinsertions: append to the log tail in queue order
            if (proc && mv) {
                const uint32_t np = tail + (uint32_t)pmm.rank(wid);
                log[np & lmask] = (uint16_t)sl;
                stamp[sl] = (StampT)np;
                uint32_t m2 = mt & ~(3u << kFreqShift);
                if (useS) m2 |= kQMain;
                else m2 |= (f - 1) << kFreqShift;
                meta[sl] = m2;
            }
            tail += (uint32_t)nmv;
            const bool pev = proc && !mv;
            const int erk = pem.rank(wid);
            uint32_t gtouched = 0;
            if (useS) {
                // ghost insertion of the evicted blocks, in eviction order;
                // entries that would leave the window within the batch are
                // not inserted
                if (gho && nev > 0) {
                    const uint32_t seq = gseq + (uint32_t)erk;
                    const uint32_t gend = gseq + (uint32_t)nev;
                    if (pev && (int64_t)seq + g_cap >= (int64_t)gend) {
                        gring[seq & grmask] = vk;
                        const uint32_t val = (hg.tag << 16) | (seq & grmask);
                        if (tclaim_m(gtable, rset, val, hg, gfree, gtouched) == kEmpty) defer_kick(val, vk, false);
                    }
                }
                s3_gins += (uint64_t)nev;
                s_size -= nmv + nev;
                s_unp -= nmv + nev;
                m_unp += nmv;
                s3_moves += (uint64_t)nmv;
            } else {
                m_unp -= nev;
                s3_reins += (uint64_t)nmv;
            }
            evict_elems(pev, sl, mt, erk, loc);
            evicted(nev);
            rem -= nev;
            const uint32_t adv = stop < kB ? (uint32_t)stop : ((lim - sp) < (uint32_t)kB ? (lim - sp) : (uint32_t)kB);
            if (adv == 0) err = kErrInternal;   // a scan that cannot advance is a bug, never a hang
            if (useS) spS = sp + adv; else spM = sp + adv;
            // the next batch's bucket snapshot must see this batch's ghost
            // claims (hybrid layout: the ghost table is in global memory)
            if constexpr (kHyb && kPol == kS3) gsync();
            else bsync();
            if (useS) {
                if (gho && nev > 0) {
                    tclaim_reset(rset, hg, gtouched);
                    if (rfl(X.novf)) {   // displacement reads ring keys written just now
                        gsync();
                        kick_pending(gseq + (uint32_t)nev);
                    }
                }
                gseq += (uint32_t)nev;
            }
        }
        curS = keptS < spS ? keptS : spS;
        curM = keptM < spM ? keptM : spM;
        const uint32_t m = curS < curM ? curS : curM;
        if (m > head) head = m;
    }

    // ============================================================ slots
    // Slot of the i-th new block (by rank) of the request.  A work-conserving
    // policy reclaims only once the never-used slots are gone, so its new
    // blocks take those first and then this request's victims' slots, and
    // no slot is ever left over.  StaticQuota reclaims inside a full
    // partition while the cache may still have room, so its new blocks take
    // this request's victims' slots first, then the free-slot stack, then
    // never-used slots; victims' slots it does not need go on the stack.
    DEV uint32_t new_slot(int i, int nfresh) const {
        if constexpr (policy == kSQ) {
            if (i < nvict) return vlist[i];
            i -= nvict;
            if (i < ftop) return fstack[ftop - 1 - i];
            return (uint32_t)(hwm + i - ftop);
        } else {
            return i < nfresh ? (uint32_t)(hwm + i) : vlist[i - nfresh];
        }
    }
    // after the request's last new block: account for the slots it took
    DEV void slots_taken(int nalloc, int nfresh) {
        if constexpr (policy == kSQ) {
            const int uv = nalloc < nvict ? nalloc : nvict;
            const int rest = nalloc - uv;
            const int us = rest < ftop ? rest : ftop;
            for (int k = tid; k < nvict - uv; k += kB) fstack[ftop + k] = vlist[uv + k];
            ftop += (nvict - uv) - us;
            hwm += rest - us;
        } else {
            hwm += nalloc < nfresh ? nalloc : nfresh;
        }
    }

    // ============================================================ one request
    DEV void put_per_request(int64_t i) {
        int32_t *o = preq + 4 * i;
        o[0] = last_h; o[1] = last_m; o[2] = last_e; o[3] = last_o;
        pr_next = i + 1;
    }
    // key at position j of the request whose keys start at ko: the copy in
    // LDS, or in the hybrid layout the trace's own (read-only) keys
    DEV uint64_t rkey(int64_t ko, uint32_t j) const {
        if constexpr (kHyb) return tkeys[ko + j];
        else return rkeys[j];
    }
    DEV Req load_req(int64_t r) const {
        Req q;
        q.g = tgroup[r];
        q.c = tcontract[r];
        q.p = tprefix[r];
        q.t = has_tick ? ttick[r] : r;
        q.ko = tkoff[r];
        q.kend = tkoff[r + 1];
        return q;
    }

    // `kn` holds keys[ko + tid] of this request and bref/badm its prefix
    // bitmap words (all prefetched); on return they hold the same for `nx`.
    // `nn` receives the descriptor of request r + 2 (loaded here, used two
    // requests later, so that no descriptor load is waited for).
    DEV bool request(int64_t r, const Req &q, int64_t &tprev, uint64_t &kn, uint32_t &bref, uint32_t &badm,
                     const Req &nx, bool has_next, Req &nn) {
        const int g = q.g, c = q.c;
        const uint32_t p = q.p;
        const int64_t t = q.t, ko = q.ko, nfull = q.nfull();
        if (g >= G || c >= K || (int64_t)p >= n_prefix || ko < 0 || nfull < 0 || ko + nfull > n_keys ||
            nfull > max_rb || t < 0 || t < tprev)
            return false;
        tprev = t;
        const int n = (int)(nfull < room ? nfull : room);
        const bool me = lane == g;

        // ---- OnRequest (Alg. 1): prior reference of (g,p), then record it.
        // Thread 0 owns the prefix bitmaps and publishes this request's two
        // bits through LDS (X.qf, written before the last barrier).  The
        // same read returns the number of table entries the previous
        // request's insert left for the displacement pass (X.novf, next to
        // X.qf): they are placed here, before this lookup reads the table.
        const uint32_t w = p >> 5, bit = 1u << (p & 31);
        const uint64_t nq = rfl64(*reinterpret_cast<const uint64_t *>(&X.novf));
        if ((uint32_t)nq != 0u) kick_pending();
        const uint32_t qf = (uint32_t)(nq >> 32);
        const bool q1 = (qf & 1u) != 0, adm = (qf & 2u) != 0;
        if (me) { c_req += 1; c_probe += (uint64_t)n; c_trunc += (uint64_t)(nfull - n); }
        const bool proven = q1 && adm;
        int64_t dg = 0;
        if constexpr (policy == kPS) dg = bcast64(me ? raw_debt(t) : 0, g);   // before this request's charge
        const bool gate_open = dg <= eps || (flags & kFlagNoGate);

        // ---- lookup, duplicates, pin + OnTouch, orphans (new blocks wait)
        PROF_MARK(0);
        int hend = n, nhit = 0, nnew = 0, ndup = 0, norph = 0;
        int npromo = 0, ngated = 0;
        // a one-step request (n <= kB) carries each position's outcome from
        // the lookup to the insertion in registers: no second pass, no
        // second ballot, and the lookup's bucket snapshot serves the insert
        uint64_t c_key = 0;
        TH c_h = {};
        uint32_t c_slot = kNoSlot, c_mt = 0, c_fm = 0;
        bool c_isN = false, c_rl = false, c_new = false;
        int c_rkN = 0, c_rkRl = 0, c_rkNew = 0, c_nmiss = 0, c_hitS = 0, c_hitM = 0;
        uint64_t kcur = kn;
        for (int base = 0; base < n; base += kB) {
            const int j = base + tid;
            const bool act = j < n;
            const uint64_t k = kcur;
            if (base + kB < n) kcur = (j + kB < n) ? tkeys[ko + j + kB] : 0ull;   // next step in flight
            const TH h = thash(k, nb, rbmask);
            // the table buckets load first: their latency overlaps the
            // duplicate-set claim below
            uint32_t te[16];
            if (act) load_buckets(table, h, te);
            // file (tag, position) in the request's duplicate set: the first
            // bucket with room along r1, r2, r2+1, ... (a claim counter each)
            uint32_t rpos = 0, nhop = 0;
            if (act) {
                if constexpr (!kHyb) rkeys[j] = k;
                uint32_t b = h.r1;
                for (;;) {
                    const uint32_t r = atomicAdd(&rcnt[b], 1u);
                    if (r < 8u) {
                        rpos = 8u * b + r;
                        rset[rpos] = (h.tag << 16) | (uint32_t)j;
                        break;
                    }
                    b = nhop == 0 ? h.r2 : ((b + 1u) & rbmask);
                    ++nhop;
                }
            }
            // resident lookup of every key (also of duplicates: harmless)
            uint32_t cand = 0, fm = 0;
            const int ntag = act ? tscan(h, te, cand, fm) : 0;
            // key, metadata and prefix id of the candidate in one round trip,
            // before the barrier: nothing writes them between the probe and
            // the ballot, except an earlier step of this request, whose slots
            // a non-duplicate key never names (a duplicate ignores them)
            uint64_t ck = 0ull;
            uint32_t cp = 0u;
            if constexpr (kPack) {   // key and prefix id: one 16-byte load
                if (ntag == 1) {
                    const GLOBAL KeyRec *rc = krec + cand;
                    ck = rc->key;
                    cp = rc->pfx;
                }
            } else {
                ck = ntag == 1 ? key[cand] : 0ull;
            }
            uint32_t mt = ntag == 1 ? meta[cand] : 0u;
            if constexpr (!kPack) cp = (policy == kPS && ntag == 1) ? pfx[cand] : 0u;
            bsync();
            // duplicate: an earlier position holds the same key.  It was filed
            // along the same bucket sequence, no later than the first bucket
            // whose counter never passed 8 (no claim ever left that bucket).
            bool dup = false;
            if (act) {
                uint32_t b = h.r1;
                for (int hop = 0;; ++hop) {
                    const uint32_t cn = rcnt[b];
                    const uint4 *q4 = reinterpret_cast<const uint4 *>(rset + 8u * b);
                    const uint4 a0 = q4[0], a1 = q4[1];
                    const uint32_t ev[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
                    // earlier positions with the key's tag (branch-free; rare),
                    // then their keys
                    uint32_t tm = 0;
#pragma unroll
                    for (int i = 0; i < 8; ++i)
                        tm |= ((ev[i] >> 16) == h.tag && (ev[i] & 0xFFFFu) < (uint32_t)j ? 1u : 0u) << i;
                    if (tm != 0u) {
#pragma unroll
                        for (int i = 0; i < 8; ++i)
                            if ((tm >> i) & 1u) dup = dup || rkey(ko, ev[i] & 0xFFFFu) == k;
                    }
                    if (dup || cn <= 8u) break;
                    b = hop == 0 ? h.r2 : ((b + 1u) & rbmask);
                }
            }
            const bool nd = act && !dup;
            int fs = (ntag == 1 && ck == k) ? (int)cand : -1;
            if (ntag > 1) {
                fs = tfind_slow(k, h);
                if (fs >= 0) mt = meta[fs];
            }
            const bool found = nd && fs >= 0;
            const uint32_t slot = (uint32_t)fs;
            uint32_t cpx = cp;
            if (policy == kPS && ntag > 1 && fs >= 0) cpx = pfx[slot];
            // Eq. 4: proven reuse of a block matching (g, c, p), not yet REUSE
            const bool eligc = policy == kPS && found && proven && (int)owner_of(mt) == g &&
                               (int)contract_of(mt) == c && cls_of(mt) != (uint32_t)kReuse && cpx == p;
            const bool inS = found && !(mt & kQMain);
            // block-wide masks: misses, found, duplicates, and the policy's
            // fourth (PrefixShield: promotion-eligible; S3-FIFO: in S)
            constexpr int kM = (policy == kPS || policy == kS3) ? 4 : 3;
            bool pa[kM];
            pa[0] = nd && !found;
            pa[1] = found;
            pa[2] = dup;
            if constexpr (policy == kPS) pa[kM - 1] = eligc;
            if constexpr (policy == kS3) pa[kM - 1] = inS;
            BMask ma[kM];
            bballot<kM>(pa, ma);
            // a one-step request leaves the set empty entry by entry
            if (n <= kB && act) {
                rset[rpos] = kEmpty;
                uint32_t b = h.r1;
                rcnt[b] = 0u;
                for (uint32_t hop = 0; hop < nhop; ++hop) {
                    b = hop == 0 ? h.r2 : ((b + 1u) & rbmask);
                    rcnt[b] = 0u;
                }
            }
            if (hend == n && ma[0].any()) hend = base + ma[0].first();
            const int lim = hend - base;   // threads below lim are in the leading run
            const bool isHit = found && tid < lim;
            const bool isOrph = found && tid >= lim;
            const bool elig = eligc && tid < lim;
            // hits and orphans leave their free queue; orphans also leave
            // their owner's resident count
            if constexpr (kQueues) wave_add(cnt, 3 * owner_of(mt) + (nseg == 1 ? 0u : cls_of(mt)), found, -1);
            wave_add(res, owner_of(mt), isOrph, -1);
            uint32_t m2 = mt | kPin;
            if (isHit) {   // pin; touch
                if constexpr (policy == kS3) {
                    const uint32_t f = freq_of(mt);
                    m2 = (m2 & ~(3u << kFreqShift)) | ((f < 3 ? f + 1 : 3u) << kFreqShift);
                } else {
                    m2 &= ~kInLog;
                    if (policy == kPS && elig && gate_open)
                        m2 = (m2 & ~(3u << kClsShift)) | ((uint32_t)kReuse << kClsShift);
                }
                meta[slot] = m2;
            }
            // orphans: the old block leaves; its slot and table entry are
            // reused by the new block of the same key
            if (isOrph) meta[slot] = kPin | (mt & ~kLowMeta);
            if (n > kB) {
                if (act) posslot[j] = dup ? kNoSlot : (found ? (uint16_t)slot : kNewMark);
            } else {
                c_key = k;
                c_h = h;
                c_fm = fm;
                c_slot = dup ? kNoSlot : (found ? slot : (uint32_t)kNewMark);
                c_mt = m2;
                c_isN = nd && !found;
                c_rl = nd;
                c_new = nd && tid >= lim;
                c_rkN = ma[0].rank(wid);
                c_nmiss = ma[0].count();
                if constexpr (policy == kS3) {
                    // new blocks: non-duplicates at or after the first miss
                    // (the non-duplicates below it are hits)
                    c_rkNew = tid - ma[2].rank(wid) - (lim - ma[2].below(lim).count());
                } else {
                    c_rkRl = tid - ma[2].rank(wid);
                }
            }
            const BMask hitm = ma[1].below(lim);
            const int nh = hitm.count(), nf = ma[1].count(), no = nf - nh;
            int ne = 0, hs = 0, os = 0;
            if constexpr (policy == kPS) ne = ma[kM - 1].below(lim).count();
            if constexpr (policy == kS3) {
                hs = ma[kM - 1].below(lim).count();
                os = ma[kM - 1].count() - hs;
            }
            nhit += nh;
            norph += no;
            nnew += (nf - nh) + ma[0].count();
            ndup += ma[2].count();
            if (gate_open) npromo += ne; else ngated += ne;
            resident -= no;
            if constexpr (policy == kS3) {
                s_unp -= hs + os;
                m_unp -= (nh - hs) + (no - os);
                s_size -= os;
            }
            c_hitS = hs;
            c_hitM = nh - hs;
        }
        if (n > kB) {   // longer requests clear the whole set (read by all steps)
            for (uint32_t i = tid; i <= rsmask; i += kB) rset[i] = kEmpty;
            for (uint32_t i = tid; i <= rbmask; i += kB) rcnt[i] = 0u;
        }
        // the next request's first keys and prefix bits, and the descriptor
        // after it, go in flight now; stores follow the loads so that waiting
        // for the loads never waits for a store.  The bitmap words go first:
        // their address needs the next request's prefix id, loaded a request
        // ago, and the compiler's wait for that load (the vector-memory
        // counter, counted in order) would otherwise also wait for the key
        // loads issued just before it.
        uint64_t knext = 0;
        uint32_t nref = 0, nadm = 0;
        if (has_next) {
            if (tid == 0) {
                const uint32_t nwd = nx.p >> 5;
                nref = bits[nwd];
                nadm = bits[npw + nwd];
            }
            knext = (tid < nx.nfull()) ? tkeys[nx.ko + tid] : 0ull;
        }
        if (r + 2 < n_req) nn = load_req(r + 2);
        if (tid == 0) {
            if (!q1) bits[w] = bref | bit;   // OnRequest: (g, p) referenced
            if (preq && r > 0) put_per_request(r - 1);
        }
        const int h = nhit, m = nnew;
        if (me) {
            c_hit += (uint64_t)h;
            c_miss += (uint64_t)(n - h);
            c_dup += (uint64_t)ndup;
            c_orph += (uint64_t)norph;
            c_promo += (uint64_t)npromo;
            c_gated += (uint64_t)ngated;
        }

        // ---- reclamation (Alg. 2): truly free blocks first
        PROF_MARK(1);
        nvict = 0;
        gseq0 = gseq;
        int e = m - (C - resident);
        if constexpr (policy == kSQ) {
            // the requester's partition: its free space is the quota less
            // its resident blocks (orphans already removed)
            bsync();
            e = m - (room - (int)rfl(res[g]));
        } else if (e > 0) {
            // the lookup's last writes (hits' metadata, queue counts) come
            // after its last barrier: make them visible to every wavefront
            bsync();
        }
        if (e < 0) e = 0;
        PROF_COUNT(0, e > 0 ? 1 : 0);
        if (e > 0) {
            if constexpr (policy == kLRU) evict_lru(e);
            else if constexpr (policy == kPS) evict_ps(e, t);
            else if constexpr (policy == kSQ) ps_take(g, -1, 3 * g, e);
            else evict_s3(e);
        }
        if (me) c_evc += (uint64_t)e;

        // ---- OnCacheFullBlocks: charge n_r = m (Eq. 2), class, admission
        PROF_MARK(2);
        uint32_t cls_new = kNormal;
        bool adm_now = adm;
        if (m > 0) {
            uint32_t cl = 0;
            if (me) {
                if (K == 1) {   // one contract (c = 0): no selection
                    const int64_t B = eff(0, t) - (int64_t)m * kScale;
                    bal[0] = B;
                    last[0] = t;
                    cl = (B < -eps || !adm) ? (uint32_t)kProb : (uint32_t)kNormal;
                } else {
#pragma unroll
                    for (int cc = 0; cc < 4; ++cc)
                        if (cc == c) {
                            const int64_t B = eff(cc, t) - (int64_t)m * kScale;
                            bal[cc] = B;
                            last[cc] = t;
                            cl = (B < -eps || !adm) ? (uint32_t)kProb : (uint32_t)kNormal;
                        }
                }
                c_charged += (uint64_t)m;
            }
            cls_new = bcast32(cl, g);
            if (tid == 0 && !adm) bits[npw + w] = badm | bit;
            adm_now = true;
        }

        // ---- insert the new blocks (never-used slots first, then the
        //      victims' slots) and release every block of the request to the
        //      free queue, deepest first -- one pass over the positions
        PROF_MARK(3);
        const int nrel = n - ndup;
        if constexpr (policy == kS3) { if (m > 0) ensure_room((uint32_t)m); }
        else if (nrel > 0) ensure_room((uint32_t)nrel);
        PROF_MARK(4);
        const uint32_t mbase = ((uint32_t)g) | ((uint32_t)c << kContractShift) | (cls_new << kClsShift) | kRes;
        const int nfresh = C - hwm;
        int nalloc = 0, seen = 0, seen_new = 0;
        if (tid == 0) X.nghost = 0;
        // A one-step insert claims table entries with counters kept in the
        // duplicate set's words (tclaim), so every wavefront must see those
        // words clear first: the lookup clears its entries after its last
        // barrier, and S3-FIFO's reclamation clears its ghost-claim counters
        // after its own last barrier.  (A longer request takes a barrier
        // before its claims, and the other policies' reclamation is preceded
        // by one.)  The barrier also orders thread 0's reset of the ghost-hit
        // count before any wavefront adds to it.
        if (n <= kB && m > 0 && (e == 0 || policy == kS3)) bsync();
        TH hh = {};
        uint32_t touched = 0;
        if (n <= kB && n > 0) {
            // one step, from the lookup's registers
            uint32_t slot = c_slot;
            // a new block's table entry: claimed now, or (both buckets full)
            // placed by the displacement pass, which records it then; an
            // orphan's slot keeps its entry
            uint32_t tpos = c_mt & ~kLowMeta;
            if (c_isN) {
                const int i = c_rkN;
                slot = new_slot(i, nfresh);
                key[slot] = c_key;
                hh = c_h;
                const uint32_t val = (hh.tag << 16) | slot;
                const uint32_t at = tclaim_m(table, rset, val, hh, c_fm, touched);
                if (at == kEmpty) defer_kick(val, c_key, true);
                tpos = at == kEmpty ? 0u : (at << kTposShift);
            }
            nalloc = c_nmiss;
            const uint32_t mt = c_new ? (mbase | tpos) : c_mt;
            if constexpr (policy == kPS) {
                if (c_new) pfx[slot] = p;
            }
            if constexpr (policy == kS3) {
                bool gh = false;
                if (c_new && g_cap > 0) gh = ghost_take(c_key);
                {
                    const uint64_t gm = ballot(gh);
                    if (lane == 0 && gm) atomicAdd(&X.nghost, (uint32_t)popc(gm));
                }
                if (c_new) {
                    const uint32_t np = tail + (uint32_t)(m - 1 - c_rkNew);
                    log[np & lmask] = (uint16_t)slot;
                    stamp[slot] = (StampT)np;
                    meta[slot] = mt | kInLog | (gh ? kQMain : 0u);
                } else if (c_rl) {
                    meta[slot] = mt & ~kPin;
                }
                s_unp += c_hitS;   // hits are unpinned where they are
                m_unp += c_hitM;
            } else if (c_rl) {
                const uint32_t np = tail + (uint32_t)(nrel - 1 - c_rkRl);
                log[np & lmask] = (uint16_t)slot;
                stamp[slot] = (StampT)np;
                meta[slot] = (mt & ~kPin) | kInLog | kRes;
            }
            if constexpr (kQueues) wave_add(cnt, 3 * owner_of(mt) + (nseg == 1 ? 0u : cls_of(mt)), c_rl, 1);
        }
        for (int base = 0; n > kB && base < n; base += kB) {
            const int j = base + tid;
            const bool act = j < n;
            uint32_t slot = act ? posslot[j] : kNoSlot;
            const bool rl = act && slot != kNoSlot;       // every non-duplicate position
            const bool isNew = rl && j >= hend;           // new block (orphans included)
            const bool isN = slot == kNewMark;            // new block without a slot yet
            // hits: their metadata; orphans: the table entry their slot keeps
            uint32_t mt = (rl && !isN) ? meta[slot] : 0u;
            // a new key reads its buckets before the barrier of the ballot
            uint64_t kk = 0;
            uint32_t e[16];
            if (isN) {
                kk = rkey(ko, (uint32_t)j);
                hh = thash(kk, nb, rbmask);
                load_buckets(table, hh, e);
            }
            bool pa[4] = {isN, rl, isNew, rl && !isNew && (mt & kQMain) != 0};
            BMask ma[4];
            bballot<4>(pa, ma);
            touched = 0;
            uint32_t tpos = mt & ~kLowMeta;
            if (isN) {
                const int i = nalloc + ma[0].rank(wid);
                slot = new_slot(i, nfresh);
                key[slot] = kk;
                const uint32_t val = (hh.tag << 16) | slot;
                const uint32_t at = tclaim(table, rset, val, hh, e, touched);
                if (at == kEmpty) defer_kick(val, kk, true);
                tpos = at == kEmpty ? 0u : (at << kTposShift);
            }
            nalloc += ma[0].count();
            if (isNew) {
                mt = mbase | tpos;
                if constexpr (policy == kPS) pfx[slot] = p;
            }
            if constexpr (policy == kS3) {
                // new blocks enter the ghost-selected queue in deepest-first
                // order; hits stay where they are; everything is unpinned
                bool gh = false;
                if (isNew && g_cap > 0) gh = ghost_take(isN ? kk : key[slot]);
                {
                    const uint64_t gm = ballot(gh);
                    if (lane == 0 && gm) atomicAdd(&X.nghost, (uint32_t)popc(gm));
                }
                if (isNew) {
                    const uint32_t np = tail + (uint32_t)(m - 1 - (seen_new + ma[2].rank(wid)));
                    log[np & lmask] = (uint16_t)slot;
                    stamp[slot] = (StampT)np;
                    meta[slot] = mt | kInLog | (gh ? kQMain : 0u);
                } else if (rl) {
                    meta[slot] = mt & ~kPin;
                }
                const int hm = ma[3].count();
                s_unp += ma[1].count() - ma[2].count() - hm;   // hits in the small queue
                m_unp += hm;
            } else if (rl) {
                const uint32_t np = tail + (uint32_t)(nrel - 1 - (seen + ma[1].rank(wid)));
                log[np & lmask] = (uint16_t)slot;
                stamp[slot] = (StampT)np;
                meta[slot] = (mt & ~kPin) | kInLog | kRes;
            }
            if constexpr (kQueues) wave_add(cnt, 3 * owner_of(mt) + (nseg == 1 ? 0u : cls_of(mt)), rl, 1);
            seen += ma[1].count();
            seen_new += ma[2].count();
            if (base + kB < n) {   // another step follows: place displaced entries first
                bsync();
                tclaim_reset(rset, hh, touched);
                kick_pending();
            }
        }
        if constexpr (policy == kS3) gsync();   // ghost-ring writes of this request are visible
        else bsync();
        tclaim_reset(rset, hh, touched);
        // entries that found both buckets full are placed by the next
        // request before its lookup (or after the last request)
        slots_taken(nalloc, nfresh);
        if (m > 0) {
            if (tid == 0) atomicAdd(&res[g], (uint32_t)m);
            resident += m;
        }
        // (one unconditional update of the log tail keeps every member of
        // the uniform state in registers)
        tail += (uint32_t)(policy == kS3 ? m : nrel);
        if constexpr (policy == kS3) {
            const int ng = (int)rfl(X.nghost);
            s_size += m - ng;
            s3_ghits += (uint64_t)ng;
            s_unp += m - ng;   // new blocks are unpinned right away
            m_unp += ng;
        }
        PROF_MARK(4);

        // ---- accounting for every group
        if (lane < G) {
            const int64_t d = raw_debt(t);
            d_sum = (int64_t)((uint64_t)d_sum + (uint64_t)d);
            if (d > d_max) d_max = d;
            const int32_t rr = (int32_t)res[lane];
            if (rr > r_max) r_max = rr;
        }
        if (resident > rmax) rmax = resident;
        last_h = h; last_m = m; last_e = e; last_o = norph;
        // prefix bits of the next request, with this request's updates
        if (has_next && (nx.p >> 5) == w) {
            nref |= bit;
            if (adm_now) nadm |= bit;
        }
        kn = knext;
        bref = nref;
        badm = nadm;
        if (tid == 0 && has_next) {
            const uint32_t nb = 1u << (nx.p & 31);
            X.qf = ((nref & nb) ? 1u : 0u) | ((nadm & nb) ? 2u : 0u);
        }
        // X.qf and all state of this request are visible (hybrid layout: the
        // new blocks' keys and prefix ids too, which the next lookup reads)
        if constexpr (kHyb) gsync();
        else bsync();
        PROF_MARK(5);
        return true;
    }

    // ============================================================ run
    DEV void init() {
        const uint32_t nte = 8u * nb;
        for (uint32_t i = tid; i < nte; i += kB) table[i] = kEmpty;
        for (int i = tid; i < C; i += kB) meta[i] = 0;
        for (int i = tid; i < 64; i += kB) res[i] = 0u;
        for (uint32_t i = tid; i <= rbmask; i += kB) rcnt[i] = 0u;
        if constexpr (kQueues)
            for (int i = tid; i < 196; i += kB) { if (i < 192) cnt[i] = 0u; cur[i] = 0u; }
        for (int i = tid; i < 2 * I.n_prefix_words; i += kB) bits[i] = 0u;
        if (policy == kS3 && g_cap > 0) {
            const uint32_t nge = 8u * gnb;
            for (uint32_t i = tid; i < nge; i += kB) gtable[i] = kEmpty;
        }
        if (tid == 0) { X.novf = 0; X.nghost = 0; X.kerr = 0; X.qf = 0; }
        for (uint32_t i = tid; i <= rsmask; i += kB) rset[i] = kEmpty;
        head = tail = 0;
        hwm = 0;
        ftop = 0;
        nvict = 0;
        resident = 0;
        s_size = s_unp = m_unp = 0;
        gseq = curS = curM = 0;
        gseq0 = 0;
        gsw = 0;
        rmax = 0;
        err = 0;
        ev_total = in_vgpr((uint64_t)0);
        s3_moves = in_vgpr((uint64_t)0);
        s3_reins = in_vgpr((uint64_t)0);
        s3_ghits = in_vgpr((uint64_t)0);
        s3_gins = in_vgpr((uint64_t)0);
        evw = 0;
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) { bal[cc] = cc < K ? beta[cc] : 0; last[cc] = 0; }
        c_req = c_probe = c_hit = c_miss = c_charged = c_evc = c_promo = c_gated = c_orph = c_dup = c_trunc = 0;
        d_max = d_sum = 0;
        r_max = 0;
        last_h = last_m = last_e = last_o = 0;
#ifdef PC_PROFILE
        if (tid < 8) { X.prof[tid] = 0; X.pcnt[tid] = 0; }
        if (tid == 0) {
            X.prof_last = X.prof_t0 = __builtin_amdgcn_s_memtime();
            X.prof_rt0 = __builtin_amdgcn_s_memrealtime();
        }
#endif
        gsync();
    }

    DEV void run(int64_t *st, int32_t *per_req) {
        preq = (per_req && I.per_req_off >= 0) ? per_req + I.per_req_off : nullptr;
        pr_next = 0;
        init();
        int32_t status = 0;
        int64_t tprev = 0, tlast = 0;
        const int64_t nreq = n_req;
        Req q = {}, nx = {};
        int64_t done = 0;
        uint64_t kn = 0;
        uint32_t bref = 0, badm = 0;
        if (nreq > 0) {
            q = load_req(0);
            if (nreq > 1) nx = load_req(1);
            kn = (q.nfull() > tid && q.ko >= 0 && q.kend <= n_keys) ? tkeys[q.ko + tid] : 0ull;
            if ((int64_t)q.p < n_prefix && tid == 0) {
                bref = bits[q.p >> 5];
                badm = bits[npw + (q.p >> 5)];
                const uint32_t nb = 1u << (q.p & 31);
                X.qf = ((bref & nb) ? 1u : 0u) | ((badm & nb) ? 2u : 0u);
            }
        }
        bsync();
        for (int64_t r = 0; r < nreq; ++r) {
            const bool has_next = r + 1 < nreq;
            // a malformed next request must not be prefetched from
            const bool nx_ok = has_next && nx.ko >= 0 && nx.nfull() >= 0 && nx.kend <= n_keys &&
                               (int64_t)nx.p < n_prefix;
            Req nn = {};
            if (!request(r, q, tprev, kn, bref, badm, nx, nx_ok, nn)) { status = -1; break; }
            ++done;
            if (err) { status = err; break; }
            tlast = tprev;
            q = nx;
            nx = nn;
        }
        // table entries the last request left for the displacement pass
        // (only their failure matters now: it is an internal error)
        kick_pending();
        if (err && status == 0) status = err;
        // the last completed request's quadruple (the others were written
        // while the request after them ran)
        if (preq && tid == 0 && done > pr_next) put_per_request(done - 1);
        X.kkey[tid] = evw;   // per-wavefront eviction counts, summed below
#ifdef PC_PROFILE
        // the instance's span on both clocks: their ratio is the shader clock
        if (tid == 0) {
            X.prof[6] = __builtin_amdgcn_s_memtime() - X.prof_t0;
            X.prof[7] = __builtin_amdgcn_s_memrealtime() - X.prof_rt0;
        }
#endif
        gsync();
        if (wid != 0) return;
        // stats record: 64 groups x 17 int64, then the instance block
        const bool ok = status == 0;
        const bool grp = lane < G;
        int64_t *o = st + lane * kGroupFields;
        const int64_t dend = (grp && ok && nreq > 0) ? raw_debt(tlast) : 0;
        const uint64_t ev_own = grp ? X.kkey[lane] + X.kkey[64 + lane] + X.kkey[128 + lane] + X.kkey[192 + lane] : 0ull;
        const uint32_t rr = grp ? res[lane] : 0u;
        const int64_t v[kGroupFields] = {(int64_t)c_req, (int64_t)c_probe, (int64_t)c_hit, (int64_t)c_miss,
                                         (int64_t)c_charged, (int64_t)ev_own, (int64_t)c_evc, (int64_t)c_promo,
                                         (int64_t)c_gated, (int64_t)c_orph, (int64_t)c_dup, (int64_t)c_trunc,
                                         dend, d_max, d_sum, (int64_t)rr, (int64_t)r_max};
#pragma unroll
        for (int f = 0; f < kGroupFields; ++f) o[f] = (ok && grp) ? v[f] : 0;
        if (lane == 0) {
            int64_t *qq = st + kInstOffset;
            qq[0] = ok ? (int64_t)ev_total : 0;
            qq[1] = ok ? (int64_t)s3_moves : 0;
            qq[2] = ok ? (int64_t)s3_reins : 0;
            qq[3] = ok ? (int64_t)s3_ghits : 0;
            qq[4] = ok ? (int64_t)s3_gins : 0;
            qq[5] = ok ? (int64_t)resident : 0;
            qq[6] = ok ? (int64_t)rmax : 0;
            qq[7] = (int64_t)(uint32_t)status;   // status in the low 32 bits
        }
#ifdef PC_PROFILE
        // phase build: the record of group 63 carries the 6 phase cycle
        // totals, the instance's span in shader cycles and in 100 MHz
        // real-time ticks, then (fields 8-11) the event counts
        if (G < 64 && lane < 8) st[63 * kGroupFields + lane] = (int64_t)X.prof[lane];
        if (G < 64 && lane < 4) st[63 * kGroupFields + 8 + lane] = (int64_t)X.pcnt[lane];
#endif
    }
};

// One instance: the compile-time copy for the default 4096-block layout when
// the host marked it (in that layout's kernel), else the general one.
template <int kLay, int kPol>
DEV void run_instance(Coll &coll, const DevInst &I, const DevTrace &T, uint8_t *sbase, uint8_t *ws, int64_t *st,
                      int32_t *per_req) {
    if constexpr (kLay != kLayWs) {
        if (I.fixc == kFixC) {
            Replayer<kLay, kPol, kFixC> rp(coll, I, T, sbase, ws);
            rp.run(st, per_req);
            return;
        }
    }
    Replayer<kLay, kPol, 0> rp(coll, I, T, sbase, ws);
    rp.run(st, per_req);
}

// One workgroup per instance.
template <int kLay>
DEV void replay_body(const DevInst *__restrict__ insts, const DevTrace *__restrict__ traces,
                     const int32_t *__restrict__ order, uint8_t *ws, int64_t *stats, int32_t *per_req) {
    extern __shared__ __align__(16) uint8_t smem[];
    __shared__ Coll coll;
    const int id = order[blockIdx.x];
    const DevInst &I = insts[id];
    const DevTrace &T = traces[I.trace];
    uint8_t *sbase;
    if constexpr (kLay == kLayWs) sbase = ws + I.ws_state;
    else sbase = smem;
    int64_t *st = stats + (int64_t)id * kRecordWords;
    if (I.policy == kLRU) run_instance<kLay, kLRU>(coll, I, T, sbase, ws, st, per_req);
    else if (I.policy == kS3) run_instance<kLay, kS3>(coll, I, T, sbase, ws, st, per_req);
    else if (I.policy == kSQ) run_instance<kLay, kSQ>(coll, I, T, sbase, ws, st, per_req);
    else run_instance<kLay, kPS>(coll, I, T, sbase, ws, st, per_req);
}
// Two instances per CU: two waves per SIMD, so at most 256 registers per
// lane.
template <int kLay>
__global__ __launch_bounds__(kB) __attribute__((amdgpu_waves_per_eu(2)))
void replay_kernel(const DevInst *__restrict__ insts, const DevTrace *__restrict__ traces,
                   const int32_t *__restrict__ order, uint8_t *ws, int64_t *stats, int32_t *per_req) {
    replay_body<kLay>(insts, traces, order, ws, stats, per_req);
}
#ifndef PC_REPLAY_GLOBAL_TU
// An instance whose LDS state takes the whole CU: no occupancy target, so
// the compiler schedules for one wave per SIMD (about 5 % less time per
// request than the same code built for two).
__global__ __launch_bounds__(kB)
void replay_kernel_solo(const DevInst *__restrict__ insts, const DevTrace *__restrict__ traces,
                        const int32_t *__restrict__ order, uint8_t *ws, int64_t *stats, int32_t *per_req) {
    replay_body<kLayLds>(insts, traces, order, ws, stats, per_req);
}
#endif

}  // namespace

// The kernels whose state is partly or wholly in global memory (hybrid and
// workspace layouts) are built in a translation unit of their own
// (pc_replay_global.hip includes this file with PC_REPLAY_GLOBAL_TU set),
// under the machine scheduler that suits them; this one holds the all-LDS
// kernels.
#ifdef PC_REPLAY_GLOBAL_TU

hipError_t replay_hybrid_set_lds_limit(int32_t lds_bytes) {
    return hipFuncSetAttribute(reinterpret_cast<const void *>(&replay_kernel<kLayHybrid>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
}

hipError_t launch_replay_global(const DevInst *d_inst, const DevTrace *d_traces, const int32_t *d_order,
                                int32_t n_launch, int32_t lds_bytes, int layout, uint8_t *ws, int64_t *stats,
                                int32_t *per_req, hipStream_t s) {
    if (layout == kLayHybrid)
        hipLaunchKernelGGL(replay_kernel<kLayHybrid>, dim3((unsigned)n_launch), dim3(kB), (size_t)lds_bytes, s,
                           d_inst, d_traces, d_order, ws, stats, per_req);
    else
        hipLaunchKernelGGL(replay_kernel<kLayWs>, dim3((unsigned)n_launch), dim3(kB), 0, s, d_inst, d_traces,
                           d_order, ws, stats, per_req);
    return hipGetLastError();
}

#else

int32_t replay_static_lds_bytes() { return (int32_t)sizeof(Coll); }

hipError_t replay_set_lds_limit(int32_t lds_bytes) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&replay_kernel<kLayLds>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
    if (e != hipSuccess) return e;
    e = hipFuncSetAttribute(reinterpret_cast<const void *>(&replay_kernel_solo),
                            hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
    if (e != hipSuccess) return e;
    return replay_hybrid_set_lds_limit(lds_bytes);
}

hipError_t launch_replay(const DevInst *d_inst, const DevTrace *d_traces, const int32_t *d_order, int32_t n_launch,
                         int32_t lds_bytes, int layout, int per_cu, uint8_t *ws, int64_t *stats, int32_t *per_req,
                         hipStream_t s) {
    if (n_launch <= 0) return hipSuccess;
    if (layout != kLayLds)
        return launch_replay_global(d_inst, d_traces, d_order, n_launch, lds_bytes, layout, ws, stats, per_req, s);
    if (per_cu == 1)
        hipLaunchKernelGGL(replay_kernel_solo, dim3((unsigned)n_launch), dim3(kB), (size_t)lds_bytes, s, d_inst,
                           d_traces, d_order, ws, stats, per_req);
    else
        hipLaunchKernelGGL(replay_kernel<kLayLds>, dim3((unsigned)n_launch), dim3(kB), (size_t)lds_bytes, s, d_inst,
                           d_traces, d_order, ws, stats, per_req);
    return hipGetLastError();
}

#endif

}  // namespace pcr
