// pc_replay.hip -- batched replay of multi-tenant prefix-cache instances on
// gfx950, one 64-lane wavefront per instance.
//
// Per request (Alg. 1 hooks and Alg. 2 reclamation of the paper):
//   OnRequest           prior-reference bit of (g,p), recorded
//   lookup              longest leading run of resident blocks; later
//                       repeats of a key inside the request are misses
//   pin + OnTouch       S3-FIFO frequency, or the debt-gated promotion of
//                       Eq. 4 using the debt before this request's charge
//   reclamation         truly free slots first, then e victims: LRU order,
//                       S3-FIFO small/main/ghost, or PrefixShield's
//                       projected-debt argmax (Eqs. 5-8) with the
//                       reuse-segmented order inside the group (Eq. 9)
//   OnCacheFullBlocks   charge n_r (Eqs. 1-2), initial class, admission
//   insert + release    new blocks take the victims' slots; every block of
//                       the request returns to the free queue deepest first
//   accounting          raw debt D_g (Eq. 3) and occupancy of every group
//
// State of one instance (capacity C, largest request n_max):
//   key[C] u64, stamp[C] u32, meta[C] u32     -- one slot per cached block
//   table[8*NB] u32  2-choice bucketized hash, entry = tag16 | slot16
//   log[R] u16       free-queue log: the slot of each appended entry; an
//                    entry at absolute position q is live iff its slot has
//                    the in-log bit and stamp == q
//   rkeys, rset, posslot, vlist   per-request keys, duplicate set,
//                    position -> slot, victims' slots
//   pfx[C] (PrefixShield), ghost table (S3-FIFO), per-group counters
// All of it sits in dynamic LDS when it fits (C up to 4096 blocks), else in
// the workspace; the code is the same, instantiated twice.  The ghost ring
// (keys of S3-FIFO's ghost entries) and the prefix bitmaps stay in HBM.
//
// Victims of one request are chosen in bulk: LRU takes the first e live log
// entries with one ballot per 64 entries; PrefixShield turns the per-victim
// argmax of Eq. 7 into runs (the winner keeps winning while its projected
// debt stays above every other candidate's) and drains each run from the
// group's per-segment cursor; S3-FIFO processes queue heads 64 at a time and
// cuts each batch where the one-at-a-time rule would switch queues.  Each
// shortcut reproduces the one-victim-at-a-time definition exactly.
#include "pc_internal.h"

namespace pcr {
namespace {

#define DEV __device__ __forceinline__

constexpr int64_t kScale = 65536;
constexpr uint16_t kNewMark = 0xFFFE;      // posslot: new block, slot not yet assigned
constexpr int32_t kErrInternal = -5;

DEV int lane_id() { return (int)__lane_id(); }
DEV uint64_t ballot(bool p) { return __ballot(p); }
DEV int popc(uint64_t m) { return __popcll(m); }
DEV int mbcnt(uint64_t m) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}
DEV int first_lane(uint64_t m) { return __ffsll((unsigned long long)m) - 1; }   // m != 0
DEV int last_lane(uint64_t m) { return 63 - __clzll((unsigned long long)m); }  // m != 0
// Lanes of one wavefront exchange data through LDS/global memory.  A wave's
// memory instructions execute in program order, so a wavefront-scope fence
// (no instruction, no wait) is enough to keep the compiler from reordering
// one lane's store after another lane's later load.
DEV void wsync() { __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront"); }
DEV uint32_t bcast32(uint32_t v, int l) { return (uint32_t)__builtin_amdgcn_readlane((int)v, l); }
DEV int64_t bcast64(int64_t v, int l) {
    uint32_t lo = bcast32((uint32_t)(uint64_t)v, l);
    uint32_t hi = bcast32((uint32_t)((uint64_t)v >> 32), l);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}
DEV uint64_t shfl64(uint64_t v, int src) {
    uint32_t lo = (uint32_t)__shfl((int)(uint32_t)v, src);
    uint32_t hi = (uint32_t)__shfl((int)(uint32_t)(v >> 32), src);
    return ((uint64_t)hi << 32) | lo;
}
DEV int64_t xor64(int64_t v, int m) {
    uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)(uint64_t)v, m);
    uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)((uint64_t)v >> 32), m);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}
DEV int64_t wave_max64(int64_t v) {
    for (int m = 32; m; m >>= 1) { int64_t u = xor64(v, m); v = u > v ? u : v; }
    return bcast64(v, 0);
}
DEV uint32_t wave_min32(uint32_t v) {
    for (int m = 32; m; m >>= 1) { uint32_t u = (uint32_t)__shfl_xor((int)v, m); v = u < v ? u : v; }
    return bcast32(v, 0);
}
DEV uint32_t wave_sum32(uint32_t v) {
    for (int m = 32; m; m >>= 1) v += (uint32_t)__shfl_xor((int)v, m);
    return bcast32(v, 0);
}
// Keep a wave-uniform value in a VGPR (it is only used in per-lane arithmetic)
// so it does not occupy scalar registers.
template <typename T>
DEV T in_vgpr(T x) {
    asm volatile("" : "+v"(x));
    return x;
}

// Key -> two buckets, 16-bit tag, duplicate-set home.  Keys are usually hash
// outputs already, but the ABI accepts any uint64, so mix with 32-bit ops.
struct TH {
    uint32_t b1, b2, tag, rhome;
};
DEV TH thash(uint64_t k, uint32_t nbmask, uint32_t rsmask) {
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
    h.b1 = x & nbmask;
    h.b2 = y & nbmask;
    if (h.b2 == h.b1) h.b2 = h.b1 ^ 1u;
    h.tag = y >> 16;
    h.rhome = (x >> 11) & rsmask;
    return h;
}

DEV uint32_t owner_of(uint32_t mt) { return mt & kOwnerMask; }
DEV uint32_t contract_of(uint32_t mt) { return (mt >> kContractShift) & 3u; }
DEV uint32_t cls_of(uint32_t mt) { return (mt >> kClsShift) & 3u; }
DEV uint32_t freq_of(uint32_t mt) { return (mt >> kFreqShift) & 3u; }

// Optional per-phase cycle accounting (build with -DPC_PROFILE); the totals
// land in the stats slot of group 63.  Nothing is skipped either way.
#ifdef PC_PROFILE
#define PROF_T(var) const uint64_t var = __builtin_amdgcn_s_memtime()
#define PROF_ADD(i, a, b) prof[i] += (b) - (a)
#else
#define PROF_T(var)
#define PROF_ADD(i, a, b)
#endif

// Descriptor of one request (loaded one request ahead).
struct Req {
    int32_t g, c;
    uint32_t p;
    int64_t t, ko, nfull;
};

template <bool kLds>
struct Replayer {
    // ---------------- configuration (wave-uniform)
    const DevInst &I;
    const DevTrace &T;
    int policy, C, flags, G, K, nseg, maxn;
    int64_t eps;
    uint32_t nbmask, rsmask, lmask, R, gnbmask, grmask;
    int32_t s_cap, g_cap, move_thr;
    int64_t rho[4], beta[4], invw[4];   // kept in VGPRs
    // ---------------- arrays
    uint64_t *key, *rkeys;
    uint32_t *stamp, *meta, *table, *rset, *cnt, *cur, *res, *pfx, *gtable;
    uint16_t *log, *posslot, *vlist;
    unsigned long long *evown;
    uint32_t *bits;
    uint64_t *gring;
    // ---------------- uniform state
    uint32_t head, tail;      // live log window [head, tail)
    int32_t hwm;              // slots [hwm, C) have never been used
    int32_t nvict;            // victims of the current request
    int32_t resident;         // resident blocks (excludes blocks being created)
    int32_t s_size, s_unp, m_unp;
    uint32_t gseq, curS, curM;
    int32_t rmax;
    int32_t err;
    // ghost ring keys prefetched for the next expiry batch
    uint64_t gpre;
    uint32_t gpre_base;
    // ---------------- statistics and group state (VGPRs; lane x = group x)
    uint64_t ev_total, s3_moves, s3_reins, s3_ghits, s3_gins;
    int64_t bal[4], last[4];
    uint64_t c_req, c_probe, c_hit, c_miss, c_charged, c_evc, c_promo, c_gated, c_orph, c_dup, c_trunc;
    int64_t d_max, d_sum;
    int32_t r_max;
    int last_h, last_m, last_e, last_o;
#ifdef PC_PROFILE
    uint64_t prof[8];
#endif

    DEV Replayer(const DevInst &inst, const DevTrace &tr, uint8_t *sbase, uint8_t *ws) : I(inst), T(tr) {
        policy = I.policy;
        C = I.capacity;
        flags = I.flags;
        G = T.n_groups;
        K = I.n_contracts;
        maxn = I.maxn;
        nseg = (policy == kPS && !(flags & kFlagNoSeg)) ? 3 : 1;
        eps = I.eps;
        nbmask = (1u << I.nb_log2) - 1u;
        rsmask = (1u << I.rs_log2) - 1u;
        R = 1u << I.log_log2;
        lmask = R - 1u;
        gnbmask = (1u << I.gnb_log2) - 1u;
        grmask = (1u << I.gr_log2) - 1u;
        s_cap = I.s_cap;
        g_cap = I.g_cap;
        move_thr = I.move_thr;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            rho[c] = in_vgpr(I.rho[c]);
            beta[c] = in_vgpr(I.beta[c]);
            invw[c] = in_vgpr(I.invw[c]);
        }
        key = reinterpret_cast<uint64_t *>(sbase + I.o_key);
        rkeys = reinterpret_cast<uint64_t *>(sbase + I.o_rkeys);
        stamp = reinterpret_cast<uint32_t *>(sbase + I.o_stamp);
        meta = reinterpret_cast<uint32_t *>(sbase + I.o_meta);
        table = reinterpret_cast<uint32_t *>(sbase + I.o_table);
        rset = reinterpret_cast<uint32_t *>(sbase + I.o_rset);
        cnt = reinterpret_cast<uint32_t *>(sbase + I.o_cnt);
        cur = reinterpret_cast<uint32_t *>(sbase + I.o_cur);
        res = reinterpret_cast<uint32_t *>(sbase + I.o_res);
        pfx = reinterpret_cast<uint32_t *>(sbase + I.o_pfx);
        gtable = reinterpret_cast<uint32_t *>(sbase + I.o_gtable);
        log = reinterpret_cast<uint16_t *>(sbase + I.o_log);
        posslot = reinterpret_cast<uint16_t *>(sbase + I.o_posslot);
        vlist = reinterpret_cast<uint16_t *>(sbase + I.o_vlist);
        evown = reinterpret_cast<unsigned long long *>(sbase + I.o_evown);
        bits = reinterpret_cast<uint32_t *>(ws + I.ws_bits);
        gring = reinterpret_cast<uint64_t *>(ws + I.ws_gring);
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
        int64_t d = 0;
#pragma unroll
        for (int c = 0; c < 4; ++c)
            if (c < K) { int64_t b = eff(c, t); if (b < 0) d -= b; }
        return d;
    }
    DEV int64_t norm_debt(int64_t t) const {  // Eq. 5, 1/w_c in Q16
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
    DEV int64_t decrement(int64_t t) const {  // Eq. 8: 1/W_g
        int64_t m = 0;
#pragma unroll
        for (int c = 0; c < 4; ++c)
            if (c < K && eff(c, t) < 0 && (m == 0 || invw[c] < m)) m = invw[c];
        return m;
    }

    // ============================================================ tables
    // Both buckets of a key: 16 entries.
    DEV void load_buckets(const uint32_t *tb, const TH &h, uint32_t e[16]) const {
        const uint4 *t4 = reinterpret_cast<const uint4 *>(tb);
        const uint4 a0 = t4[2 * h.b1], a1 = t4[2 * h.b1 + 1], c0 = t4[2 * h.b2], c1 = t4[2 * h.b2 + 1];
        e[0] = a0.x; e[1] = a0.y; e[2] = a0.z; e[3] = a0.w; e[4] = a1.x; e[5] = a1.y; e[6] = a1.z; e[7] = a1.w;
        e[8] = c0.x; e[9] = c0.y; e[10] = c0.z; e[11] = c0.w; e[12] = c1.x; e[13] = c1.y; e[14] = c1.z; e[15] = c1.w;
    }
    DEV uint32_t epos(const TH &h, int i) const { return i < 8 ? 8 * h.b1 + i : 8 * h.b2 + (i - 8); }
    // slot of key k in the main table, or -1
    DEV int tfind(uint64_t k, const TH &h) const {
        uint32_t e[16];
        load_buckets(table, h, e);
        int s = -1;
#pragma unroll
        for (int i = 0; i < 16; ++i)
            if (s < 0 && e[i] != kEmpty && (e[i] >> 16) == h.tag && key[e[i] & 0xFFFFu] == k) s = (int)(e[i] & 0xFFFFu);
        return s;
    }
    // clear the entry holding exactly `val` (if present)
    DEV void tclear_exact(uint32_t *tb, uint32_t val, const TH &h) {
        uint32_t e[16];
        load_buckets(tb, h, e);
        int at = -1;
#pragma unroll
        for (int i = 0; i < 16; ++i)
            if (at < 0 && e[i] == val) at = i;
        if (at >= 0) tb[epos(h, at)] = kEmpty;
    }
    // Parallel insert of a new entry; false when both buckets are full.
    DEV bool tinsert(uint32_t *tb, uint32_t val, const TH &h) {
        uint32_t e[16];
        load_buckets(tb, h, e);
        int n1 = 0, n2 = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) { n1 += e[i] == kEmpty; n2 += e[8 + i] == kEmpty; }
        const int first = n2 > n1 ? 8 : 0;
        for (int pass = 0; pass < 2; ++pass) {
            const int base = pass == 0 ? first : 8 - first;
            for (int w = 0; w < 8; ++w) {
                if (e[base + w] != kEmpty) continue;
                if (atomicCAS(&tb[epos(h, base + w)], kEmpty, val) == kEmpty) return true;
            }
        }
        return false;
    }
    // Serial cuckoo displacement for an entry that found both buckets full.
    template <bool kMain>
    DEV bool kick(uint32_t val, uint64_t k) {
        uint32_t *tb = kMain ? table : gtable;
        const uint32_t msk = kMain ? nbmask : gnbmask;
        uint32_t cv = val;
        uint64_t ck = k;
        uint32_t from = 0xFFFFFFFFu;
        for (int it = 0; it < 512; ++it) {
            const TH h = thash(ck, msk, rsmask);
            for (int i = 0; i < 16; ++i) {
                const uint32_t p = epos(h, i);
                if (tb[p] == kEmpty) { tb[p] = cv; return true; }
            }
            uint32_t b = (h.b1 == from) ? h.b2 : h.b1;
            if (from == 0xFFFFFFFFu && (it & 1)) b = h.b2;
            const uint32_t w = (uint32_t)(it * 5 + (uint32_t)(ck >> 7)) & 7u;
            const uint32_t victim = tb[8 * b + w];
            tb[8 * b + w] = cv;
            cv = victim;
            ck = kMain ? key[victim & 0xFFFFu] : gring[victim & grmask];
            from = b;
        }
        return false;
    }
    template <bool kMain>
    DEV void kick_lanes(uint64_t over, uint32_t val, uint64_t k) {
        wsync();
        while (over) {
            const int l = first_lane(over);
            over &= over - 1;
            const uint32_t v = bcast32(val, l);
            const uint64_t kk = (uint64_t)bcast64((int64_t)k, l);
            bool ok = true;
            if (lane_id() == 0) ok = kick<kMain>(v, kk);
            if (!bcast32(ok ? 1u : 0u, 0)) err = kErrInternal;
            wsync();
        }
    }

    // ============================================================ eviction core
    DEV void evict_lanes(bool v, uint32_t s) {
        const uint64_t vm = ballot(v);
        if (v) {
            const uint32_t mt = meta[s];
            const uint32_t o = owner_of(mt);
            atomicAdd(&evown[o], 1ull);
            atomicSub(&res[o], 1u);
            const uint64_t k = key[s];
            const TH h = thash(k, nbmask, rsmask);
            tclear_exact(table, (h.tag << 16) | s, h);
            meta[s] = 0;
            vlist[nvict + mbcnt(vm)] = (uint16_t)s;
        }
        const int nv = popc(vm);
        nvict += nv;
        resident -= nv;
        ev_total += (uint64_t)nv;
    }

    // Compaction of the free-queue log: live entries keep their order and
    // are renumbered from `head`; all cursors restart at `head`.
    DEV void compact() {
        wsync();
        const int lane = lane_id();
        uint32_t nw = head;
        for (uint32_t p0 = head; p0 < tail; p0 += 64) {
            const uint32_t pos = p0 + lane;
            const bool valid = pos < tail;
            const uint32_t s = valid ? log[pos & lmask] : 0;
            const bool live = valid && (meta[s] & kInLog) && stamp[s] == pos;
            const uint64_t lm = ballot(live);
            wsync();
            if (live) {
                const uint32_t np = nw + (uint32_t)mbcnt(lm);
                log[np & lmask] = (uint16_t)s;
                stamp[s] = np;
            }
            nw += (uint32_t)popc(lm);
            wsync();
        }
        tail = nw;
        if (policy == kPS)
            for (int i = lane; i < 196; i += 64) cur[i] = head;
        curS = curM = head;
        wsync();
    }
    DEV void ensure_room(uint32_t k) {
        if (tail + k - head <= R) return;
        if (policy == kPS) {   // lowest cursor of a non-empty queue bounds every live entry
            uint32_t m = tail;
            for (int i = lane_id(); i < 192; i += 64)
                if (cnt[i] > 0 && cur[i] < m) m = cur[i];
            m = wave_min32(m);
            if (m > head) head = m;
        } else if (policy == kS3) {
            const uint32_t m = curS < curM ? curS : curM;
            if (m > head) head = m;
        }
        if (tail + k - head > R) compact();
    }

    // ---------------------------------------------------------------- LRU
    DEV void evict_lru(int e) {
        const int lane = lane_id();
        int rem = e;
        while (rem > 0 && err == 0) {
            const uint32_t pos = head + lane;
            const bool valid = pos < tail;
            const uint32_t s = valid ? log[pos & lmask] : 0;
            const bool live = valid && (meta[s] & kInLog) && stamp[s] == pos;
            const uint64_t lm = ballot(live);
            const bool v = live && mbcnt(lm) < rem;
            const uint64_t vm = ballot(v);
            const int nv = popc(vm);
            wsync();
            evict_lanes(v, s);
            if (nv == rem) head = head + (uint32_t)last_lane(vm) + 1;
            else head = (head + 64 < tail) ? head + 64 : tail;
            rem -= nv;
            if (nv == 0 && head >= tail) err = kErrInternal;
            wsync();
        }
    }

    // ---------------------------------------------------------------- PrefixShield
    // Take k victims from queue ci in free-queue order.  x < 0: any owner;
    // s < 0: any class (no segmentation).
    DEV void ps_take(int x, int s, int ci, int k) {
        const int lane = lane_id();
        uint32_t c = cur[ci];
        int rem = k;
        while (rem > 0 && err == 0) {
            const uint32_t pos = c + lane;
            const bool valid = pos < tail;
            const uint32_t sl = valid ? log[pos & lmask] : 0;
            const uint32_t mt = valid ? meta[sl] : 0;
            const bool live = valid && (mt & kInLog) && stamp[sl] == pos;
            const bool match = live && (x < 0 || (int)owner_of(mt) == x) && (s < 0 || (int)cls_of(mt) == s);
            const uint64_t mm = ballot(match);
            const bool v = match && mbcnt(mm) < rem;
            const uint64_t vm = ballot(v);
            const int nv = popc(vm);
            wsync();
            if (v) atomicSub(&cnt[3 * owner_of(mt) + (s < 0 ? 0u : (uint32_t)s)], 1u);
            evict_lanes(v, sl);
            if (nv == rem) c = c + (uint32_t)last_lane(vm) + 1;
            else c = (c + 64 < tail) ? c + 64 : tail;
            rem -= nv;
            if (nv == 0 && c >= tail) err = kErrInternal;
            wsync();
        }
        if (lane == 0) cur[ci] = c;
        wsync();
    }
    // Oldest live entry of queue (x, s); advances that queue's cursor to it.
    DEV uint32_t ps_headpos(int x, int s) {
        const int lane = lane_id();
        const int ci = 3 * x + (s < 0 ? 0 : s);
        uint32_t c = cur[ci];
        uint32_t found = 0xFFFFFFFFu;
        while (c < tail) {
            const uint32_t pos = c + lane;
            const bool valid = pos < tail;
            const uint32_t sl = valid ? log[pos & lmask] : 0;
            const uint32_t mt = valid ? meta[sl] : 0;
            const bool live = valid && (mt & kInLog) && stamp[sl] == pos;
            const bool match = live && (int)owner_of(mt) == x && (s < 0 || (int)cls_of(mt) == s);
            const uint64_t mm = ballot(match);
            if (mm) { found = c + (uint32_t)first_lane(mm); c = found; break; }
            c = (c + 64 < tail) ? c + 64 : tail;
        }
        wsync();
        if (lane == 0) cur[ci] = c;
        wsync();
        return found;
    }
    DEV void evict_ps(int e, int64_t t) {
        const int lane = lane_id();
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
            int gs = first_lane(tied);
            if (popc(tied) > 1) {   // ties: lowest non-empty segment, then oldest head entry
                uint32_t seg = 3;
                if (grp)
                    for (int s = nseg - 1; s >= 0; --s)
                        if (cnt[3 * lane + s] > 0) seg = (uint32_t)s;
                const int mseg = (int)wave_min32(((tied >> lane) & 1) ? seg : 3u);
                tied &= ballot(seg == (uint32_t)mseg);
                gs = first_lane(tied);
                if (popc(tied) > 1) {
                    uint32_t best = 0xFFFFFFFFu;
                    for (uint64_t tm = tied; tm; tm &= tm - 1) {
                        const int x = first_lane(tm);
                        const uint32_t hp = ps_headpos(x, nseg == 1 ? -1 : mseg);
                        if (hp < best) { best = hp; gs = x; }
                    }
                }
            }
            const int64_t Pg = bcast64(P, gs), Dg = bcast64(D, gs);
            const int ag = (int)bcast32(avail, gs);
            const int64_t p2 = wave_max64((inE && lane != gs) ? P : -1);
            const int64_t thr = p2 > eps ? p2 : eps;
            // g* keeps winning strictly while P - i*D > max(second, eps)
            const int64_t k1 = Pg > thr ? (Pg - thr + Dg - 1) / Dg : 0;
            int64_t k = k1 > 1 ? k1 : 1;
            if (k > rem) k = rem;
            if (k > ag) k = ag;
            if (nseg == 1) {
                ps_take(gs, -1, 3 * gs, (int)k);
            } else {
                int kk = (int)k;
                for (int s = 0; s < 3 && kk > 0; ++s) {
                    const int cs = (int)cnt[3 * gs + s];
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
    DEV void ghost_prefetch() {
        if (g_cap > 0) {
            gpre_base = gseq;
            gpre = gring[(gseq - (uint32_t)g_cap + (uint32_t)lane_id()) & grmask];
        }
    }
    // Ghost insertion of the keys of lanes `v`, in lane order.  The ghost
    // keeps the last g_cap insertions: entries older than the batch that
    // leave the window are removed, and batch entries that would already
    // have left it by the batch's end are never inserted.
    DEV void ghost_insert(bool v, uint64_t k) {
        const uint64_t vm = ballot(v);
        const int nv = popc(vm);
        s3_gins += (uint64_t)nv;
        if (g_cap > 0 && nv > 0) {
            const int rk = mbcnt(vm);
            const uint32_t seq = gseq + (uint32_t)rk;
            const uint32_t gend = gseq + (uint32_t)nv;
            const uint64_t kpre = shfl64(gpre, rk);   // gring[(seq - g_cap) & grmask], prefetched
            if (v && (int64_t)seq >= (int64_t)g_cap) {
                const uint32_t x = seq - (uint32_t)g_cap;
                if (x < gseq) {
                    const uint32_t xp = x & grmask;
                    const uint64_t kx = gpre_base == gseq ? kpre : gring[xp];
                    const TH hx = thash(kx, gnbmask, rsmask);
                    tclear_exact(gtable, (hx.tag << 16) | xp, hx);
                }
            }
            wsync();
            const bool ins = v && (int64_t)seq + g_cap >= (int64_t)gend;
            const TH h = thash(k, gnbmask, rsmask);
            const uint32_t val = (h.tag << 16) | (seq & grmask);
            bool ok = true;
            if (v) gring[seq & grmask] = k;
            if (ins) ok = tinsert(gtable, val, h);
            const uint64_t over = ballot(ins && !ok);
            if (over) kick_lanes<false>(over, val, k);
            wsync();
            gseq += (uint32_t)nv;
            ghost_prefetch();
        } else {
            gseq += (uint32_t)nv;
        }
    }
    // ghost hit for key k: remove it and report true
    DEV bool ghost_take(uint64_t k) {
        const TH h = thash(k, gnbmask, rsmask);
        uint32_t e[16];
        load_buckets(gtable, h, e);
        int at = -1;
        for (int i = 0; i < 16; ++i)
            if (at < 0 && e[i] != kEmpty && (e[i] >> 16) == h.tag && gring[e[i] & grmask] == k) at = i;
        if (at >= 0) gtable[epos(h, at)] = kEmpty;
        return at >= 0;
    }
    DEV void evict_s3(int e) {
        const int lane = lane_id();
        const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
        int rem = e;
        uint32_t spS = curS, spM = curM;
        uint32_t keptS = 0xFFFFFFFFu, keptM = 0xFFFFFFFFu;
        while (rem > 0 && err == 0) {
            if (tail + 64 - head > R) {
                ensure_room(64);
                spS = curS; spM = curM;
                keptS = keptM = 0xFFFFFFFFu;
            }
            const bool useS = (s_size >= s_cap && s_unp > 0) || (m_unp == 0);
            const uint32_t sp = useS ? spS : spM;
            const uint32_t lim = tail;
            if (sp >= lim) { err = kErrInternal; break; }
            const uint32_t pos = sp + lane;
            const bool valid = pos < lim;
            const uint32_t sl = valid ? log[pos & lmask] : 0;
            const uint32_t mt = valid ? meta[sl] : 0;
            const bool live = valid && (mt & kInLog) && stamp[sl] == pos;
            const bool inQ = live && (useS ? !(mt & kQMain) : (mt & kQMain) != 0);
            const bool cand = inQ && !(mt & kPin);
            const uint64_t candm = ballot(cand);
            const int crk = mbcnt(candm);
            const uint32_t f = freq_of(mt);
            bool ok;
            bool mv;
            if (useS) {   // small queue: move (accessed) or evict into the ghost
                mv = cand && (int)f >= move_thr;
                const uint64_t mvm = ballot(mv);
                const int mb = popc(mvm & below);
                const int eb = popc(candm & ~mvm & below);
                const bool useS_i = (s_size - crk >= s_cap && s_unp - crk > 0) || (m_unp + mb == 0);
                ok = cand && useS_i && eb < rem;
            } else {      // main queue: reinsert (freq > 0) or evict
                mv = cand && f > 0;
                const uint64_t mvm = ballot(mv);
                const int eb = popc(candm & ~mvm & below);
                ok = cand && eb < rem && (m_unp - eb) > 0;
            }
            const uint64_t bad = candm & ~ballot(ok);
            const int stop = bad ? first_lane(bad) : 64;
            const bool proc = cand && lane < stop;
            const bool pmove = proc && mv, pev = proc && !mv;
            const uint64_t pmm = ballot(pmove), pem = ballot(pev);
            const int nmv = popc(pmm), nev = popc(pem);
            // live entries of this queue that stay behind the scan point
            const uint64_t km = ballot(inQ && !proc && lane < stop) | (bad ? (1ull << stop) : 0ull);
            if (km) {
                const uint32_t kp = sp + (uint32_t)first_lane(km);
                if (useS) { if (kp < keptS) keptS = kp; } else { if (kp < keptM) keptM = kp; }
            }
            wsync();
            // moves / reinsertions: append to the log tail in queue order
            if (pmove) {
                const uint32_t np = tail + (uint32_t)mbcnt(pmm);
                log[np & lmask] = (uint16_t)sl;
                stamp[sl] = np;
                uint32_t m2 = mt & ~(3u << kFreqShift);
                if (useS) m2 |= kQMain;
                else m2 |= (f - 1) << kFreqShift;
                meta[sl] = m2;
            }
            tail += (uint32_t)nmv;
            if (useS) {
                ghost_insert(pev, key[sl]);
                s_size -= nmv + nev;
                s_unp -= nmv + nev;
                m_unp += nmv;
                s3_moves += (uint64_t)nmv;
            } else {
                m_unp -= nev;
                s3_reins += (uint64_t)nmv;
            }
            evict_lanes(pev, sl);
            rem -= nev;
            const uint32_t adv = stop < 64 ? (uint32_t)stop : ((lim - sp) < 64 ? (lim - sp) : 64u);
            if (adv == 0) err = kErrInternal;   // a scan that cannot advance is a bug, never a hang
            if (useS) spS = sp + adv; else spM = sp + adv;
            wsync();
        }
        curS = keptS < spS ? keptS : spS;
        curM = keptM < spM ? keptM : spM;
        const uint32_t m = curS < curM ? curS : curM;
        if (m > head) head = m;
    }

    // ============================================================ one request
    DEV Req load_req(int64_t r) const {
        Req q;
        q.g = T.group[r];
        q.c = T.contract[r];
        q.p = T.prefix[r];
        q.t = T.tick ? T.tick[r] : r;
        q.ko = T.key_off[r];
        q.nfull = T.key_off[r + 1] - q.ko;
        return q;
    }

    // `kn` holds keys[ko + lane] of this request and bref/badm its prefix
    // bitmap words (all prefetched); on return they hold the same for `nx`.
    DEV bool request(int64_t r, const Req &q, int64_t &tprev, uint64_t &kn, uint32_t &bref, uint32_t &badm,
                     const Req &nx, bool has_next) {
        PROF_T(p0);
        const int lane = lane_id();
        const int g = q.g, c = q.c;
        const uint32_t p = q.p;
        const int64_t t = q.t, ko = q.ko, nfull = q.nfull;
        if (g >= G || c >= K || (int64_t)p >= T.n_prefix || ko < 0 || nfull < 0 || ko + nfull > T.n_keys ||
            nfull > T.max_req_blocks || t < 0 || t < tprev)
            return false;
        tprev = t;
        const int n = (int)(nfull < C ? nfull : C);
        const bool me = lane == g;

        // ---- OnRequest (Alg. 1): prior reference of (g,p), then record it
        const uint32_t w = p >> 5, bit = 1u << (p & 31);
        const bool q1 = (bref & bit) != 0, adm = (badm & bit) != 0;
        if (lane == 0 && !q1) bits[w] = bref | bit;
        if (me) { c_req += 1; c_probe += (uint64_t)n; c_trunc += (uint64_t)(nfull - n); }
        const bool proven = q1 && adm;
        int64_t dg = 0;
        if (policy == kPS) dg = bcast64(me ? raw_debt(t) : 0, g);   // before this request's charge
        const bool gate_open = dg <= eps || (flags & kFlagNoGate);

        // ---- lookup, duplicates, pin + OnTouch, orphans (new blocks wait)
        PROF_T(p1);
        PROF_ADD(0, p0, p1);
        for (uint32_t i = lane; i <= rsmask; i += 64) rset[i] = kEmpty;
        wsync();
        int hend = n, nhit = 0, nnew = 0, ndup = 0, norph = 0;
        int npromo = 0, ngated = 0;
        uint64_t kcur = kn;
        for (int base = 0; base < n; base += 64) {
            const int j = base + lane;
            const bool act = j < n;
            const uint64_t k = kcur;
            if (base + 64 < n) kcur = (j + 64 < n) ? T.keys[ko + j + 64] : 0ull;   // next chunk in flight
            const TH h = thash(k, nbmask, rsmask);
            const uint32_t mine = (h.tag << 16) | (uint32_t)j;
            uint32_t rpos = 0;
            if (act) {   // first occurrence in the request keeps the smallest position
                rkeys[j] = k;
                uint32_t idx = h.rhome;
                for (;;) {
                    const uint32_t old = atomicCAS(&rset[idx], kEmpty, mine);
                    if (old == kEmpty) { rpos = idx; break; }
                    if ((old >> 16) == h.tag && rkeys[old & 0xFFFFu] == k) {
                        atomicMin(&rset[idx], mine);
                        rpos = idx;
                        break;
                    }
                    idx = (idx + 1) & rsmask;
                }
            }
            wsync();
            const bool dup = act && rset[rpos] != mine;
            const bool nd = act && !dup;
            const int fs = nd ? tfind(k, h) : -1;
            const bool found = fs >= 0;
            const uint64_t missm = ballot(nd && !found);
            if (hend == n && missm) hend = base + first_lane(missm);
            const bool isHit = found && j < hend;
            const bool isOrph = found && j >= hend;
            const uint32_t slot = (uint32_t)fs;
            const uint32_t mt = found ? meta[slot] : 0u;
            // Eq. 4: proven reuse of a block matching (g, c, p), not yet REUSE
            bool elig = false;
            if (policy == kPS && isHit && proven && (int)owner_of(mt) == g && (int)contract_of(mt) == c &&
                cls_of(mt) != (uint32_t)kReuse)
                elig = pfx[slot] == p;
            if (policy == kPS) {
                const int ne = popc(ballot(elig));
                if (gate_open) npromo += ne; else ngated += ne;
            }
            if (isHit) {   // pin; touch
                uint32_t m2 = mt | kPin;
                if (policy == kS3) {
                    const uint32_t f = freq_of(mt);
                    m2 = (m2 & ~(3u << kFreqShift)) | ((f < 3 ? f + 1 : 3u) << kFreqShift);
                } else {
                    m2 &= ~kInLog;
                    if (policy == kPS) {
                        atomicSub(&cnt[3 * owner_of(mt) + (nseg == 1 ? 0u : cls_of(mt))], 1u);
                        if (elig && gate_open) m2 = (m2 & ~(3u << kClsShift)) | ((uint32_t)kReuse << kClsShift);
                    }
                }
                meta[slot] = m2;
            }
            if (policy == kS3) {
                const bool inM = (mt & kQMain) != 0;
                const int hs = popc(ballot(isHit && !inM)), hm = popc(ballot(isHit && inM));
                const int os = popc(ballot(isOrph && !inM)), om = popc(ballot(isOrph && inM));
                s_unp -= hs + os;
                m_unp -= hm + om;
                s_size -= os;
            }
            // orphans: the old block leaves; its slot and table entry are
            // reused by the new block of the same key
            if (isOrph) {
                const uint32_t o = owner_of(mt);
                atomicSub(&res[o], 1u);
                if (policy == kPS) atomicSub(&cnt[3 * o + (nseg == 1 ? 0u : cls_of(mt))], 1u);
                meta[slot] = kPin;
            }
            if (act) posslot[j] = dup ? kNoSlot : (found ? (uint16_t)slot : kNewMark);
            const int no = popc(ballot(isOrph));
            norph += no;
            resident -= no;
            nhit += popc(ballot(isHit));
            nnew += popc(ballot(nd && !isHit));
            ndup += popc(ballot(dup));
            wsync();
        }
        // the next request's first 64 keys and prefix bits go in flight now
        uint64_t knext = 0;
        uint32_t nref = 0, nadm = 0;
        if (has_next) {
            knext = (lane < nx.nfull) ? T.keys[nx.ko + lane] : 0ull;
            const uint32_t nwd = nx.p >> 5;
            nref = bits[nwd];
            nadm = bits[I.n_prefix_words + nwd];
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
        PROF_T(p2);
        PROF_ADD(1, p1, p2);
        nvict = 0;
        int e = m - (C - resident);
        if (e < 0) e = 0;
        if (e > 0) {
            if (policy == kLRU) evict_lru(e);
            else if (policy == kPS) evict_ps(e, t);
            else evict_s3(e);
        }
        if (me) c_evc += (uint64_t)e;

        // ---- OnCacheFullBlocks: charge n_r = m (Eq. 2), class, admission
        PROF_T(p3);
        PROF_ADD(2, p2, p3);
        uint32_t cls_new = kNormal;
        bool adm_now = adm;
        if (m > 0) {
            uint32_t cl = 0;
            if (me) {
#pragma unroll
                for (int cc = 0; cc < 4; ++cc)
                    if (cc == c) {
                        const int64_t B = eff(cc, t) - (int64_t)m * kScale;
                        bal[cc] = B;
                        last[cc] = t;
                        cl = (B < -eps || !adm) ? (uint32_t)kProb : (uint32_t)kNormal;
                    }
                c_charged += (uint64_t)m;
            }
            cls_new = bcast32(cl, g);
            if (lane == 0 && !adm) bits[I.n_prefix_words + w] = badm | bit;
            adm_now = true;
        }

        // ---- insert the new blocks: never-used slots first, then the
        //      victims' slots; queue order is deepest first
        PROF_T(p4);
        PROF_ADD(3, p3, p4);
        if (policy == kS3 && m > 0) ensure_room((uint32_t)m);
        const uint32_t mbase = ((uint32_t)g) | ((uint32_t)c << kContractShift) | (cls_new << kClsShift) | kRes | kPin;
        const int nfresh = C - hwm;
        int before = 0, nalloc = 0;
        int n_ins_S = 0, n_ins_M = 0;
        for (int base = hend; base < n; base += 64) {
            const int j = base + lane;
            const bool act = j < n;
            uint32_t slot = act ? posslot[j] : kNoSlot;
            const bool isN = slot == kNewMark;
            const uint64_t am = ballot(isN);
            uint64_t kk = 0;
            if (isN) {
                const int i = nalloc + mbcnt(am);
                slot = i < nfresh ? (uint32_t)(hwm + i) : vlist[i - nfresh];
                kk = rkeys[j];
                key[slot] = kk;
                posslot[j] = (uint16_t)slot;
            }
            nalloc += popc(am);
            const bool nw = act && slot != kNoSlot;
            const uint64_t nm = ballot(nw);
            if (nw) {
                meta[slot] = mbase;
                if (policy == kPS) pfx[slot] = p;
            }
            bool ok = true;
            uint32_t val = 0;
            if (isN) {
                const TH hh = thash(kk, nbmask, rsmask);
                val = (hh.tag << 16) | slot;
                ok = tinsert(table, val, hh);
            }
            const uint64_t over = ballot(isN && !ok);
            if (over) kick_lanes<true>(over, val, kk);
            if (policy == kS3) {
                bool gh = false;
                if (nw && g_cap > 0) gh = ghost_take(isN ? kk : key[slot]);
                const uint32_t rank = (uint32_t)(m - 1 - (before + mbcnt(nm)));
                if (nw) {
                    const uint32_t np = tail + rank;
                    log[np & lmask] = (uint16_t)slot;
                    stamp[slot] = np;
                    meta[slot] = mbase | kInLog | (gh ? kQMain : 0u);
                }
                const int ng = popc(ballot(nw && gh));
                n_ins_M += ng;
                n_ins_S += popc(nm) - ng;
            }
            before += popc(nm);
            wsync();
        }
        hwm += nalloc < nfresh ? nalloc : nfresh;
        if (m > 0) {
            if (lane == 0) atomicAdd(&res[g], (uint32_t)m);
            resident += m;
            if (policy == kS3) {
                tail += (uint32_t)m;
                s_size += n_ins_S;
                s3_ghits += (uint64_t)n_ins_M;
            }
        }
        wsync();

        // ---- release: back to the free queue, deepest first
        PROF_T(p5);
        PROF_ADD(4, p4, p5);
        const int nrel = n - ndup;
        if (policy != kS3 && nrel > 0) ensure_room((uint32_t)nrel);
        int seen = 0;
        for (int base = 0; base < n; base += 64) {
            const int j = base + lane;
            const bool act = j < n;
            const uint32_t slot = act ? posslot[j] : kNoSlot;
            const bool rl = act && slot != kNoSlot;
            const uint64_t rm = ballot(rl);
            const uint32_t mt = rl ? meta[slot] : 0u;
            if (policy == kS3) {
                const bool inM = (mt & kQMain) != 0;
                if (rl) meta[slot] = mt & ~kPin;
                s_unp += popc(ballot(rl && !inM));
                m_unp += popc(ballot(rl && inM));
            } else if (rl) {
                const uint32_t np = tail + (uint32_t)(nrel - 1 - (seen + mbcnt(rm)));
                log[np & lmask] = (uint16_t)slot;
                stamp[slot] = np;
                meta[slot] = (mt & ~kPin) | kInLog | kRes;
                if (policy == kPS) atomicAdd(&cnt[3 * owner_of(mt) + (nseg == 1 ? 0u : cls_of(mt))], 1u);
            }
            seen += popc(rm);
        }
        if (policy != kS3) tail += (uint32_t)nrel;
        wsync();

        // ---- accounting for every group
        PROF_T(p6);
        PROF_ADD(5, p5, p6);
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
        PROF_T(p7);
        PROF_ADD(6, p6, p7);
        return true;
    }

    // ============================================================ run
    DEV void init() {
        const int lane = lane_id();
        const uint32_t nte = 8u * (nbmask + 1u);
        for (uint32_t i = lane; i < nte; i += 64) table[i] = kEmpty;
        for (int i = lane; i < C; i += 64) meta[i] = 0;
        for (int i = lane; i < 64; i += 64) { evown[i] = 0ull; res[i] = 0u; }
        if (policy == kPS)
            for (int i = lane; i < 196; i += 64) { if (i < 192) cnt[i] = 0u; cur[i] = 0u; }
        for (int i = lane; i < 2 * I.n_prefix_words; i += 64) bits[i] = 0u;
        if (policy == kS3 && g_cap > 0) {
            const uint32_t nge = 8u * (gnbmask + 1u);
            for (uint32_t i = lane; i < nge; i += 64) gtable[i] = kEmpty;
        }
        head = tail = 0;
        hwm = 0;
        nvict = 0;
        resident = 0;
        s_size = s_unp = m_unp = 0;
        gseq = curS = curM = 0;
        gpre = 0;
        gpre_base = 0xFFFFFFFFu;
        rmax = 0;
        err = 0;
        ev_total = in_vgpr((uint64_t)0);
        s3_moves = in_vgpr((uint64_t)0);
        s3_reins = in_vgpr((uint64_t)0);
        s3_ghits = in_vgpr((uint64_t)0);
        s3_gins = in_vgpr((uint64_t)0);
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) { bal[cc] = cc < K ? beta[cc] : 0; last[cc] = 0; }
        c_req = c_probe = c_hit = c_miss = c_charged = c_evc = c_promo = c_gated = c_orph = c_dup = c_trunc = 0;
        d_max = d_sum = 0;
        r_max = 0;
        last_h = last_m = last_e = last_o = 0;
#ifdef PC_PROFILE
        for (int i = 0; i < 8; ++i) prof[i] = 0;
#endif
        wsync();
    }

    DEV void run(int64_t *st, int32_t *per_req) {
        init();
        const int lane = lane_id();
        int32_t status = 0;
        int64_t tprev = 0, tlast = 0;
        const int64_t nreq = T.n_req;
        Req q = {};
        uint64_t kn = 0;
        uint32_t bref = 0, badm = 0;
        if (nreq > 0) {
            q = load_req(0);
            kn = (q.nfull > lane && q.ko >= 0 && q.ko + q.nfull <= T.n_keys) ? T.keys[q.ko + lane] : 0ull;
            if ((int64_t)q.p < T.n_prefix) {
                bref = bits[q.p >> 5];
                badm = bits[I.n_prefix_words + (q.p >> 5)];
            }
        }
        for (int64_t r = 0; r < nreq; ++r) {
            const bool has_next = r + 1 < nreq;
            Req nx = {};
            if (has_next) nx = load_req(r + 1);
            // a malformed next request must not be prefetched from
            const bool nx_ok = has_next && nx.ko >= 0 && nx.nfull >= 0 && nx.ko + nx.nfull <= T.n_keys &&
                               (int64_t)nx.p < T.n_prefix;
            if (!request(r, q, tprev, kn, bref, badm, nx, nx_ok)) { status = -1; break; }
            if (err) { status = err; break; }
            tlast = tprev;
            if (per_req && I.per_req_off >= 0 && lane == 0) {
                int32_t *o = per_req + I.per_req_off + 4 * r;
                o[0] = last_h; o[1] = last_m; o[2] = last_e; o[3] = last_o;
            }
            q = nx;
        }
        wsync();
        // stats record: 64 groups x 17 int64, then the instance block
        const bool ok = status == 0;
        const bool grp = lane < G;
        int64_t *o = st + lane * kGroupFields;
        const int64_t dend = (grp && ok && nreq > 0) ? raw_debt(tlast) : 0;
        const uint64_t ev_own = grp ? evown[lane] : 0ull;
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
        if (lane < 8) st[63 * kGroupFields + lane] = (int64_t)prof[lane];
#endif
    }
};

template <bool kLds>
__global__ __launch_bounds__(64) void replay_kernel(const DevInst *__restrict__ insts,
                                                    const DevTrace *__restrict__ traces,
                                                    const int32_t *__restrict__ order, uint8_t *ws,
                                                    int64_t *stats, int32_t *per_req) {
    extern __shared__ __align__(16) uint8_t smem[];
    const int id = order[blockIdx.x];
    const DevInst &I = insts[id];
    const DevTrace &T = traces[I.trace];
    uint8_t *sbase;
    if constexpr (kLds) sbase = smem;
    else sbase = ws + I.ws_state;
    Replayer<kLds> rp(I, T, sbase, ws);
    rp.run(stats + (int64_t)id * kRecordWords, per_req);
}

}  // namespace

hipError_t launch_replay(const DevInst *d_inst, const DevTrace *d_traces, const int32_t *d_order, int32_t n_launch,
                         int32_t lds_bytes, bool in_lds, uint8_t *ws, int64_t *stats, int32_t *per_req,
                         hipStream_t s) {
    if (n_launch <= 0) return hipSuccess;
    if (in_lds) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&replay_kernel<true>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(replay_kernel<true>, dim3((unsigned)n_launch), dim3(64), (size_t)lds_bytes, s, d_inst,
                           d_traces, d_order, ws, stats, per_req);
    } else {
        hipLaunchKernelGGL(replay_kernel<false>, dim3((unsigned)n_launch), dim3(64), 0, s, d_inst, d_traces,
                           d_order, ws, stats, per_req);
    }
    return hipGetLastError();
}

}  // namespace pcr
