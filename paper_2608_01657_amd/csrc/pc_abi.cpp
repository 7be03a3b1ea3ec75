// pc_abi.cpp -- the C ABI of libpcreplay (declared in include/pc.h): host
// validation, workspace planning, descriptor upload and kernel launches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "pc.h"
#include "pc_internal.h"

namespace {

thread_local std::string g_err;

int32_t fail(int32_t code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}
int32_t ok() {
    g_err.clear();
    return PC_OK;
}
int32_t hip_fail(hipError_t e, const char *what) {
    return fail(PC_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

int ceil_log2(int64_t v) {
    int b = 0;
    while (((int64_t)1 << b) < v) ++b;
    return b;
}
int64_t align_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

// LDS of one CU on the current device (cached per device): the most one
// workgroup may allocate.  Without a device (host-only planning), that of
// gfx950, the one target of this library: 160 KiB.
constexpr int64_t kGfx950LdsPerCu = 160 * 1024;
int64_t lds_per_cu() {
    static std::mutex mu;
    static int64_t cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return kGfx950LdsPerCu;
    std::lock_guard<std::mutex> lk(mu);
    if (cache[dev] == 0) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess || v <= 0)
            v = (int)kGfx950LdsPerCu;
        cache[dev] = v;
    }
    return cache[dev];
}

// Compute units of the current device (cached per device); without a
// device, the 256 of an MI355X.
int64_t cu_count() {
    static std::mutex mu;
    static int64_t cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    std::lock_guard<std::mutex> lk(mu);
    if (cache[dev] == 0) {
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
        cache[dev] = v;
    }
    return cache[dev];
}

// One kernel launch: instances of one layout whose LDS footprints allow the
// same number of workgroups per CU, with the LDS of the largest of them.
struct Launch {
    int layout = pcr::kLayLds;
    int per_cu = 0;
    int32_t lds_bytes = 0;
    int32_t first = 0, count = 0;    // range of Plan::order
    double cost = 0;                 // of its costliest instance
    double est = 0;                  // estimated duration (cost units), see validate_and_plan
};

struct Plan {
    std::vector<pcr::DevInst> di;
    std::vector<pcr::DevTrace> dt;
    std::vector<int32_t> order;      // instances, launch by launch, costliest first
    std::vector<Launch> launches;    // costliest launch (and fewest per CU) first
    int32_t lds_bytes = 0;           // largest dynamic LDS of any launch
    int64_t hdr_bytes = 0;
    int64_t ws_bytes = 0;
};

constexpr int64_t kMaxRho = (int64_t)1 << 40;
constexpr int64_t kMaxBeta = (int64_t)1 << 50;

int32_t validate_and_plan(const pc_trace_desc *traces, int32_t n_traces, const pc_instance_desc *inst,
                          int32_t n_inst, int64_t lds_cu, int64_t n_cu, Plan &P) {
    if (n_traces < 0 || n_inst < 0) return fail(PC_EINVAL, "negative count");
    if ((n_traces > 0 && !traces) || (n_inst > 0 && !inst)) return fail(PC_EINVAL, "null descriptor array");
    P.dt.resize(n_traces);
    for (int i = 0; i < n_traces; ++i) {
        const pc_trace_desc &t = traces[i];
        if (t.n_req < 0 || t.n_keys < 0 || t.n_prefix < 0 || t.max_req_blocks < 0)
            return fail(PC_EINVAL, "trace %d: negative size", i);
        if (t.n_groups < 1 || t.n_groups > PC_MAX_GROUPS)
            return fail(PC_EINVAL, "trace %d: n_groups %d outside 1..64", i, t.n_groups);
        if (t.n_req > 0 && (!t.d_key_off || !t.d_group || !t.d_contract || !t.d_prefix))
            return fail(PC_EINVAL, "trace %d: null request array", i);
        if (t.n_keys > 0 && !t.d_keys) return fail(PC_EINVAL, "trace %d: null keys", i);
        if (t.n_req > 0 && t.n_prefix < 1) return fail(PC_EINVAL, "trace %d: n_prefix must be >= 1", i);
        if (t.n_prefix > ((int64_t)1 << 32)) return fail(PC_EINVAL, "trace %d: n_prefix too large", i);
        pcr::DevTrace &d = P.dt[i];
        d.keys = t.d_keys;
        d.key_off = t.d_key_off;
        d.group = t.d_group;
        d.contract = t.d_contract;
        d.prefix = t.d_prefix;
        d.tick = t.d_tick;
        d.n_req = t.n_req;
        d.n_keys = t.n_keys;
        d.n_prefix = t.n_prefix;
        d.n_groups = t.n_groups;
        d.max_req_blocks = t.max_req_blocks;
    }
    P.di.resize(n_inst);
    std::vector<int64_t> state_ws(n_inst, 0);
    int64_t off = 0;
    // header: DevInst[], DevTrace[], order[]
    off = align_up(off + (int64_t)sizeof(pcr::DevInst) * n_inst, 256);
    off = align_up(off + (int64_t)sizeof(pcr::DevTrace) * n_traces, 256);
    off = align_up(off + (int64_t)sizeof(int32_t) * n_inst, 256);
    P.hdr_bytes = off;
    int64_t per_req = 0;
    std::vector<double> cost(n_inst, 0.0);
    std::vector<int> per_cu(n_inst, 0);
    std::vector<pcr::StatePlan> plan_lds(n_inst), plan_hyb(n_inst), plan_ws(n_inst);
    for (int i = 0; i < n_inst; ++i) {
        const pc_instance_desc &s = inst[i];
        if (s.trace < 0 || s.trace >= n_traces) return fail(PC_EINVAL, "instance %d: trace index %d", i, s.trace);
        if (s.policy < PC_LRU || s.policy > PC_STATICQUOTA) return fail(PC_EINVAL, "instance %d: policy %d", i, s.policy);
        if (s.capacity < 1 || s.capacity > PC_MAX_CAPACITY)
            return fail(PC_EINVAL, "instance %d: capacity %d outside 1..%d", i, s.capacity, PC_MAX_CAPACITY);
        if (s.flags & ~(PC_FLAG_NO_SEGMENTATION | PC_FLAG_NO_DEBT_GATE))
            return fail(PC_EINVAL, "instance %d: unknown flags 0x%x", i, s.flags);
        if (s.n_contracts < 1 || s.n_contracts > PC_MAX_CONTRACTS)
            return fail(PC_EINVAL, "instance %d: n_contracts %d outside 1..4", i, s.n_contracts);
        if (s.s3_small_permille < 0 || s.s3_small_permille > 1000 || s.s3_move_threshold < 0)
            return fail(PC_EINVAL, "instance %d: S3-FIFO parameters", i);
        if (s.reserved != 0) return fail(PC_EINVAL, "instance %d: reserved field must be 0", i);
        if (s.eps_q16 < 0 || s.eps_q16 > kMaxBeta) return fail(PC_EINVAL, "instance %d: eps_q16 out of range", i);
        const pc_trace_desc &t = traces[s.trace];
        pcr::DevInst &d = P.di[i];
        std::memset(&d, 0, sizeof(d));
        d.trace = s.trace;
        d.policy = s.policy;
        d.capacity = s.capacity;
        d.flags = s.flags;
        d.n_contracts = s.n_contracts;
        d.eps = s.eps_q16;
        int64_t rmin = 0;
        for (int c = 0; c < s.n_contracts; ++c) {
            if (s.contract[c].rho_q16 <= 0 || s.contract[c].rho_q16 > kMaxRho)
                return fail(PC_EINVAL, "instance %d contract %d: rho_q16 must be in 1..2^40", i, c);
            if (s.contract[c].beta_q16 < 0 || s.contract[c].beta_q16 > kMaxBeta)
                return fail(PC_EINVAL, "instance %d contract %d: beta_q16 must be in 0..2^50", i, c);
            d.rho[c] = s.contract[c].rho_q16;
            d.beta[c] = s.contract[c].beta_q16;
            if (c == 0 || d.rho[c] < rmin) rmin = d.rho[c];
        }
        // 1/w_c in Q16 (Eq. 5); Eq. 8's decrement 1/W_g must be positive, and
        // Q16 holds 1/w_c only down to 2^-16
        for (int c = 0; c < s.n_contracts; ++c) {
            d.invw[c] = (rmin << 16) / d.rho[c];
            if (d.invw[c] < 1)
                return fail(PC_EINVAL, "instance %d contract %d: refill rates of one instance may differ by at most "
                            "a factor 2^16", i, c);
        }
        int64_t scap = (int64_t)s.capacity * s.s3_small_permille / 1000;
        if (scap < 1) scap = 1;
        d.s_cap = (int32_t)scap;
        d.g_cap = (int32_t)(s.capacity - scap);
        d.move_thr = s.s3_move_threshold;
        int64_t maxn = std::min<int64_t>(t.max_req_blocks, s.capacity);
        // a candidate for the kernel's default-layout copy is laid out for
        // requests of kFixMaxn blocks (maxn only sizes buffers)
        if (s.capacity == pcr::kFixC && maxn <= pcr::kFixMaxn && d.s_cap == pcr::kFixScap &&
            d.move_thr == pcr::kFixMoveThr)
            maxn = pcr::kFixMaxn;
        d.maxn = (int32_t)maxn;
        d.log_log2 = ceil_log2(s.capacity + maxn + 128);
        const bool ghost = s.policy == PC_S3FIFO && d.g_cap > 0;
        if (ghost) {
            d.gnb_log2 = std::max(1, ceil_log2((int64_t)d.g_cap * 3 / 16 + 1));
            // ghost ring: 4 g_cap + 256 positions (at most 2^16), see the ghost
            // sweep: any ring of at least 2 g_cap + 256 gives the same ghost; a
            // longer one (HBM) lets each scan batch sweep fewer table entries
            d.gr_log2 = std::min(16, ceil_log2(4 * (int64_t)d.g_cap + 256));
        }
        d.n_prefix_words = (int32_t)((t.n_prefix + 31) / 32);
        // the state in each layout (table size, offsets, instances per CU)
        plan_lds[i] = pcr::plan_state(pcr::kLayLds, s.policy, s.capacity, maxn, d.log_log2, d.gnb_log2, ghost, lds_cu);
        plan_hyb[i] = pcr::plan_state(pcr::kLayHybrid, s.policy, s.capacity, maxn, d.log_log2, d.gnb_log2, ghost,
                                      lds_cu);
        plan_ws[i] = pcr::plan_state(pcr::kLayWs, s.policy, s.capacity, maxn, d.log_log2, d.gnb_log2, ghost, lds_cu);
        if (plan_ws[i].f.end > INT32_MAX) return fail(PC_EINVAL, "instance %d: state too large", i);
        // first the layout that lets the most instances share a CU
        // (all-LDS on a tie: its probes read no HBM)
        const int nl = plan_lds[i].per_cu, nh = plan_hyb[i].per_cu;
        d.layout = nl > 0 && nl >= nh ? pcr::kLayLds : nh > 0 ? pcr::kLayHybrid : pcr::kLayWs;
        per_cu[i] = d.layout == pcr::kLayLds ? nl : d.layout == pcr::kLayHybrid ? nh : pcr::kMaxWgPerCu;
        // replay time of the instance, in LRU probe units: cycles per request
        // measured with the phase-counter build relative to LRU's (S3-FIFO
        // 1.7-1.8x, PrefixShield 1.5x), plus a per-request share; the
        // costliest instances start first
        const double per_probe = s.policy == PC_S3FIFO ? 1.75 : s.policy == PC_PREFIXSHIELD ? 1.5 : 1.0;
        cost[i] = (double)t.n_keys * per_probe + (double)t.n_req * 16.0;
        d.per_req_off = per_req;
        per_req += 4 * t.n_req;
    }
    // When the whole batch fits the CUs at once, instances whose densest
    // layout is the hybrid one take the all-LDS layout instead (it reads no
    // HBM per probe), costliest first, as long as the batch still fits:
    // with free CUs a request's latency is what counts.
    {
        double demand = 0;
        for (int i = 0; i < n_inst; ++i) demand += 1.0 / per_cu[i];
        std::vector<int32_t> up;
        for (int i = 0; i < n_inst; ++i)
            if (P.di[i].layout != pcr::kLayLds && plan_lds[i].per_cu > 0) up.push_back(i);
        std::stable_sort(up.begin(), up.end(), [&](int32_t a, int32_t b) { return cost[a] > cost[b]; });
        for (int32_t i : up) {
            const double extra = 1.0 / plan_lds[i].per_cu - 1.0 / per_cu[i];
            if (demand + extra > (double)n_cu) break;
            demand += extra;
            P.di[i].layout = pcr::kLayLds;
            per_cu[i] = plan_lds[i].per_cu;
        }
    }
    // state offsets of the chosen layout; the kernel's compile-time copy
    for (int i = 0; i < n_inst; ++i) {
        const pc_instance_desc &s = inst[i];
        pcr::DevInst &d = P.di[i];
        const pcr::StatePlan &pl = d.layout == pcr::kLayLds ? plan_lds[i]
                                   : d.layout == pcr::kLayHybrid ? plan_hyb[i] : plan_ws[i];
        const pcr::StateOffsets &f = pl.f;
        d.nb = pl.nb;
        d.rs_log2 = pl.rs_log2;
        d.o_key = f.o_key; d.o_stamp = f.o_stamp; d.o_meta = f.o_meta; d.o_table = f.o_table; d.o_log = f.o_log;
        d.o_rkeys = f.o_rkeys; d.o_rset = f.o_rset; d.o_posslot = f.o_posslot; d.o_vlist = f.o_vlist;
        d.o_rcnt = f.o_rcnt; d.o_res = f.o_res; d.o_pfx = f.o_pfx; d.o_cnt = f.o_cnt; d.o_cur = f.o_cur;
        d.o_fstack = f.o_fstack; d.o_gtable = f.o_gtable;
        d.state_bytes = (int32_t)f.end;
        d.fixc = 0;
        if (d.layout != pcr::kLayWs) {
            const bool s3 = s.policy == PC_S3FIFO;
            const pcr::StatePlan x = pcr::fix_plan(d.layout, s.policy);
            const pcr::StateOffsets &g = x.f;
            const bool offs = f.o_key == g.o_key && f.o_stamp == g.o_stamp && f.o_meta == g.o_meta &&
                              f.o_table == g.o_table && f.o_log == g.o_log && f.o_rkeys == g.o_rkeys &&
                              f.o_rset == g.o_rset && f.o_posslot == g.o_posslot && f.o_vlist == g.o_vlist &&
                              f.o_rcnt == g.o_rcnt && f.o_res == g.o_res && f.o_pfx == g.o_pfx &&
                              f.o_cnt == g.o_cnt && f.o_cur == g.o_cur && f.o_fstack == g.o_fstack &&
                              f.o_gtable == g.o_gtable && f.end == g.end;
            const bool fix = offs && s.capacity == pcr::kFixC && d.maxn == pcr::kFixMaxn &&
                             d.s_cap == pcr::kFixScap && s.n_contracts == 1 && s.eps_q16 == 0 && s.flags == 0 &&
                             d.g_cap == pcr::kFixGcap && d.move_thr == pcr::kFixMoveThr && d.nb == x.nb &&
                             d.rs_log2 == x.rs_log2 && d.log_log2 == pcr::kFixLogLog2 &&
                             d.gnb_log2 == (s3 ? pcr::kFixGnbLog2S3 : 0) && d.gr_log2 == (s3 ? pcr::kFixGrLog2S3 : 0);
            d.fixc = fix ? pcr::kFixC : 0;
        }
    }
    // global regions per instance
    for (int i = 0; i < n_inst; ++i) {
        pcr::DevInst &d = P.di[i];
        if (d.layout == pcr::kLayWs) { d.ws_state = off; off = align_up(off + d.state_bytes, 256); }
        if (d.layout == pcr::kLayHybrid) {
            d.ws_key = off;
            if (d.policy == PC_PREFIXSHIELD) {   // key and prefix id in one 16-byte record per slot
                d.ws_pfx = off + 8;
                off = align_up(off + 16LL * d.capacity, 256);
            } else {
                off = align_up(off + 8LL * d.capacity, 256);
            }
            if (d.policy == PC_S3FIFO && d.g_cap > 0) {
                d.ws_gtable = off;
                off = align_up(off + (32LL << d.gnb_log2), 256);
            }
        }
        d.ws_bits = off;
        off = align_up(off + 8LL * d.n_prefix_words, 256);
        if (d.policy == PC_S3FIFO && d.g_cap > 0) {
            d.ws_gring = off;
            off = align_up(off + (8LL << d.gr_log2), 256);
        }
    }
    P.ws_bytes = std::max<int64_t>(off, 256);
    // launches: one per (layout, instances per CU), each sized to its
    // largest LDS state; instances inside a launch costliest first, the
    // longest launch first
    std::vector<int32_t> ids(n_inst);
    for (int i = 0; i < n_inst; ++i) ids[i] = i;
    auto key_of = [&](int32_t i) { return std::make_pair(P.di[i].layout, per_cu[i]); };
    std::sort(ids.begin(), ids.end(), [&](int32_t a, int32_t b) {
        if (key_of(a) != key_of(b)) return key_of(a) < key_of(b);
        return cost[a] > cost[b] || (cost[a] == cost[b] && a < b);
    });
    for (int32_t k = 0; k < n_inst;) {
        Launch L;
        L.layout = P.di[ids[k]].layout;
        L.per_cu = per_cu[ids[k]];
        L.first = k;
        L.cost = cost[ids[k]];
        double total = 0;
        while (k < n_inst && key_of(ids[k]) == key_of(ids[L.first])) {
            if (L.layout != pcr::kLayWs) L.lds_bytes = std::max(L.lds_bytes, P.di[ids[k]].state_bytes);
            total += cost[ids[k]];
            ++k;
        }
        L.count = k - L.first;
        // duration: its costliest instance, or its work spread over every
        // slot of the GPU, whichever is longer; state in HBM makes every
        // request several times slower
        L.est = std::max(L.cost, total / ((double)L.per_cu * (double)n_cu)) * (L.layout == pcr::kLayWs ? 3.0 : 1.0);
        P.lds_bytes = std::max(P.lds_bytes, L.lds_bytes);
        P.launches.push_back(L);
    }
    std::stable_sort(P.launches.begin(), P.launches.end(), [](const Launch &a, const Launch &b) {
        return a.est > b.est;
    });
    P.order.clear();
    for (Launch &L : P.launches) {
        const int32_t f = (int32_t)P.order.size();
        P.order.insert(P.order.end(), ids.begin() + L.first, ids.begin() + L.first + L.count);
        L.first = f;
    }
    return PC_OK;
}

// Pinned staging for descriptor uploads, reused once the previous copy is done.
struct Staging {
    std::mutex mu;
    void *buf = nullptr;
    size_t cap = 0;
    hipEvent_t done = nullptr;
    bool pending = false;
};
Staging g_stage;

}  // namespace

extern "C" {

const char *pc_last_error(void) { return g_err.c_str(); }

int32_t pc_block_offsets(const int32_t *d_req_len, int64_t n_req, int32_t block_size, int64_t *d_key_off,
                         void *stream) {
    if (block_size != PC_BLOCK_TOKENS) return fail(PC_EUNSUPPORTED, "block_size %d (only 16)", block_size);
    if (n_req < 0) return fail(PC_EINVAL, "n_req < 0");
    if (!d_key_off || (n_req > 0 && !d_req_len)) return fail(PC_EINVAL, "null pointer");
    hipError_t e = pcr::launch_block_offsets(d_req_len, n_req, d_key_off, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "block offsets launch");
    return ok();
}

int32_t pc_hash_blocks(const int32_t *d_tokens, int64_t n_tokens, const int64_t *d_req_tok_off,
                       const int32_t *d_req_len, const int32_t *d_req_ns, const int64_t *d_key_off, int64_t n_req,
                       int32_t block_size, uint64_t *d_keys, int64_t n_keys, int32_t *d_status, void *stream) {
    if (block_size != PC_BLOCK_TOKENS) return fail(PC_EUNSUPPORTED, "block_size %d (only 16)", block_size);
    if (n_req < 0 || n_tokens < 0 || n_keys < 0) return fail(PC_EINVAL, "negative size");
    if (!d_status) return fail(PC_EINVAL, "null status pointer");
    if (n_req > 0 && (!d_req_tok_off || !d_req_len || !d_req_ns || !d_key_off))
        return fail(PC_EINVAL, "null request array");
    if (n_tokens > 0 && !d_tokens) return fail(PC_EINVAL, "null tokens");
    if (n_keys > 0 && !d_keys) return fail(PC_EINVAL, "null keys");
    if (((uintptr_t)d_tokens & 3) != 0) return fail(PC_EINVAL, "d_tokens must be 4-byte aligned");
    hipError_t e = pcr::launch_hash(d_tokens, n_tokens, d_req_tok_off, d_req_len, d_req_ns, d_key_off, n_req, d_keys,
                                    n_keys, d_status, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "hash launch");
    return ok();
}

int64_t pc_replay_workspace_bytes(const pc_trace_desc *traces, int32_t n_traces, const pc_instance_desc *inst,
                                  int32_t n_inst) {
    Plan P;
    int32_t rc = validate_and_plan(traces, n_traces, inst, n_inst, lds_per_cu(), cu_count(), P);
    if (rc != PC_OK) return rc;
    ok();
    return P.ws_bytes;
}

int32_t pc_replay_state_bytes(const pc_trace_desc *traces, int32_t n_traces, const pc_instance_desc *inst,
                              int32_t n_inst, int64_t *bytes_out, int32_t *layout_out) {
    if (n_inst > 0 && (!bytes_out || !layout_out)) return fail(PC_EINVAL, "null output");
    Plan P;
    int32_t rc = validate_and_plan(traces, n_traces, inst, n_inst, lds_per_cu(), cu_count(), P);
    if (rc != PC_OK) return rc;
    for (int i = 0; i < n_inst; ++i) {
        bytes_out[i] = P.di[i].state_bytes;
        const pcr::DevInst &d = P.di[i];
        if (d.layout == pcr::kLayHybrid)   // keys, prefix ids, ghost table in the workspace
            bytes_out[i] += (d.policy == PC_PREFIXSHIELD ? 16LL : 8LL) * d.capacity +
                            (d.policy == PC_S3FIFO && d.g_cap > 0 ? (32LL << d.gnb_log2) : 0);
        layout_out[i] = d.layout;
    }
    return ok();
}

}  // extern "C"

namespace {

// Descriptor header of a planned batch (DevInst[], DevTrace[], order[]), as
// the kernels find it at the start of the workspace.
void fill_header(const Plan &P, int32_t n_traces, int32_t n_inst, uint8_t *h) {
    const size_t o_tr = align_up((int64_t)sizeof(pcr::DevInst) * n_inst, 256);
    const size_t o_ord = align_up((int64_t)o_tr + (int64_t)sizeof(pcr::DevTrace) * n_traces, 256);
    std::memset(h, 0, (size_t)P.hdr_bytes);
    std::memcpy(h, P.di.data(), sizeof(pcr::DevInst) * n_inst);
    if (n_traces) std::memcpy(h + o_tr, P.dt.data(), sizeof(pcr::DevTrace) * n_traces);
    std::memcpy(h + o_ord, P.order.data(), sizeof(int32_t) * n_inst);
}

// Library streams (default priority) that the launches of one batch fork
// onto, so that launches of different footprints run side by side; joined
// back into the caller's stream with events.  One set per device.
constexpr int kForkStreams = 4;
struct ForkStreams {
    std::mutex mu;
    bool ready[64] = {};
    hipStream_t s[64][kForkStreams] = {};
    hipEvent_t fork[64] = {}, join[64][kForkStreams] = {};
};
ForkStreams g_fork;

int32_t fork_streams(int dev) {
    if (g_fork.ready[dev]) return PC_OK;
    hipError_t e;
    for (int k = 0; k < kForkStreams; ++k) {
        e = hipStreamCreateWithFlags(&g_fork.s[dev][k], hipStreamNonBlocking);
        if (e != hipSuccess) return hip_fail(e, "library stream");
        e = hipEventCreateWithFlags(&g_fork.join[dev][k], hipEventDisableTiming);
        if (e != hipSuccess) return hip_fail(e, "library event");
    }
    e = hipEventCreateWithFlags(&g_fork.fork[dev], hipEventDisableTiming);
    if (e != hipSuccess) return hip_fail(e, "library event");
    g_fork.ready[dev] = true;
    return PC_OK;
}

// Launches of a planned batch whose header is already queued for upload to
// the start of `ws` on stream s.  With `fork`, launches go round-robin onto
// the library streams (after s reaches this point) and s waits for all of
// them; else they run one after another on s.
int32_t launch_planned(const Plan &P, int32_t n_traces, int32_t n_inst, uint8_t *ws, void *d_stats,
                       int32_t *d_per_request, hipStream_t s, bool fork) {
    const size_t o_tr = align_up((int64_t)sizeof(pcr::DevInst) * n_inst, 256);
    const size_t o_ord = align_up((int64_t)o_tr + (int64_t)sizeof(pcr::DevTrace) * n_traces, 256);
    const pcr::DevInst *d_inst = (const pcr::DevInst *)ws;
    const pcr::DevTrace *d_tr = (const pcr::DevTrace *)(ws + o_tr);
    const int32_t *d_ord = (const int32_t *)(ws + o_ord);
    hipError_t e;
    if (P.lds_bytes > 0) {
        e = pcr::replay_set_lds_limit(P.lds_bytes);
        if (e != hipSuccess) return hip_fail(e, "replay LDS limit");
    }
    const int nl = (int)P.launches.size();
    if (!fork || nl < 2) {
        for (const Launch &L : P.launches) {
            e = pcr::launch_replay(d_inst, d_tr, d_ord + L.first, L.count, L.lds_bytes, L.layout, L.per_cu, ws,
                                   (int64_t *)d_stats, d_per_request, s);
            if (e != hipSuccess) return hip_fail(e, "replay launch");
        }
        return ok();
    }
    int dev = 0;
    e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "current device");
    if (dev < 0 || dev >= 64) return fail(PC_EUNSUPPORTED, "device %d (at most 64 devices)", dev);
    std::lock_guard<std::mutex> lk(g_fork.mu);
    int32_t rc = fork_streams(dev);
    if (rc != PC_OK) return rc;
    e = hipEventRecord(g_fork.fork[dev], s);
    if (e != hipSuccess) return hip_fail(e, "fork event");
    const int used = std::min(nl, kForkStreams);
    for (int k = 0; k < used; ++k) {
        e = hipStreamWaitEvent(g_fork.s[dev][k], g_fork.fork[dev], 0);
        if (e != hipSuccess) return hip_fail(e, "fork wait");
    }
    // longest launch first, each onto the stream with the least estimated
    // work queued so far
    double load[kForkStreams] = {};
    for (int l = 0; l < nl; ++l) {
        const Launch &L = P.launches[l];
        int k = 0;
        for (int j = 1; j < used; ++j)
            if (load[j] < load[k]) k = j;
        load[k] += L.est;
        e = pcr::launch_replay(d_inst, d_tr, d_ord + L.first, L.count, L.lds_bytes, L.layout, L.per_cu, ws,
                               (int64_t *)d_stats, d_per_request, g_fork.s[dev][k]);
        if (e != hipSuccess) return hip_fail(e, "replay launch");
    }
    for (int k = 0; k < used; ++k) {
        e = hipEventRecord(g_fork.join[dev][k], g_fork.s[dev][k]);
        if (e != hipSuccess) return hip_fail(e, "join event");
        e = hipStreamWaitEvent(s, g_fork.join[dev][k], 0);
        if (e != hipSuccess) return hip_fail(e, "join wait");
    }
    return ok();
}

struct StaticScratch {
    std::mutex mu;
    void *ptr[64] = {};
    // descriptor header staging (pageable host memory: the copy from it has
    // completed when hipMemcpyAsync returns)
    std::vector<uint8_t> host;
};
StaticScratch g_static;

}  // namespace

// ---- the entry point that allocates nothing takes its workspace from this
// array.  Each GPU the library runs on holds its own copy until the process
// ends.  Host code never uses the array's name as an address (on the host it
// only names the symbol): the device address comes from hipGetSymbolAddress,
// once per device with that device current, and is kept in g_static.ptr.
static __device__ __align__(256) uint8_t scratch[PC_STATIC_WORKSPACE_BYTES];

extern "C" {

int32_t pc_replay_batch(const pc_trace_desc *traces, int32_t n_traces, const pc_instance_desc *inst, int32_t n_inst,
                        void *d_workspace, int64_t workspace_bytes, void *d_stats, int32_t *d_per_request,
                        void *stream) {
    Plan P;
    int32_t rc = validate_and_plan(traces, n_traces, inst, n_inst, lds_per_cu(), cu_count(), P);
    if (rc != PC_OK) return rc;
    if (n_inst == 0) return ok();
    if (!d_workspace || !d_stats) return fail(PC_EINVAL, "null workspace or stats");
    if (((uintptr_t)d_workspace & 255) != 0) return fail(PC_EINVAL, "workspace must be 256-byte aligned");
    if (workspace_bytes < P.ws_bytes)
        return fail(PC_ENOMEM, "workspace %lld bytes < required %lld", (long long)workspace_bytes, (long long)P.ws_bytes);
    hipStream_t s = (hipStream_t)stream;
    uint8_t *ws = (uint8_t *)d_workspace;
    const size_t nbytes = (size_t)P.hdr_bytes;
    {
        std::lock_guard<std::mutex> lk(g_stage.mu);
        hipError_t e;
        if (g_stage.pending) {
            e = hipEventSynchronize(g_stage.done);
            if (e != hipSuccess) return hip_fail(e, "staging wait");
            g_stage.pending = false;
        }
        if (g_stage.cap < nbytes) {
            if (g_stage.buf) (void)hipHostFree(g_stage.buf);
            g_stage.buf = nullptr;
            g_stage.cap = 0;
            e = hipHostMalloc(&g_stage.buf, nbytes, hipHostMallocDefault);
            if (e != hipSuccess) return hip_fail(e, "pinned staging allocation");
            g_stage.cap = nbytes;
        }
        if (!g_stage.done) {
            e = hipEventCreateWithFlags(&g_stage.done, hipEventDisableTiming);
            if (e != hipSuccess) return hip_fail(e, "event create");
        }
        fill_header(P, n_traces, n_inst, (uint8_t *)g_stage.buf);
        e = hipMemcpyAsync(ws, g_stage.buf, nbytes, hipMemcpyHostToDevice, s);
        if (e != hipSuccess) return hip_fail(e, "descriptor upload");
        e = hipEventRecord(g_stage.done, s);
        if (e != hipSuccess) return hip_fail(e, "event record");
        g_stage.pending = true;
    }
    return launch_planned(P, n_traces, n_inst, ws, d_stats, d_per_request, s, true);
}

int32_t pc_replay_batch_static(const pc_trace_desc *traces, int32_t n_traces, const pc_instance_desc *inst,
                               int32_t n_inst, void *d_stats, int32_t *d_per_request, void *stream) {
    Plan P;
    int32_t rc = validate_and_plan(traces, n_traces, inst, n_inst, lds_per_cu(), cu_count(), P);
    if (rc != PC_OK) return rc;
    if (n_inst == 0) return ok();
    if (!d_stats) return fail(PC_EINVAL, "null stats");
    if (P.ws_bytes > (int64_t)PC_STATIC_WORKSPACE_BYTES)
        return fail(PC_ENOMEM, "batch needs %lld workspace bytes, more than the %lld of the static workspace",
                    (long long)P.ws_bytes, (long long)PC_STATIC_WORKSPACE_BYTES);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "current device");
    if (dev < 0 || dev >= 64) return fail(PC_EUNSUPPORTED, "device %d (at most 64 devices)", dev);
    hipStream_t s = (hipStream_t)stream;
    std::lock_guard<std::mutex> lk(g_static.mu);
    if (!g_static.ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "static workspace address");
        if (!p || ((uintptr_t)p & 255) != 0) return fail(PC_EDEVICE, "static workspace is not 256-byte aligned");
        g_static.ptr[dev] = p;
    }
    uint8_t *ws = (uint8_t *)g_static.ptr[dev];
    const size_t nbytes = (size_t)P.hdr_bytes;
    if (g_static.host.size() < nbytes) g_static.host.resize(nbytes);
    fill_header(P, n_traces, n_inst, g_static.host.data());
    e = hipMemcpyAsync(ws, g_static.host.data(), nbytes, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return hip_fail(e, "descriptor upload");
    return launch_planned(P, n_traces, n_inst, ws, d_stats, d_per_request, s, false);
}

int32_t pc_get_stats(const void *d_stats, int32_t n_inst, int32_t instance, pc_group_stats *groups_out,
                     int32_t max_groups, pc_instance_stats *inst_out, void *stream) {
    if (!d_stats || n_inst < 0) return fail(PC_EINVAL, "null stats or negative n_inst");
    if (instance < -1 || instance >= n_inst) return fail(PC_EINVAL, "instance %d out of range", instance);
    if (max_groups < 0 || max_groups > PC_MAX_GROUPS) return fail(PC_EINVAL, "max_groups outside 0..64");
    if ((max_groups > 0 && !groups_out) || !inst_out) return fail(PC_EINVAL, "null output");
    const int32_t first = instance < 0 ? 0 : instance;
    const int32_t count = instance < 0 ? n_inst : 1;
    std::vector<int64_t> buf((size_t)count * pcr::kRecordWords);
    hipStream_t s = (hipStream_t)stream;
    hipError_t e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "stream synchronize");
    if (count > 0) {
        e = hipMemcpy(buf.data(), (const int64_t *)d_stats + (size_t)first * pcr::kRecordWords,
                      buf.size() * sizeof(int64_t), hipMemcpyDeviceToHost);
        if (e != hipSuccess) return hip_fail(e, "stats copy");
    }
    for (int32_t i = 0; i < count; ++i) {
        const int64_t *rec = buf.data() + (size_t)i * pcr::kRecordWords;
        for (int32_t gidx = 0; gidx < max_groups; ++gidx) {
            const int64_t *g = rec + gidx * pcr::kGroupFields;
            pc_group_stats &o = groups_out[(size_t)i * max_groups + gidx];
            o.requests = (uint64_t)g[0]; o.probes = (uint64_t)g[1]; o.hits = (uint64_t)g[2]; o.misses = (uint64_t)g[3];
            o.charged = (uint64_t)g[4]; o.evicted_owned = (uint64_t)g[5]; o.evictions_caused = (uint64_t)g[6];
            o.promotions = (uint64_t)g[7]; o.gated = (uint64_t)g[8]; o.orphans = (uint64_t)g[9];
            o.dups = (uint64_t)g[10]; o.truncated = (uint64_t)g[11];
            o.debt_end_q16 = g[12]; o.debt_max_q16 = g[13]; o.debt_sum_q16 = g[14];
            o.resident_end = g[15]; o.resident_max = g[16];
        }
        const int64_t *q = rec + pcr::kInstOffset;
        pc_instance_stats &o = inst_out[i];
        o.evictions = (uint64_t)q[0]; o.s3_moves = (uint64_t)q[1]; o.s3_reinserts = (uint64_t)q[2];
        o.s3_ghost_hits = (uint64_t)q[3]; o.s3_ghost_inserts = (uint64_t)q[4];
        o.resident_end = q[5]; o.resident_max = q[6];
        o.status = (int32_t)(uint32_t)q[7];
        o.reserved = 0;
    }
    return ok();
}

}  // extern "C"

static_assert(sizeof(pc_group_stats) == 136, "pc_group_stats layout");
static_assert(sizeof(pc_instance_stats) == 64, "pc_instance_stats layout");
static_assert(PC_STATS_RECORD_BYTES == pcr::kRecordWords * 8, "stats record size");
