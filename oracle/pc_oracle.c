/*
 * pc_oracle.c -- reference oracle for the PrefixShield replay hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this file.  Only the test-suite, the smoke check and the benchmark's
 * CPU-baseline leg use it.  It shares no code, header, table or constant
 * generator with the GPU library; both are written separately from the
 * paper (arXiv 2608.01657, "Preserving Admission Responsibility in
 * Multi-Tenant LLM Prefix Caches").
 *
 * It is deliberately plain: one request at a time, one victim at a time,
 * textbook linked lists and an open-addressed map, integers only.
 *
 * What it computes
 * ----------------
 * 1. Block keys (the paper leaves the content hash to the serving engine,
 *    Sec. III-A / Sec. IV).  This build's chained key, PCH64:
 *      t_i   token id reinterpreted as uint32
 *      d_k   = sum_{i<8} ((t_{16k+2i} + K_{2i}) mod 2^32) * ((t_{16k+2i+1} + K_{2i+1}) mod 2^32)
 *              mod 2^64                       (NH-style block digest)
 *      H_-1  = fmix64(ns + 1)                 (namespace = accounting group)
 *      H_k   = A * H_{k-1} + fmix64(d_k)      mod 2^64
 *      key_k = fmix64(H_k)
 *    fmix64 is the public MurmurHash3 64-bit finalizer, A = 0x9E3779B97F4A7C15,
 *    K_i = floor(frac(sqrt(p_i)) * 2^31) + 1 for the first 16 primes p_i.
 *    Only full 16-token blocks get keys (Sec. III-B, "full KV blocks").
 *
 * 2. Replay of a request trace against one cache instance, following the
 *    request hooks of Algorithm 1 and the batch reclamation of Algorithm 2,
 *    with Eqs. 1-9 in Q16 fixed point (2^16 = one block).  Policies: LRU
 *    (vLLM's free-queue order, Sec. V-A), S3-FIFO (Sec. V-A baseline),
 *    PrefixShield, and StaticQuota (Sec. V-A baseline: equal fixed
 *    partitions of floor(C/G) blocks, LRU inside each, no borrowing).  The per-request step order, and every point where the
 *    paper is silent, is listed in the repository's design notes; the
 *    comments below name the paper passage each step follows.
 *
 * Parity status: the hash is this build's own definition (no value in the
 * paper to pin against); its tests pin structure and closed forms.  The
 * S3-FIFO internals follow this build's reading of the paper's one-line
 * description and are pinned only by invariants and a brute force.
 */
#define _POSIX_C_SOURCE 199309L   /* clock_gettime (reclamation timing only) */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <time.h>

/* ------------------------------------------------------------------------ */
/* PCH64 block keys                                                          */
/* ------------------------------------------------------------------------ */

static const uint32_t ORC_NH_KEY[16] = {
    0x3504f334u, 0x5db3d743u, 0x1e3779bau, 0x52a7fa9eu,
    0x28872940u, 0x4d82b447u, 0x0fc1ecd6u, 0x2df0668du,
    0x65ddceafu, 0x314d1496u, 0x48ac80aeu, 0x0a97f66du,
    0x33999334u, 0x475a2544u, 0x6d861707u, 0x23daa40fu};
#define ORC_CHAIN_A 0x9E3779B97F4A7C15ULL

uint64_t orc_fmix64(uint64_t z) {
    z ^= z >> 33;
    z *= 0xff51afd7ed558ccdULL;
    z ^= z >> 33;
    z *= 0xc4ceb9fe1a85ec53ULL;
    z ^= z >> 33;
    return z;
}

/* Block digest of 16 tokens. */
uint64_t orc_block_digest(const int32_t *tok) {
    uint64_t d = 0;
    for (int i = 0; i < 8; i++) {
        uint32_t a = (uint32_t)tok[2 * i] + ORC_NH_KEY[2 * i];
        uint32_t b = (uint32_t)tok[2 * i + 1] + ORC_NH_KEY[2 * i + 1];
        d += (uint64_t)a * (uint64_t)b;
    }
    return d;
}

/* Keys of every full block of one request; returns the number written. */
int64_t orc_hash_request(const int32_t *tok, int64_t len, uint32_t ns, uint64_t *out) {
    int64_t nb = len / 16;
    uint64_t H = orc_fmix64((uint64_t)ns + 1u);
    for (int64_t k = 0; k < nb; k++) {
        H = H * ORC_CHAIN_A + orc_fmix64(orc_block_digest(tok + 16 * k));
        out[k] = orc_fmix64(H);
    }
    return nb;
}

/* Hash a whole trace; key_off_out gets n_req+1 CSR offsets. */
int orc_hash_trace(const int32_t *tokens, const int64_t *tok_off, const int32_t *len,
                   const uint8_t *ns, int64_t n_req, uint64_t *keys_out, int64_t *key_off_out) {
    int64_t pos = 0;
    for (int64_t r = 0; r < n_req; r++) {
        if (len[r] < 0) return -1;
        key_off_out[r] = pos;
        pos += orc_hash_request(tokens + tok_off[r], len[r], ns[r], keys_out + pos);
    }
    key_off_out[n_req] = pos;
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Small open-addressed map uint64 -> int64 (linear probing, backward-shift  */
/* deletion).  Textbook; used for key->block, the ghost, and per-request     */
/* duplicate detection.                                                      */
/* ------------------------------------------------------------------------ */

typedef struct {
    uint64_t *k;
    int64_t *v;
    uint32_t *gen;   /* slot occupied iff gen[i] == cur */
    uint32_t cur;
    uint64_t mask;
    int bits;
    int64_t size;
} Map;

static int map_init(Map *m, int64_t min_cap) {
    int bits = 4;
    while (((int64_t)1 << bits) < 2 * min_cap + 2) bits++;
    uint64_t n = (uint64_t)1 << bits;
    m->k = (uint64_t *)calloc(n, sizeof(uint64_t));
    m->v = (int64_t *)calloc(n, sizeof(int64_t));
    m->gen = (uint32_t *)calloc(n, sizeof(uint32_t));
    m->cur = 1;
    m->mask = n - 1;
    m->bits = bits;
    m->size = 0;
    return (m->k && m->v && m->gen) ? 0 : -1;
}
static void map_free(Map *m) { free(m->k); free(m->v); free(m->gen); }
static uint64_t map_home(const Map *m, uint64_t key) {
    return (key * 0x9E3779B97F4A7C15ULL) >> (64 - m->bits);
}
static int map_get(const Map *m, uint64_t key, int64_t *val) {
    for (uint64_t i = map_home(m, key);; i = (i + 1) & m->mask) {
        if (m->gen[i] != m->cur) return 0;
        if (m->k[i] == key) { if (val) *val = m->v[i]; return 1; }
    }
}
static void map_put(Map *m, uint64_t key, int64_t val) {
    for (uint64_t i = map_home(m, key);; i = (i + 1) & m->mask) {
        if (m->gen[i] != m->cur) { m->gen[i] = m->cur; m->k[i] = key; m->v[i] = val; m->size++; return; }
        if (m->k[i] == key) { m->v[i] = val; return; }
    }
}
static void map_del(Map *m, uint64_t key) {
    uint64_t i = map_home(m, key);
    for (;; i = (i + 1) & m->mask) {
        if (m->gen[i] != m->cur) return;
        if (m->k[i] == key) break;
    }
    m->size--;
    uint64_t j = i;
    for (;;) {
        j = (j + 1) & m->mask;
        if (m->gen[j] != m->cur) break;
        uint64_t h = map_home(m, m->k[j]);
        /* move j back into hole i unless its home lies cyclically in (i, j] */
        int stay = (i <= j) ? (i < h && h <= j) : (i < h || h <= j);
        if (!stay) { m->k[i] = m->k[j]; m->v[i] = m->v[j]; i = j; }
    }
    m->gen[i] = 0;
}
static void map_clear(Map *m) { m->cur++; m->size = 0; if (m->cur == 0) { memset(m->gen, 0, (m->mask + 1) * sizeof(uint32_t)); m->cur = 1; } }

/* ------------------------------------------------------------------------ */
/* Replay                                                                    */
/* ------------------------------------------------------------------------ */

enum { ORC_LRU = 0, ORC_S3FIFO = 1, ORC_PS = 2, ORC_SQ = 3 };
enum { ORC_NO_SEGMENTATION = 1, ORC_NO_DEBT_GATE = 2 };
enum { PROB = 0, NORMAL = 1, REUSE = 2 };      /* Sec. III-A retention classes */
#define SCALE 65536LL

/* output field order (per group) */
enum {
    G_REQUESTS, G_PROBES, G_HITS, G_MISSES, G_CHARGED, G_EVICTED_OWNED,
    G_EVICTIONS_CAUSED, G_PROMOTIONS, G_GATED, G_ORPHANS, G_DUPS, G_TRUNCATED,
    G_DEBT_END, G_DEBT_MAX, G_DEBT_SUM, G_RESIDENT_END, G_RESIDENT_MAX, G_NFIELDS
};
/* output field order (per instance) */
enum {
    I_EVICTIONS, I_S3_MOVES, I_S3_REINSERTS, I_S3_GHOST_HITS, I_S3_GHOST_INSERTS,
    I_RESIDENT_END, I_RESIDENT_MAX, I_NFIELDS
};

typedef struct {
    uint64_t key;
    int32_t owner, contract;
    uint32_t prefix;
    int32_t cls, freq;
    int32_t pinned;
    uint64_t stamp;
    int32_t list, prev, next;
} Block;

typedef struct { int32_t head, tail; int64_t count; } List;

typedef struct {
    int policy, flags, G, K;
    int64_t C;
    int64_t rho[4], beta[4], invw[4], eps;
    int64_t s_cap, g_cap, move_thr;

    Block *blk;
    int32_t *free_ids;
    int64_t n_free;
    Map map;          /* key -> block id of resident blocks */
    List *lists;      /* LRU: 1; PS: G*3; S3: 2 (S, M); SQ: G (one per partition) */
    int64_t quota;    /* SQ: blocks per group partition */
    int n_lists;

    int64_t bal[64][4], last[64][4];
    int64_t resident[64];
    int64_t resident_total;

    uint8_t *referenced, *admitted;   /* per logical prefix id */
    uint64_t stampctr;

    /* S3-FIFO */
    int64_t s_size, s_unpinned, m_unpinned;
    Map ghost;            /* key -> ghost insertion sequence */
    uint64_t *ghost_ring; /* key of each of the last g_cap insertions */
    int64_t gseq;

    int64_t *gs;          /* [G][G_NFIELDS] */
    int64_t *is;          /* [I_NFIELDS] */
} Inst;

/* ---- linked lists (free-queue order: head = oldest) ---- */
static void list_append(Inst *s, int32_t L, int32_t b) {
    List *l = &s->lists[L];
    Block *x = &s->blk[b];
    x->list = L; x->prev = l->tail; x->next = -1;
    if (l->tail >= 0) s->blk[l->tail].next = b; else l->head = b;
    l->tail = b; l->count++;
}
static void list_unlink(Inst *s, int32_t b) {
    Block *x = &s->blk[b];
    if (x->list < 0) return;
    List *l = &s->lists[x->list];
    if (x->prev >= 0) s->blk[x->prev].next = x->next; else l->head = x->next;
    if (x->next >= 0) s->blk[x->next].prev = x->prev; else l->tail = x->prev;
    l->count--; x->list = -1; x->prev = x->next = -1;
}
static int32_t ps_list(const Inst *s, int32_t owner, int32_t cls) {
    int seg = (s->flags & ORC_NO_SEGMENTATION) ? 0 : cls;
    return owner * 3 + seg;
}

/* ---- Eq. 1: lazily refilled balance, exact in unbounded integers ---- */
static int64_t eff_balance(const Inst *s, int g, int c, int64_t t) {
    int64_t dt = t - s->last[g][c];
    int64_t gap = s->beta[c] - s->bal[g][c];          /* >= 0 */
    __int128 add = (__int128)s->rho[c] * (__int128)dt;
    if (add >= (__int128)gap) return s->beta[c];
    return s->bal[g][c] + (int64_t)add;
}
/* Eq. 3: raw debt, summed over the group's contracts */
static int64_t raw_debt(const Inst *s, int g, int64_t t) {
    int64_t d = 0;
    for (int c = 0; c < s->K; c++) { int64_t b = eff_balance(s, g, c, t); if (b < 0) d += -b; }
    return d;
}
/* Eq. 5: normalized debt, each term debt_c * (1/w_c) with 1/w_c in Q16 */
static int64_t norm_debt(const Inst *s, int g, int64_t t) {
    int64_t d = 0;
    for (int c = 0; c < s->K; c++) {
        int64_t b = eff_balance(s, g, c, t);
        if (b < 0) d += (int64_t)(((__int128)(-b) * (__int128)s->invw[c]) >> 16);
    }
    return d;
}
/* Eq. 8: 1/W_g, the smallest one-block decrement among indebted contracts
   (0 when no contract of the group is indebted; every invw_c is >= 1, so an
   indebted group always has a positive decrement) */
static int64_t debt_decrement(const Inst *s, int g, int64_t t) {
    int64_t m = -1;
    for (int c = 0; c < s->K; c++)
        if (eff_balance(s, g, c, t) < 0 && (m < 0 || s->invw[c] < m)) m = s->invw[c];
    return m < 0 ? 0 : m;
}

static int32_t alloc_block(Inst *s) {
    if (s->n_free <= 0) return -1;
    return s->free_ids[--s->n_free];
}
/* remove a resident, unpinned block from the cache (eviction or orphan drop) */
static void drop_block(Inst *s, int32_t b) {
    Block *x = &s->blk[b];
    list_unlink(s, b);
    map_del(&s->map, x->key);
    s->resident[x->owner]--;
    s->resident_total--;
    s->free_ids[s->n_free++] = b;
}

static void s3_ghost_insert(Inst *s, uint64_t key) {
    /* the ghost keeps the last g_cap insertions; the one falling out of the
       window is forgotten (unless the same key was re-inserted since) */
    s->is[I_S3_GHOST_INSERTS]++;
    if (s->g_cap > 0) {
        int64_t slot = s->gseq % s->g_cap;
        if (s->gseq >= s->g_cap) {
            uint64_t old = s->ghost_ring[slot];
            int64_t oseq;
            if (map_get(&s->ghost, old, &oseq) && oseq == s->gseq - s->g_cap) map_del(&s->ghost, old);
        }
        s->ghost_ring[slot] = key;
        map_put(&s->ghost, key, s->gseq);
    }
    s->gseq++;
}
static int s3_ghost_take(Inst *s, uint64_t key) {
    int64_t seq;
    if (!map_get(&s->ghost, key, &seq)) return 0;
    if (seq < s->gseq - s->g_cap) return 0;
    map_del(&s->ghost, key);
    return 1;
}

/* S3-FIFO: evict exactly one unpinned block (small FIFO / main FIFO / ghost) */
static int32_t s3_evict_one(Inst *s) {
    List *S = &s->lists[0], *M = &s->lists[1];
    for (;;) {
        int useS = (s->s_size >= s->s_cap && s->s_unpinned > 0) || (s->m_unpinned == 0);
        if (useS) {
            int32_t b = S->head;
            while (b >= 0 && s->blk[b].pinned) b = s->blk[b].next;
            if (b < 0) return -1;
            Block *x = &s->blk[b];
            if (x->freq >= s->move_thr) {
                list_unlink(s, b); s->s_size--; s->s_unpinned--;
                x->freq = 0; list_append(s, 1, b); s->m_unpinned++;
                s->is[I_S3_MOVES]++;
                continue;
            }
            s->s_size--; s->s_unpinned--;
            s3_ghost_insert(s, x->key);
            return b;
        } else {
            int32_t b = M->head;
            while (b >= 0 && s->blk[b].pinned) b = s->blk[b].next;
            if (b < 0) return -1;
            Block *x = &s->blk[b];
            if (x->freq > 0) {
                list_unlink(s, b); x->freq--; list_append(s, 1, b);
                s->is[I_S3_REINSERTS]++;
                continue;
            }
            s->m_unpinned--;
            return b;
        }
    }
}

/* PrefixShield: pick one victim (one iteration of Algorithm 2's loop). */
static int32_t ps_pick(Inst *s, int64_t *P, const int64_t *D) {
    int nseg = (s->flags & ORC_NO_SEGMENTATION) ? 1 : 3;
    int best = -1, best_seg = 0;
    uint64_t best_hs = 0;
    for (int x = 0; x < s->G; x++) {
        if (P[x] <= s->eps) continue;              /* Eq. 6: indebted */
        int seg = -1;
        for (int q = 0; q < nseg; q++) if (s->lists[x * 3 + q].count > 0) { seg = q; break; }
        if (seg < 0) continue;                     /* owns no candidate */
        uint64_t hs = s->blk[s->lists[x * 3 + seg].head].stamp;
        /* Eq. 7 argmax; ties by retention segment, then native queue order */
        if (best < 0 || P[x] > P[best] ||
            (P[x] == P[best] && (seg < best_seg || (seg == best_seg && hs < best_hs)))) {
            best = x; best_seg = seg; best_hs = hs;
        }
    }
    if (best >= 0) {
        int32_t v = s->lists[best * 3 + best_seg].head;
        P[best] -= D[best];                        /* Eq. 8 */
        if (P[best] < 0) P[best] = 0;
        return v;
    }
    /* no indebted candidate owner: global segment order (Eq. 9 fallback) */
    for (int q = 0; q < nseg; q++) {
        int32_t v = -1;
        for (int x = 0; x < s->G; x++) {
            int32_t h = s->lists[x * 3 + q].head;
            if (h >= 0 && (v < 0 || s->blk[h].stamp < s->blk[v].stamp)) v = h;
        }
        if (v >= 0) return v;
    }
    return -1;
}

static void account_all(Inst *s, int64_t t) {
    for (int x = 0; x < s->G; x++) {
        int64_t *o = s->gs + (int64_t)x * G_NFIELDS;
        int64_t d = raw_debt(s, x, t);
        o[G_DEBT_SUM] = (int64_t)((uint64_t)o[G_DEBT_SUM] + (uint64_t)d);
        if (d > o[G_DEBT_MAX]) o[G_DEBT_MAX] = d;
        if (s->resident[x] > o[G_RESIDENT_MAX]) o[G_RESIDENT_MAX] = s->resident[x];
    }
    if (s->resident_total > s->is[I_RESIDENT_MAX]) s->is[I_RESIDENT_MAX] = s->resident_total;
}

/*
 * Replay one instance.
 *   keys/key_off : full-block keys, CSR offsets [n_req+1]
 *   group, contract, prefix, tick (tick may be NULL: tick = request index)
 *   policy 0 LRU, 1 S3-FIFO, 2 PrefixShield, 3 StaticQuota; flags 1 no
 *   segmentation, 2 no debt gate
 *   rho_q16/beta_q16 [n_contracts]
 *   group_stats_out [n_groups][17], inst_stats_out [7]
 *   per_req_out (optional) [n_req][4]: hits, new blocks, evictions, orphans
 *   reclaim_ns_out (optional) [n_req]: wall-clock nanoseconds of the
 *     request's reclamation (Alg. 2's victim selection and removal), 0 when
 *     it evicted nothing -- a measurement of the plain selector, nothing
 *     else changes
 * Returns 0, or a negative value for invalid input.
 */
static int replay_impl(const uint64_t *keys, const int64_t *key_off, const uint8_t *group,
                       const uint8_t *contract, const uint32_t *prefix, const int64_t *tick,
                       int64_t n_req, int32_t n_groups, int64_t n_prefix,
                       int32_t policy, int64_t capacity, int32_t flags, int32_t n_contracts,
                       const int64_t *rho_q16, const int64_t *beta_q16, int64_t eps_q16,
                       int32_t s3_small_permille, int32_t s3_move_threshold,
                       int64_t *group_stats_out, int64_t *inst_stats_out, int32_t *per_req_out,
                       int64_t *reclaim_ns_out) {
    if (policy < 0 || policy > 3 || capacity < 1 || n_groups < 1 || n_groups > 64 ||
        n_contracts < 1 || n_contracts > 4 || eps_q16 < 0 || n_req < 0 || n_prefix < 0)
        return -1;
    if (s3_small_permille < 0 || s3_small_permille > 1000 || s3_move_threshold < 0) return -1;
    Inst S;
    memset(&S, 0, sizeof(S));
    Inst *s = &S;
    s->policy = policy; s->flags = flags; s->G = n_groups; s->K = n_contracts;
    s->C = capacity; s->eps = eps_q16;
    s->quota = capacity / n_groups;   /* SQ partitions; C mod G blocks stay unused */
    int64_t rho_min = 0;
    for (int c = 0; c < n_contracts; c++) {
        if (rho_q16[c] <= 0 || beta_q16[c] < 0) return -1;
        s->rho[c] = rho_q16[c]; s->beta[c] = beta_q16[c];
        if (c == 0 || rho_q16[c] < rho_min) rho_min = rho_q16[c];
    }
    /* 1/w_c = rho_min/rho_c, Q16, rounded down.  Eq. 8 needs a positive
       decrement 1/W_g, and Q16 represents 1/w_c only down to 2^-16: rates
       that differ by more than a factor 2^16 are rejected. */
    for (int c = 0; c < n_contracts; c++) {
        s->invw[c] = (int64_t)(((__int128)rho_min << 16) / s->rho[c]);
        if (s->invw[c] < 1) return -1;
    }
    for (int64_t r = 0; r < n_req; r++) {
        if (group[r] >= n_groups || contract[r] >= n_contracts || prefix[r] >= n_prefix) return -1;
        if (key_off[r + 1] < key_off[r]) return -1;
        if (tick && (tick[r] < 0 || (r > 0 && tick[r] < tick[r - 1]))) return -1;
    }
    int64_t max_n = 0;
    for (int64_t r = 0; r < n_req; r++) {
        int64_t n = key_off[r + 1] - key_off[r];
        if (n > capacity) n = capacity;
        if (n > max_n) max_n = n;
    }
    s->s_cap = capacity * s3_small_permille / 1000;
    if (s->s_cap < 1) s->s_cap = 1;
    s->g_cap = capacity - s->s_cap;
    s->move_thr = s3_move_threshold;

    int rc = -2;
    s->blk = (Block *)calloc((size_t)capacity + 1, sizeof(Block));
    s->free_ids = (int32_t *)malloc(((size_t)capacity + 1) * sizeof(int32_t));
    s->n_lists = (policy == ORC_PS) ? 3 * n_groups : (policy == ORC_S3FIFO ? 2 : (policy == ORC_SQ ? n_groups : 1));
    s->lists = (List *)malloc((size_t)s->n_lists * sizeof(List));
    s->referenced = (uint8_t *)calloc((size_t)n_prefix + 1, 1);
    s->admitted = (uint8_t *)calloc((size_t)n_prefix + 1, 1);
    s->ghost_ring = (uint64_t *)calloc((size_t)(s->g_cap > 0 ? s->g_cap : 1), sizeof(uint64_t));
    int32_t *pos_blk = (int32_t *)malloc(((size_t)max_n + 1) * sizeof(int32_t));
    int32_t *hit_pos = (int32_t *)malloc(((size_t)max_n + 1) * sizeof(int32_t));
    int32_t *new_pos = (int32_t *)malloc(((size_t)max_n + 1) * sizeof(int32_t));
    uint8_t *is_dup = (uint8_t *)malloc((size_t)max_n + 1);
    Map seen;
    memset(&seen, 0, sizeof(seen));
    if (!s->blk || !s->free_ids || !s->lists || !s->referenced || !s->admitted || !s->ghost_ring ||
        !pos_blk || !hit_pos || !new_pos || !is_dup)
        goto out;
    if (map_init(&s->map, capacity) || map_init(&s->ghost, s->g_cap + 1) || map_init(&seen, max_n + 1))
        goto out;
    for (int i = 0; i < s->n_lists; i++) { s->lists[i].head = s->lists[i].tail = -1; s->lists[i].count = 0; }
    for (int64_t i = 0; i < capacity; i++) s->free_ids[i] = (int32_t)(capacity - 1 - i);
    s->n_free = capacity;
    for (int g = 0; g < n_groups; g++)
        for (int c = 0; c < n_contracts; c++) { s->bal[g][c] = s->beta[c]; s->last[g][c] = 0; }
    s->gs = group_stats_out;
    s->is = inst_stats_out;
    memset(s->gs, 0, sizeof(int64_t) * (size_t)n_groups * G_NFIELDS);
    memset(s->is, 0, sizeof(int64_t) * I_NFIELDS);

    int64_t t = 0;
    for (int64_t r = 0; r < n_req; r++) {
        const int g = group[r], c = contract[r];
        const uint32_t p = prefix[r];
        t = tick ? tick[r] : r;
        const uint64_t *k = keys + key_off[r];
        int64_t *o = s->gs + (int64_t)g * G_NFIELDS;

        /* Alg. 1 OnRequest: prior reference count of (g,p), then record it */
        const int q_ge1 = s->referenced[p];
        s->referenced[p] = 1;
        o[G_REQUESTS]++;
        int64_t n_full = key_off[r + 1] - key_off[r];
        /* a request can hold at most the space it may fill: the cache, or
           under StaticQuota its group's partition */
        const int64_t room = policy == ORC_SQ ? s->quota : s->C;
        int64_t n = n_full < room ? n_full : room;
        o[G_TRUNCATED] += n_full - n;
        o[G_PROBES] += n;

        /* Native lookup: the hit is the longest leading run of resident
           blocks (Sec. III-B, n_cached).  A repeated key within the request
           is a duplicate: a miss that plays no further part. */
        map_clear(&seen);
        int64_t h = 0, n_hit = 0, n_new = 0, n_dup = 0, n_orph = 0;
        int in_run = 1;
        for (int64_t j = 0; j < n; j++) {
            is_dup[j] = 0; pos_blk[j] = -1;
            if (map_get(&seen, k[j], NULL)) { is_dup[j] = 1; n_dup++; continue; }
            map_put(&seen, k[j], j);
            int64_t b;
            int resident = map_get(&s->map, k[j], &b);
            if (in_run && resident) {
                /* hit: the running request holds (pins) the block */
                Block *x = &s->blk[b];
                x->pinned = 1;
                if (policy == ORC_S3FIFO) {
                    if (x->list == 0) s->s_unpinned--; else s->m_unpinned--;
                } else {
                    list_unlink(s, (int32_t)b);
                }
                pos_blk[j] = (int32_t)b;
                hit_pos[n_hit++] = (int32_t)j;
                continue;
            }
            in_run = 0;
            if (resident) {
                /* resident block behind the first miss: dropped, then
                   re-materialized as a new block (never an eviction) */
                Block *x = &s->blk[b];
                if (policy == ORC_S3FIFO) {
                    if (x->list == 0) { s->s_size--; s->s_unpinned--; } else s->m_unpinned--;
                }
                drop_block(s, (int32_t)b);
                o[G_ORPHANS]++;
                n_orph++;
            }
            new_pos[n_new++] = (int32_t)j;
        }
        h = n_hit;
        o[G_HITS] += h;
        o[G_MISSES] += n - h;
        o[G_DUPS] += n_dup;
        const int64_t m = n_new;

        /* Alg. 1 OnTouch (debt read before this request's charge) */
        if (policy == ORC_S3FIFO) {
            for (int64_t i = 0; i < n_hit; i++) {
                Block *x = &s->blk[pos_blk[hit_pos[i]]];
                if (x->freq < 3) x->freq++;
            }
        } else if (policy == ORC_PS) {
            const int proven = q_ge1 && s->admitted[p];
            const int64_t d = raw_debt(s, g, t);
            for (int64_t i = 0; i < n_hit; i++) {
                Block *x = &s->blk[pos_blk[hit_pos[i]]];
                if (proven && x->owner == g && x->contract == c && x->prefix == p && x->cls != REUSE) {
                    if (d <= s->eps || (flags & ORC_NO_DEBT_GATE)) {   /* Eq. 4 */
                        x->cls = REUSE; o[G_PROMOTIONS]++;
                    } else {
                        o[G_GATED]++;
                    }
                }
            }
        }

        /* Alg. 2: truly free blocks first, then reclaim e victims.  Under
           StaticQuota the free space is what the requester's partition has
           left, and only its own blocks are reclaimed. */
        int64_t free_now = policy == ORC_SQ ? s->quota - s->resident[g] : s->C - s->resident_total;
        int64_t e = m - free_now;
        if (e < 0) e = 0;
        int64_t P[64], D[64];
        struct timespec ts0 = {0, 0}, ts1 = {0, 0};
        if (reclaim_ns_out) {
            reclaim_ns_out[r] = 0;
            if (e > 0) clock_gettime(CLOCK_MONOTONIC, &ts0);
        }
        if (policy == ORC_PS && e > 0)
            for (int x = 0; x < s->G; x++) { P[x] = norm_debt(s, x, t); D[x] = debt_decrement(s, x, t); }
        for (int64_t i = 0; i < e; i++) {
            int32_t v;
            if (policy == ORC_LRU) v = s->lists[0].head;
            else if (policy == ORC_SQ) v = s->lists[g].head;
            else if (policy == ORC_PS) v = ps_pick(s, P, D);
            else v = s3_evict_one(s);
            if (v < 0) { rc = -3; goto out; }
            Block *x = &s->blk[v];
            s->gs[(int64_t)x->owner * G_NFIELDS + G_EVICTED_OWNED]++;
            o[G_EVICTIONS_CAUSED]++;
            s->is[I_EVICTIONS]++;
            drop_block(s, v);
        }
        if (reclaim_ns_out && e > 0) {
            clock_gettime(CLOCK_MONOTONIC, &ts1);
            reclaim_ns_out[r] = (int64_t)(ts1.tv_sec - ts0.tv_sec) * 1000000000LL + (ts1.tv_nsec - ts0.tv_nsec);
        }

        /* Alg. 1 OnCacheFullBlocks: charge n_r = m new full blocks (Eq. 2),
           choose their initial class, record the successful admission */
        int32_t cls = NORMAL;
        if (m > 0) {
            int64_t B = eff_balance(s, g, c, t) - m * SCALE;
            s->bal[g][c] = B;
            s->last[g][c] = t;
            o[G_CHARGED] += m;
            cls = (B < -s->eps || !s->admitted[p]) ? PROB : NORMAL;
            s->admitted[p] = 1;
        }
        for (int64_t i = m - 1; i >= 0; i--) {       /* deepest block first */
            int64_t j = new_pos[i];
            int32_t b = alloc_block(s);
            if (b < 0) { rc = -3; goto out; }
            Block *x = &s->blk[b];
            memset(x, 0, sizeof(*x));
            x->key = k[j]; x->owner = g; x->contract = c; x->prefix = p;
            x->cls = cls; x->freq = 0; x->pinned = 1; x->list = -1; x->prev = x->next = -1;
            map_put(&s->map, k[j], b);
            s->resident[g]++;
            s->resident_total++;
            pos_blk[j] = b;
            if (policy == ORC_S3FIFO) {
                if (s3_ghost_take(s, k[j])) {
                    list_append(s, 1, b); s->is[I_S3_GHOST_HITS]++;
                } else {
                    list_append(s, 0, b); s->s_size++;
                }
            }
        }

        /* Release: the request's blocks return to the free queue, deepest
           first, so a chain is reclaimed tail-first */
        for (int64_t j = n - 1; j >= 0; j--) {
            if (is_dup[j]) continue;
            Block *x = &s->blk[pos_blk[j]];
            x->pinned = 0;
            if (policy == ORC_S3FIFO) {
                if (x->list == 0) s->s_unpinned++; else s->m_unpinned++;
            } else {
                x->stamp = ++s->stampctr;
                list_append(s, policy == ORC_LRU ? 0 : (policy == ORC_SQ ? x->owner : ps_list(s, x->owner, x->cls)),
                            pos_blk[j]);
            }
        }

        if (per_req_out) {
            per_req_out[4 * r + 0] = (int32_t)h;
            per_req_out[4 * r + 1] = (int32_t)m;
            per_req_out[4 * r + 2] = (int32_t)e;
            per_req_out[4 * r + 3] = (int32_t)n_orph;
        }
        account_all(s, t);
    }
    for (int x = 0; x < s->G; x++) {
        int64_t *o = s->gs + (int64_t)x * G_NFIELDS;
        o[G_DEBT_END] = n_req > 0 ? raw_debt(s, x, t) : 0;
        o[G_RESIDENT_END] = s->resident[x];
    }
    s->is[I_RESIDENT_END] = s->resident_total;
    rc = 0;
out:
    free(s->blk); free(s->free_ids); free(s->lists); free(s->referenced); free(s->admitted);
    free(s->ghost_ring); free(pos_blk); free(hit_pos); free(new_pos); free(is_dup);
    if (s->map.k) map_free(&s->map);
    if (s->ghost.k) map_free(&s->ghost);
    if (seen.k) map_free(&seen);
    return rc;
}

int orc_group_fields(void) { return G_NFIELDS; }
int orc_inst_fields(void) { return I_NFIELDS; }

int orc_replay(const uint64_t *keys, const int64_t *key_off, const uint8_t *group,
               const uint8_t *contract, const uint32_t *prefix, const int64_t *tick,
               int64_t n_req, int32_t n_groups, int64_t n_prefix,
               int32_t policy, int64_t capacity, int32_t flags, int32_t n_contracts,
               const int64_t *rho_q16, const int64_t *beta_q16, int64_t eps_q16,
               int32_t s3_small_permille, int32_t s3_move_threshold,
               int64_t *group_stats_out, int64_t *inst_stats_out, int32_t *per_req_out) {
    return replay_impl(keys, key_off, group, contract, prefix, tick, n_req, n_groups, n_prefix, policy, capacity,
                       flags, n_contracts, rho_q16, beta_q16, eps_q16, s3_small_permille, s3_move_threshold,
                       group_stats_out, inst_stats_out, per_req_out, NULL);
}

/* orc_replay that also times each request's reclamation (reclaim_ns_out). */
int orc_replay_timed(const uint64_t *keys, const int64_t *key_off, const uint8_t *group,
                     const uint8_t *contract, const uint32_t *prefix, const int64_t *tick,
                     int64_t n_req, int32_t n_groups, int64_t n_prefix,
                     int32_t policy, int64_t capacity, int32_t flags, int32_t n_contracts,
                     const int64_t *rho_q16, const int64_t *beta_q16, int64_t eps_q16,
                     int32_t s3_small_permille, int32_t s3_move_threshold,
                     int64_t *group_stats_out, int64_t *inst_stats_out, int32_t *per_req_out,
                     int64_t *reclaim_ns_out) {
    return replay_impl(keys, key_off, group, contract, prefix, tick, n_req, n_groups, n_prefix, policy, capacity,
                       flags, n_contracts, rho_q16, beta_q16, eps_q16, s3_small_permille, s3_move_threshold,
                       group_stats_out, inst_stats_out, per_req_out, reclaim_ns_out);
}
