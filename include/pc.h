/*
 * pc.h -- C ABI of the MI355X prefix-cache replay library (libpcreplay.so).
 *
 * The library runs the data-parallel hot path of PrefixShield (arXiv
 * 2608.01657): cutting token sequences into full 16-token KV blocks with
 * chained 64-bit block keys, and replaying many independent multi-tenant
 * prefix-cache instances (LRU, S3-FIFO, PrefixShield) over those keys, one
 * GPU workgroup (four wavefronts) per instance, with admission debt metered
 * per accounting group.
 *
 * Conventions (every entry point):
 *   - Pointers named d_* are DEVICE pointers owned by the caller; they must
 *     stay valid until the work queued on `stream` has completed.  The
 *     library never allocates device memory.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     All calls except pc_get_stats and pc_last_error are asynchronous.
 *   - Return value: PC_OK (0) or a negative PC_E* code; pc_last_error()
 *     then describes the failure.  Host-side validation happens before any
 *     device work is queued; a rejected call queues nothing.
 *   - Everything is integer: keys are uint64, balances and debts are int64
 *     in Q16 fixed point (2^16 = one block).
 */
#ifndef PC_H
#define PC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PC_OK 0
#define PC_EINVAL (-1)        /* bad argument (null pointer, size, range, ...)        */
#define PC_ENOMEM (-2)        /* caller-provided workspace too small                  */
#define PC_EDEVICE (-3)       /* HIP runtime or launch error                          */
#define PC_EUNSUPPORTED (-4)  /* a parameter the GPU path does not implement          */
#define PC_EINTERNAL (-5)     /* internal table overflow (never expected)             */

#define PC_BLOCK_TOKENS 16    /* the only block size the GPU path implements          */
#define PC_MAX_GROUPS 64
#define PC_MAX_CONTRACTS 4
#define PC_MAX_CAPACITY 32767

/* Thread-local description of the last failure on this host thread. */
const char *pc_last_error(void);

/* ------------------------------------------------------------------------
 * Block cutting.  Each request is cut into floor(len / 16) full blocks; a
 * partial tail gets no key (Sec. III-B: only full KV blocks are metered).
 *
 * pc_block_offsets: d_key_off[r] = sum_{i<r} floor(d_req_len[i] / 16) for
 * r = 0..n_req (n_req+1 int64 values, CSR offsets of each request's keys).
 * d_req_len values must be >= 0 (negative lengths count as 0 blocks).
 * ------------------------------------------------------------------------ */
int32_t pc_block_offsets(const int32_t *d_req_len, int64_t n_req, int32_t block_size,
                         int64_t *d_key_off, void *stream);

/* ------------------------------------------------------------------------
 * Chained block keys (PCH64; the paper keeps the serving engine's native
 * content hash, Sec. III-A and IV, so this key is the library's own).
 * For a request in namespace ns (its accounting group, Sec. II-C) with
 * tokens t (int32, reinterpreted as uint32):
 *   d_k   = sum_{i<8} ((t[16k+2i] + K[2i]) mod 2^32) * ((t[16k+2i+1] + K[2i+1]) mod 2^32)  mod 2^64
 *   H_-1  = fmix64(ns + 1),  H_k = A*H_{k-1} + fmix64(d_k) mod 2^64,  key_k = fmix64(H_k)
 * where fmix64 is the MurmurHash3 finalizer, A = 0x9E3779B97F4A7C15 and
 * K[i] = floor(frac(sqrt(p_i)) * 2^31) + 1 for the first 16 primes.
 *
 *   d_tokens   [n_tokens] int32, 4-byte aligned (else PC_EINVAL); a
 *              request may start at any token, and requests may alias.
 *   d_req_tok_off, d_req_len, d_req_ns  [n_req]: start, length, namespace;
 *              a request holds fewer than 2^30 tokens (4 GiB).
 *   d_key_off  [n_req+1] output of pc_block_offsets (or any offsets with
 *              room for floor(len/16) keys per request).
 *   d_keys     [n_keys] output.
 *   d_status   one int32 in device memory, set to PC_EINVAL by the kernel if
 *              any request's token or key range falls outside the buffers,
 *              or its length is negative or 2^30 or more (that request is
 *              skipped); the caller zeroes it beforehand.
 * ------------------------------------------------------------------------ */
int32_t pc_hash_blocks(const int32_t *d_tokens, int64_t n_tokens,
                       const int64_t *d_req_tok_off, const int32_t *d_req_len,
                       const int32_t *d_req_ns, const int64_t *d_key_off, int64_t n_req,
                       int32_t block_size, uint64_t *d_keys, int64_t n_keys,
                       int32_t *d_status, void *stream);

/* ------------------------------------------------------------------------
 * Replay.
 * ------------------------------------------------------------------------ */
/* Policies (Sec. V-A): LRU is the engine's free-queue order; S3-FIFO and
 * StaticQuota are the paper's baselines; PrefixShield is its method (Sec.
 * III).  StaticQuota gives every accounting group a fixed partition of
 * floor(capacity / n_groups) blocks with LRU inside it and no borrowing: a
 * request probes at most its partition (the rest counts as truncated) and
 * reclaims only its own group's blocks. */
enum { PC_LRU = 0, PC_S3FIFO = 1, PC_PREFIXSHIELD = 2, PC_STATICQUOTA = 3 };
enum { PC_FLAG_NO_SEGMENTATION = 1,   /* Sec. V-D ablation: one retention segment    */
       PC_FLAG_NO_DEBT_GATE = 2 };    /* Sec. V-D ablation: promote regardless of debt */

/* One request trace, all arrays in device memory.  Request r probes the
 * keys d_keys[d_key_off[r] .. d_key_off[r+1]).  Group = accounting group
 * (also the lookup namespace), contract = service contract, prefix =
 * logical prefix id, dense per (group, prefix) (Sec. III-A).  Ticks are the
 * monotonic accounting clock (Eq. 1); NULL means tick = request index. */
typedef struct {
    const uint64_t *d_keys;
    const int64_t *d_key_off;      /* [n_req+1], non-decreasing, within [0, n_keys] */
    const uint8_t *d_group;        /* [n_req] < n_groups                            */
    const uint8_t *d_contract;     /* [n_req] < the instance's n_contracts          */
    const uint32_t *d_prefix;      /* [n_req] < n_prefix                            */
    const int64_t *d_tick;         /* [n_req] >= 0, non-decreasing, or NULL         */
    int64_t n_req;
    int64_t n_keys;
    int64_t n_prefix;
    int32_t n_groups;              /* 1..64                                         */
    int32_t max_req_blocks;        /* >= every d_key_off[r+1]-d_key_off[r]          */
} pc_trace_desc;

/* A service contract (Eqs. 1-2).  The contracts of one instance are weighted
 * by w_c = rho_c / rho_min (Eq. 5), and 1/w_c is kept in Q16, so their refill
 * rates may differ by a factor 2^16 at most (else PC_EINVAL): Eq. 8's
 * per-victim decrement 1/W_g is then at least one Q16 unit. */
typedef struct {
    int64_t rho_q16;               /* refill rate per tick, > 0 (Prop. 1), <= 2^40  */
    int64_t beta_q16;              /* burst capacity, 0..2^50                        */
} pc_contract;

typedef struct {
    int32_t trace;                 /* index into the traces array                  */
    int32_t policy;                /* PC_LRU / PC_S3FIFO / PC_PREFIXSHIELD /
                                      PC_STATICQUOTA                                */
    int32_t capacity;              /* usable blocks, 1..PC_MAX_CAPACITY             */
    int32_t flags;                 /* PC_FLAG_*                                     */
    int32_t n_contracts;           /* 1..4                                          */
    int32_t s3_small_permille;     /* S3-FIFO small-queue share, 0..1000 (100)      */
    int32_t s3_move_threshold;     /* S3-FIFO small->main access count, >= 0 (1)    */
    int32_t reserved;              /* must be 0                                     */
    int64_t eps_q16;               /* debt tolerance epsilon, 0..2^50 (Sec. III-B)  */
    pc_contract contract[PC_MAX_CONTRACTS];
} pc_instance_desc;

/* Per instance, per accounting group; exact integers. */
typedef struct {
    uint64_t requests, probes, hits, misses, charged, evicted_owned, evictions_caused,
        promotions, gated, orphans, dups, truncated;
    int64_t debt_end_q16;          /* raw debt D_g (Eq. 3) at the last request's tick */
    int64_t debt_max_q16;          /* max over requests of D_g after the request      */
    int64_t debt_sum_q16;          /* sum over requests of D_g after the request      */
    int64_t resident_end, resident_max;
} pc_group_stats;

typedef struct {
    uint64_t evictions, s3_moves, s3_reinserts, s3_ghost_hits, s3_ghost_inserts;
    int64_t resident_end, resident_max;
    int32_t status;                /* PC_OK, or PC_EINVAL if a request was malformed
                                      (the instance stopped there; counters zeroed) */
    int32_t reserved;
} pc_instance_stats;

/* Device stats record of one instance: 64 pc_group_stats then one
 * pc_instance_stats.  d_stats for n_inst instances needs
 * n_inst * PC_STATS_RECORD_BYTES bytes. */
#define PC_STATS_RECORD_BYTES (64 * 136 + 64)

/* Workspace bytes pc_replay_batch needs for this batch (< 0: invalid input,
 * see pc_last_error). */
int64_t pc_replay_workspace_bytes(const pc_trace_desc *traces, int32_t n_traces,
                                  const pc_instance_desc *inst, int32_t n_inst);

/* Per-instance replay state (the cache metadata: block keys and metadata,
 * stamps, the free-queue log, the block and ghost tables, per-request
 * scratch) that pc_replay_batch would use for this batch: bytes_out[i]
 * bytes, laid out as layout_out[i] says:
 *   PC_LAYOUT_LDS     all of it in LDS
 *   PC_LAYOUT_HYBRID  block keys and prefix ids in the workspace, the rest
 *                     in LDS (chosen when it lets more instances share a CU)
 *   PC_LAYOUT_WS      all of it in the workspace (when it does not fit LDS)
 * Host only; validates like pc_replay_workspace_bytes.  The per-prefix
 * bitmaps and the S3-FIFO ghost ring live in the workspace and are not
 * counted. */
#define PC_LAYOUT_LDS 0
#define PC_LAYOUT_HYBRID 1
#define PC_LAYOUT_WS 2
int32_t pc_replay_state_bytes(const pc_trace_desc *traces, int32_t n_traces,
                              const pc_instance_desc *inst, int32_t n_inst,
                              int64_t *bytes_out, int32_t *layout_out);

/* Replay every instance over its trace, one workgroup per instance; queued
 * on `stream` (instances of different LDS footprints run as separate
 * launches on library streams that fork from and join back into it).  Per request it runs the hooks of Alg. 1 (OnRequest, OnTouch
 * with the debt gate of Eq. 4, OnCacheFullBlocks metering Eqs. 1-3) and,
 * when the cache is full, the reclamation of Alg. 2 (PrefixShield: Eqs. 5-9;
 * LRU, S3-FIFO and StaticQuota: the baselines of Sec. V-A) under the same
 * debt accounting.
 *   d_workspace   device memory of at least pc_replay_workspace_bytes()
 *                 bytes, 256-byte aligned; its contents need not be zeroed.
 *   d_stats       n_inst * PC_STATS_RECORD_BYTES bytes, written at the end.
 *   d_per_request optional (NULL): per-request int32 quadruples (hits, new
 *                 blocks, evictions, orphans); instance i's block starts at
 *                 4 * sum_{j<i} traces[inst[j].trace].n_req.
 * Instances are independent; their order does not affect any result. */
int32_t pc_replay_batch(const pc_trace_desc *traces, int32_t n_traces,
                        const pc_instance_desc *inst, int32_t n_inst,
                        void *d_workspace, int64_t workspace_bytes, void *d_stats,
                        int32_t *d_per_request, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops and harnesses that forbid allocation): the same
 * replay as pc_replay_batch, with the workspace taken from a static device
 * array of PC_STATIC_WORKSPACE_BYTES that the library holds on every GPU it
 * runs on, until the process ends.  The call allocates no device memory and
 * no pinned host memory; the caller still passes d_stats and d_per_request
 * (as for pc_replay_batch).
 *   - A batch whose workspace (pc_replay_workspace_bytes) exceeds
 *     PC_STATIC_WORKSPACE_BYTES is rejected with PC_ENOMEM, queuing nothing.
 *   - Every call on one GPU uses that GPU's one array.  The kernels clear
 *     what they need, so a call never depends on an earlier call's
 *     contents, but calls whose work overlaps on one GPU (other streams, or
 *     another host thread) race on the array and give undefined results:
 *     order them on one stream.
 *   - The descriptor upload copies from pageable host memory, which the
 *     runtime has read when the call returns. */
#define PC_STATIC_WORKSPACE_BYTES (64LL << 20)
int32_t pc_replay_batch_static(const pc_trace_desc *traces, int32_t n_traces,
                               const pc_instance_desc *inst, int32_t n_inst, void *d_stats,
                               int32_t *d_per_request, void *stream);

/* Synchronize `stream`, copy the stats of one instance (or of all n_inst
 * when instance == -1) to the host and decode them: per-group hits, misses
 * and evictions, charged blocks (Eq. 2), the raw debt D_g of Eq. 3 (final,
 * maximum and sum over requests, whose mean is the "mean debt" of Sec. V-D)
 * and occupancy (Table III).
 *   groups_out  [max_groups] (or [n_inst][max_groups] for instance == -1)
 *   inst_out    [1] (or [n_inst]) */
int32_t pc_get_stats(const void *d_stats, int32_t n_inst, int32_t instance,
                     pc_group_stats *groups_out, int32_t max_groups,
                     pc_instance_stats *inst_out, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* PC_H */
