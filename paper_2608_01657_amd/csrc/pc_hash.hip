// pc_hash.hip -- block cutting and chained block keys on gfx950.
//
// Block cutting (Sec. III-B: only full KV blocks count): request r owns
// floor(len_r / 16) keys at CSR offset key_off[r].
//
// PCH64 keys (the paper keeps the engine's native content hash, Sec. III-A
// and Sec. IV, so the key function is this library's own):
//   d_k   = sum_{i<8} ((t[16k+2i] + K[2i]) mod 2^32) * ((t[16k+2i+1] + K[2i+1]) mod 2^32)
//   c_k   = fmix64(d_k)
//   H_k   = A * H_{k-1} + c_k  (mod 2^64),  H_-1 = fmix64(ns + 1)
//   key_k = fmix64(H_k)
// The chain is an affine recurrence with an odd multiplier, so it unrolls to
//   H_k = A^k (A H_-1 + sum_{j<=k} A^-j c_j)   (A^-1: the inverse of A mod 2^64)
// and a wavefront computes 64 consecutive H_k as a plain prefix sum of
// A^-j c_j between two per-lane multiplications, instead of a serial loop.
#include "pc_internal.h"

namespace pcr {

namespace {

__constant__ uint32_t kNH[16] = {
    0x3504f334u, 0x5db3d743u, 0x1e3779bau, 0x52a7fa9eu,
    0x28872940u, 0x4d82b447u, 0x0fc1ecd6u, 0x2df0668du,
    0x65ddceafu, 0x314d1496u, 0x48ac80aeu, 0x0a97f66du,
    0x33999334u, 0x475a2544u, 0x6d861707u, 0x23daa40fu};

constexpr uint64_t kA = 0x9E3779B97F4A7C15ull;

constexpr uint64_t pow_a(int e) {
    uint64_t r = 1, b = kA;
    while (e) {
        if (e & 1) r *= b;
        b *= b;
        e >>= 1;
    }
    return r;
}
constexpr uint64_t kA1 = pow_a(1);

// A^-1 mod 2^64 by Newton's iteration x <- x (2 - A x): A x = 1 holds mod 2^3
// for x = A (A odd), and every step doubles the number of correct bits.
constexpr uint64_t inv_a() {
    uint64_t x = kA;
    for (int i = 0; i < 6; ++i) x *= 2 - kA * x;
    return x;
}
constexpr uint64_t kAinv = inv_a();
static_assert(kA * kAinv == 1, "A^-1 mod 2^64");

// b^0 .. b^63: the per-lane multipliers A^L and A^-L of lane L
struct PowTab {
    uint64_t v[64];
    constexpr explicit PowTab(uint64_t b) : v() {
        uint64_t x = 1;
        for (int i = 0; i < 64; ++i) {
            v[i] = x;
            x *= b;
        }
    }
};
__constant__ PowTab kApowL = PowTab(kA);
__constant__ PowTab kAinvL = PowTab(kAinv);

#define GLOBAL __attribute__((address_space(1)))

__device__ __forceinline__ uint64_t fmix64(uint64_t z) {
    z ^= z >> 33;
    z *= 0xff51afd7ed558ccdull;
    z ^= z >> 33;
    z *= 0xc4ceb9fe1a85ec53ull;
    z ^= z >> 33;
    return z;
}

__device__ __forceinline__ uint64_t shfl64(uint64_t v, int src) {
    uint32_t lo = __shfl((int)(uint32_t)v, src);
    uint32_t hi = __shfl((int)(uint32_t)(v >> 32), src);
    return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l) {
    uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)v, l);
    uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
    return ((uint64_t)hi << 32) | lo;
}
// x + x[quad_perm(ctrl)] within each group of 4 lanes (DPP, no LDS)
template <int kCtrl>
__device__ __forceinline__ uint64_t quad_add(uint64_t x) {
    int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)x, kCtrl, 0xF, 0xF, false);
    int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(x >> 32), kCtrl, 0xF, 0xF, false);
    return x + (((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// DPP move of a 64-bit value: lane L receives the source lane kCtrl names
// (row_shr:n = 0x110+n, row_bcast:15 = 0x142, row_bcast:31 = 0x143); lanes
// with no source, and rows outside kRowMask, receive 0.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint64_t dpp64(uint64_t x) {
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)x, kCtrl, kRowMask, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(x >> 32), kCtrl, kRowMask, 0xF, false);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

// Inclusive wavefront sum scan of a 64-bit value in DPP steps (no LDS):
// within each row of 16 lanes, then rows 1 and 3 add the last lane of the
// row before them, then rows 2 and 3 add lane 31.
__device__ __forceinline__ int64_t wave_scan_add64(int64_t x) {
    uint64_t v = (uint64_t)x;
    v += dpp64<0x111, 0xF>(v);
    v += dpp64<0x112, 0xF>(v);
    v += dpp64<0x114, 0xF>(v);
    v += dpp64<0x118, 0xF>(v);
    v += dpp64<0x142, 0xA>(v);
    v += dpp64<0x143, 0xC>(v);
    return (int64_t)v;
}

// ---------------------------------------------------------------- offsets
// Three launches: per-chunk sums (written where the chunk ends), a scan of
// the chunk sums in place, then each chunk's exclusive scan from its base.
// Thread t of a chunk owns its requests 4t..4t+3 (coalesced), and every
// length load is issued before any is used.
constexpr int kScanThreads = 256;
constexpr int kScanChunk = 4 * kScanThreads;

__device__ __forceinline__ int64_t nblocks_of(int32_t len) { return len > 0 ? (int64_t)(len / 16) : 0; }

// blocks of requests start + 4t .. start + 4t + 3 (0 past n); the loads are
// clamped into [0, n) so that none sits under a branch
__device__ __forceinline__ void chunk_blocks(const int32_t *__restrict__ len, int64_t start, int64_t n,
                                             int64_t (&nb)[4]) {
    int32_t x[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t e = start + 4 * threadIdx.x + i;
        x[i] = len[e < n ? e : n - 1];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) nb[i] = start + 4 * threadIdx.x + i < n ? nblocks_of(x[i]) : 0;
}

__device__ int64_t block_incl_scan(int64_t v, int64_t *sh /* [kScanThreads/64] */) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    v = wave_scan_add64(v);
    if (lane == 63) sh[w] = v;
    __syncthreads();
    int64_t add = 0;
    for (int i = 0; i < w; ++i) add += sh[i];
    __syncthreads();
    return v + add;
}

// A: sum of chunk b -> key_off[min((b+1)*CH, n)]
__global__ __launch_bounds__(kScanThreads) void offsets_reduce(const int32_t *__restrict__ len, int64_t n,
                                                               int64_t *__restrict__ key_off) {
    __shared__ int64_t sh[kScanThreads / 64];
    const int64_t start = (int64_t)blockIdx.x * kScanChunk;
    int64_t nb[4];
    chunk_blocks(len, start, n, nb);
    const int64_t s = block_incl_scan(nb[0] + nb[1] + nb[2] + nb[3], sh);
    if (threadIdx.x == kScanThreads - 1) key_off[start + kScanChunk < n ? start + kScanChunk : n] = s;
}

// B: inclusive scan of the chunk sums in place; key_off[0] = 0
__global__ __launch_bounds__(kScanThreads) void offsets_chunks(int64_t n, int64_t nchunks,
                                                               int64_t *__restrict__ key_off) {
    __shared__ int64_t sh[kScanThreads / 64];
    __shared__ int64_t last;
    int64_t carry = 0;
    for (int64_t c0 = 0; c0 < nchunks; c0 += kScanThreads) {
        const int64_t c = c0 + threadIdx.x;
        int64_t pos = 0;
        int64_t v = 0;
        if (c < nchunks) {
            pos = (c + 1) * kScanChunk < n ? (c + 1) * kScanChunk : n;
            v = key_off[pos];
        }
        const int64_t incl = block_incl_scan(v, sh);
        if (c < nchunks) key_off[pos] = carry + incl;
        if (threadIdx.x == kScanThreads - 1) last = incl;
        __syncthreads();
        carry += last;
        __syncthreads();
    }
    if (threadIdx.x == 0) key_off[0] = 0;
}

// C: exclusive scan inside each chunk, starting from the chunk's offset
__global__ __launch_bounds__(kScanThreads) void offsets_fill(const int32_t *__restrict__ len, int64_t n,
                                                             int64_t *__restrict__ key_off) {
    __shared__ int64_t sh[kScanThreads / 64];
    const int64_t start = (int64_t)blockIdx.x * kScanChunk;
    const int64_t base_off = blockIdx.x == 0 ? 0 : key_off[start];
    int64_t nb[4];
    chunk_blocks(len, start, n, nb);
    const int64_t loc = nb[0] + nb[1] + nb[2] + nb[3];
    int64_t run = base_off + block_incl_scan(loc, sh) - loc;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t e = start + 4 * threadIdx.x + i;
        if (e < n) key_off[e] = run;
        run += nb[i];
    }
}

// ---------------------------------------------------------------- keys
// Workgroup sizes of the key kernel (wavefronts), chosen per call by how
// often the tokens are read (launch_hash).
constexpr int kHashWavesStream = 16;
constexpr int kHashWavesReuse = 4;

// Token loads of one 64-block step: lane 4*bq + r4 holds, for q = 0..3,
// tokens [4*r4, 4*r4 + 4) of block 16q + bq of the step.  The loads are
// 16 bytes at 4-byte alignment (a request may start at any token).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_a4 __attribute__((ext_vector_type(4), aligned(4)));
struct Step {
    u32x4 v[4];
};

// Issue every load of the step starting at block `it` before any of them is
// used.  Lanes past the request's last block re-read that block (same cache
// lines, no extra DRAM traffic), so no load sits under a branch and every
// address lies inside the request.
__device__ __forceinline__ void issue(Step &S, const GLOBAL int32_t *__restrict__ tok, int32_t it, int32_t nb,
                                      int bq, int r4) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        int32_t blk = it + 16 * q + bq;
        blk = blk < nb ? blk : nb - 1;
        // byte offset < 2^32: the kernel skips requests of 2^30 tokens or more
        const uint32_t byte = (uint32_t)blk * 64u + (uint32_t)r4 * 16u;
        S.v[q] = *reinterpret_cast<const GLOBAL u32x4_a4 *>(reinterpret_cast<const GLOBAL uint8_t *>(tok) + byte);
    }
}

// Keys of one 64-block step from its loaded tokens; H carries H_{k-1} of
// the step's first block in and the last block's H_k out.
__device__ __forceinline__ void step_keys(const Step &S, int nblk, int lane, int r4, uint32_t k0, uint32_t k1,
                                          uint32_t k2, uint32_t k3, int src, uint64_t apw, uint64_t ainv,
                                          uint64_t &H, GLOBAL uint64_t *__restrict__ out) {
    uint64_t dsel = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const uint32_t t0 = S.v[q].x, t1 = S.v[q].y, t2 = S.v[q].z, t3 = S.v[q].w;
        uint64_t part = (uint64_t)(t0 + k0) * (uint64_t)(t1 + k1) + (uint64_t)(t2 + k2) * (uint64_t)(t3 + k3);
        part = quad_add<0xB1>(part);   // quad_perm [1,0,3,2]
        part = quad_add<0x4E>(part);   // quad_perm [2,3,0,1]
        if (q == r4) dsel = part;      // lane 4b+q keeps block 16q+b
    }
    const uint64_t c = fmix64(dsel);
    // lane L now holds A^-L c of block L of the step; lane 0 also carries
    // the chain in: H_L = A^L (A H + sum_{j<=L} A^-j c_j)
    uint64_t u = shfl64(c, src) * ainv;
    if (lane == 0) u += kA1 * H;
    const uint64_t v = (uint64_t)wave_scan_add64((int64_t)u) * apw;
    H = readlane64(v, nblk - 1);
    // every lane stores (no branch, so the compiler can count the loads in
    // flight exactly): lanes past the last block write the last block's key
    // again, the same value to the same address
    out[lane < nblk ? lane : nblk - 1] = fmix64(lane < nblk ? v : H);
}

// All keys of one request, two steps in flight: the loads of step s+1 are
// issued before step s is computed (two buffers, so no register copy has
// to wait for a load).
__device__ __forceinline__ void hash_request(const GLOBAL int32_t *__restrict__ tok, int32_t nb, uint64_t H,
                                             GLOBAL uint64_t *__restrict__ out, int lane) {
    const int r4 = lane & 3, bq = lane >> 2;
    const uint32_t k0 = kNH[4 * r4], k1 = kNH[4 * r4 + 1], k2 = kNH[4 * r4 + 2], k3 = kNH[4 * r4 + 3];
    const int src = 4 * (lane & 15) + (lane >> 4);      // lane holding block `lane`'s digest
    const uint64_t apw = kApowL.v[lane], ainv = kAinvL.v[lane];
    Step S0, S1;
    issue(S0, tok, 0, nb, bq, r4);
    for (int32_t it = 0;;) {
        issue(S1, tok, it + 64, nb, bq, r4);
        step_keys(S0, nb - it < 64 ? nb - it : 64, lane, r4, k0, k1, k2, k3, src, apw, ainv, H, out + it);
        it += 64;
        if (it >= nb) break;
        issue(S0, tok, it + 64, nb, bq, r4);
        step_keys(S1, nb - it < 64 ? nb - it : 64, lane, r4, k0, k1, k2, k3, src, apw, ainv, H, out + it);
        it += 64;
        if (it >= nb) break;
    }
}

template <int kWaves>
__global__ __launch_bounds__(64 * kWaves) void hash_kernel(
    const int32_t *__restrict__ tokens, int64_t n_tokens, const int64_t *__restrict__ tok_off,
    const int32_t *__restrict__ req_len, const int32_t *__restrict__ req_ns,
    const int64_t *__restrict__ key_off, int64_t n_req, uint64_t *__restrict__ keys, int64_t n_keys,
    int32_t *__restrict__ status) {
    const int lane = threadIdx.x & 63;
    // one request per wavefront (wave-uniform, so the descriptor is read
    // with scalar loads)
    const int64_t r = (int64_t)blockIdx.x * kWaves + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (r >= n_req) return;
    const int64_t off = tok_off[r];
    const int32_t len = req_len[r];
    const int64_t ko = key_off[r];
    const int64_t nb = len > 0 ? len / 16 : 0;
    // a request of 2^30 tokens or more would take byte offsets past 2^32
    if (len < 0 || len >= (1 << 30) || off < 0 || off + (int64_t)len > n_tokens || ko < 0 || ko + nb > n_keys) {
        if (lane == 0) atomicExch(status, -1);
        return;
    }
    if (nb == 0) return;
    const uint64_t H = fmix64((uint64_t)(uint32_t)req_ns[r] + 1u);
    hash_request((const GLOBAL int32_t *)(tokens + off), (int32_t)nb, H, (GLOBAL uint64_t *)(keys + ko), lane);
}

}  // namespace

hipError_t launch_block_offsets(const int32_t *len, int64_t n_req, int64_t *key_off, hipStream_t s) {
    const int64_t nchunks = (n_req + kScanChunk - 1) / kScanChunk;
    if (nchunks > 0)
        hipLaunchKernelGGL(offsets_reduce, dim3((unsigned)nchunks), dim3(kScanThreads), 0, s, len, n_req, key_off);
    hipLaunchKernelGGL(offsets_chunks, dim3(1), dim3(kScanThreads), 0, s, n_req, nchunks, key_off);
    if (nchunks > 0)
        hipLaunchKernelGGL(offsets_fill, dim3((unsigned)nchunks), dim3(kScanThreads), 0, s, len, n_req, key_off);
    return hipGetLastError();
}

hipError_t launch_hash(const int32_t *tokens, int64_t n_tokens, const int64_t *tok_off, const int32_t *len,
                       const int32_t *ns, const int64_t *key_off, int64_t n_req, uint64_t *keys,
                       int64_t n_keys, int32_t *status, hipStream_t s) {
    if (n_req <= 0) return hipSuccess;
    // Requests that each read their own tokens (n_keys full blocks cover at
    // most about twice the token buffer) stream them from HBM: there, 16
    // wavefronts per workgroup take 4 % less time than 4 (a quarter of the
    // workgroups to dispatch; 1.67 vs 1.74 ms on 16 x 50,000 one-touch
    // requests, 8.6 GB).  Requests that re-read shared token ranges (prefix
    // reuse: the re-reads come from L2) are many and short: there, 4-wave
    // workgroups take 18 % less time (5.4 vs 6.6 ms on 64 x 100,000 chat
    // requests), since a workgroup keeps its CU slots until its longest
    // request ends.
    const bool stream = n_keys <= 2 * (n_tokens / 16);
    if (stream) {
        const int64_t blocks = (n_req + kHashWavesStream - 1) / kHashWavesStream;
        hipLaunchKernelGGL(hash_kernel<kHashWavesStream>, dim3((unsigned)blocks), dim3(64 * kHashWavesStream), 0, s,
                           tokens, n_tokens, tok_off, len, ns, key_off, n_req, keys, n_keys, status);
    } else {
        const int64_t blocks = (n_req + kHashWavesReuse - 1) / kHashWavesReuse;
        hipLaunchKernelGGL(hash_kernel<kHashWavesReuse>, dim3((unsigned)blocks), dim3(64 * kHashWavesReuse), 0, s,
                           tokens, n_tokens, tok_off, len, ns, key_off, n_req, keys, n_keys, status);
    }
    return hipGetLastError();
}

}  // namespace pcr
