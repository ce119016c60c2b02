// Chained block hashing (pc_hash_blocks).
//
// Block identity is a function of the whole token prefix (a KV state is
// reusable only if everything before it matches, Sec. 2.2); blocks are 16
// tokens (Sec. 3.1).  The hash is fixed in pc.h: splitmix64's finalizer used
// as a step S(x, w) = mix64((x ^ w) + gamma), folded over the block's
// token-pair words from 0 (the digest) and chained block to block.
//
// GPU mapping, two phases.  (1) Digests are independent per block: one wave
// takes one request and lane j hashes block j, so a wave reads 4 KiB of
// tokens in one coalesced sweep and writes 64 digests contiguously.  (2) The
// chain is serial inside a request: one lane owns one request and walks its
// digests in place; the digests move between HBM and an LDS tile one request
// at a time (coalesced 512-byte accesses) and are chained from LDS.  A wave
// refills lanes from a global request counter as their requests end, so long
// and short requests mix without idle lanes.  Per 16-token block the
// work is nine splitmix steps (two 64x64 multiplies each) and 64 bytes of
// tokens read.
#include "pc_internal.h"

namespace pc {

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__device__ __forceinline__ uint64_t hstep(uint64_t x, uint64_t w) {
    return mix64((x ^ w) + 0x9E3779B97F4A7C15ull);
}

__device__ __forceinline__ uint64_t word(uint32_t a, uint32_t b) {
    return (uint64_t)a | ((uint64_t)b << 32);
}

// digest of one 16-token block at a 16-byte aligned address
__device__ __forceinline__ uint64_t digest16(const int32_t *p) {
    const uint4 *q = reinterpret_cast<const uint4 *>(p);
    uint4 a = q[0], b = q[1], c = q[2], d = q[3];
    uint64_t h = 0;
    h = hstep(h, word(a.x, a.y));
    h = hstep(h, word(a.z, a.w));
    h = hstep(h, word(b.x, b.y));
    h = hstep(h, word(b.z, b.w));
    h = hstep(h, word(c.x, c.y));
    h = hstep(h, word(c.z, c.w));
    h = hstep(h, word(d.x, d.y));
    h = hstep(h, word(d.z, d.w));
    return h;
}

// any even block size, any 4-byte alignment
__device__ __forceinline__ uint64_t digest_any(const int32_t *p, uint32_t B) {
    uint64_t h = 0;
    for (uint32_t k = 0; k < B; k += 2) h = hstep(h, word((uint32_t)p[k], (uint32_t)p[k + 1]));
    return h;
}

constexpr int HASH_THREADS = 256;

// true when every token and block of request r lies inside the arrays
__device__ __forceinline__ bool request_in_bounds(uint64_t st, uint32_t len, uint32_t nb, uint64_t out,
                                                  uint64_t n_tokens, uint64_t n_blocks) {
    return st <= n_tokens && len <= n_tokens - st && out <= n_blocks && nb <= n_blocks - out;
}

// Phase 1: digests.  One wave per request, lane = block: a wave reads 64
// consecutive 64-byte token blocks (4 KiB, fully coalesced) and writes 64
// consecutive 8-byte digests into the key array.  Requests come from an
// atomic counter so long and short requests balance across waves.
__global__ __launch_bounds__(HASH_THREADS) void hash_digest_kernel(
    const int32_t *__restrict__ tokens, uint64_t n_tokens, const uint64_t *__restrict__ tok_start,
    const uint32_t *__restrict__ tok_len, uint32_t n_seqs, uint32_t B,
    const uint64_t *__restrict__ blk_off, uint64_t n_blocks, uint64_t *__restrict__ keys,
    uint32_t *__restrict__ counter, int32_t *__restrict__ err) {
    const int lane = threadIdx.x & (WAVE - 1);
    while (true) {
        uint32_t r = 0;
        if (lane == 0) r = atomicAdd(counter, 1u);
        r = __shfl(r, 0, WAVE);
        if (r >= n_seqs) break;
        const uint32_t len = tok_len[r];
        const uint64_t st = tok_start[r];
        const uint32_t nb = len / B;
        const uint64_t out = blk_off[r];
        if (!request_in_bounds(st, len, nb, out, n_tokens, n_blocks)) {
            if (lane == 0) atomicOr(err, DEV_ERR_BAD_LAYOUT);
            continue;
        }
        const int32_t *tp = tokens + st;
        const bool fast = (B == 16) && ((reinterpret_cast<uintptr_t>(tp) & 15) == 0);
        for (uint32_t j = lane; j < nb; j += WAVE) {
            const int32_t *p = tp + (uint64_t)j * B;
            keys[out + j] = fast ? digest16(p) : digest_any(p, B);
        }
    }
}

// Phase 2: the chain, serial inside a request.  A wave owns up to 64
// requests (one per lane) and advances all of them by up to 32 blocks per
// round.  Memory moves per request, not per lane: for each of its requests
// the wave loads the next 32 digests with one coalesced 256-byte access into
// an LDS tile (row = request, padded against bank conflicts), every lane then
// chains its own row in LDS, and the keys (and depths) go back the same way.
// Lanes whose request ended take the next one from an atomic counter at the
// start of the round.
__device__ __forceinline__ uint64_t readlane64(uint64_t v, int i) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, i);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), i);
    return (uint64_t)lo | ((uint64_t)hi << 32);
}

constexpr int CHAIN_THREADS = 128;                       // two waves per workgroup
constexpr int CHAIN_WAVES = CHAIN_THREADS / WAVE;
constexpr int CHAIN_SPAN = 32;                           // blocks per request per round
constexpr int CHAIN_ROW = CHAIN_SPAN + 1;                // padded LDS row
constexpr int GATHER_BATCH = 16;                         // requests per load round

__global__ __launch_bounds__(CHAIN_THREADS) void hash_chain_kernel(
    const uint32_t *__restrict__ tok_len, uint32_t n_seqs, uint32_t B,
    const uint64_t *__restrict__ parent, uint64_t root, const uint64_t *__restrict__ blk_off,
    uint64_t n_blocks, uint64_t *__restrict__ keys, uint32_t *__restrict__ depth,
    uint32_t *__restrict__ counter) {
    __shared__ uint64_t s_tile[CHAIN_WAVES][WAVE * CHAIN_ROW];
    const int lane = threadIdx.x & (WAVE - 1);
    const int w = threadIdx.x / WAVE;
    uint64_t *tile = s_tile[w];
    bool done = false, busy = false;
    uint32_t b = 0, nb = 0;
    uint64_t key = 0, out = 0;
    while (true) {
        const bool need = !done && !busy;
        const uint64_t needmask = ballot(need);
        if (needmask) {
            const int leader = __ffsll((unsigned long long)needmask) - 1;
            uint32_t base = 0;
            if (lane == leader) base = atomicAdd(counter, (uint32_t)__popcll(needmask));
            base = __shfl(base, leader, WAVE);
            if (need) {
                const uint32_t r = base + mbcnt(needmask);
                if (r >= n_seqs) {
                    done = true;
                } else {
                    nb = tok_len[r] / B;
                    out = blk_off[r];
                    b = 0;
                    key = parent ? parent[r] : root;
                    // phase 1 wrote digests only for in-bounds requests
                    busy = nb > 0 && out <= n_blocks && nb <= n_blocks - out;
                }
            }
        }
        const uint64_t active = ballot(busy);
        if (active == 0) {
            if (ballot(!done) == 0) break;
            continue;
        }
        const uint32_t m = busy ? (nb - b < (uint32_t)CHAIN_SPAN ? nb - b : (uint32_t)CHAIN_SPAN) : 0u;
        const uint64_t pos = out + b;
        // gather: row i <- the next m_i digests of lane i's request.  Loads
        // for GATHER_BATCH requests are issued before their LDS stores, so a
        // round waits for a few memory latencies instead of one per request.
        {
            uint64_t act = active;
            while (act) {
                int ids[GATHER_BATCH];
                uint64_t v[GATHER_BATCH];
#pragma unroll
                for (int q = 0; q < GATHER_BATCH; ++q) {
                    ids[q] = -1;
                    v[q] = 0;
                    if (act) {
                        const int i = __ffsll((unsigned long long)act) - 1;   // wave-uniform
                        act &= act - 1;
                        ids[q] = i;
                        const uint32_t mi = (uint32_t)__builtin_amdgcn_readlane((int)m, i);
                        const uint64_t pi = readlane64(pos, i);
                        if ((uint32_t)lane < mi) v[q] = keys[pi + lane];
                    }
                }
#pragma unroll
                for (int q = 0; q < GATHER_BATCH; ++q) {
                    if (ids[q] >= 0) {
                        const uint32_t mi = (uint32_t)__builtin_amdgcn_readlane((int)m, ids[q]);
                        if ((uint32_t)lane < mi) tile[ids[q] * CHAIN_ROW + lane] = v[q];
                    }
                }
            }
        }
        __builtin_amdgcn_wave_barrier();
        if (busy) {
            uint64_t *row = tile + lane * CHAIN_ROW;
            for (uint32_t j = 0; j < m; ++j) {
                key = hstep(key, row[j]);
                row[j] = key;
            }
        }
        __builtin_amdgcn_wave_barrier();
        // scatter back: keys and depths of row i, coalesced (LDS reads for a
        // batch of requests first, then their stores)
        {
            uint64_t act = active;
            while (act) {
                int ids[GATHER_BATCH];
                uint64_t v[GATHER_BATCH];
#pragma unroll
                for (int q = 0; q < GATHER_BATCH; ++q) {
                    ids[q] = -1;
                    v[q] = 0;
                    if (act) {
                        const int i = __ffsll((unsigned long long)act) - 1;
                        act &= act - 1;
                        ids[q] = i;
                        v[q] = tile[i * CHAIN_ROW + (lane < CHAIN_SPAN ? lane : 0)];
                    }
                }
#pragma unroll
                for (int q = 0; q < GATHER_BATCH; ++q) {
                    if (ids[q] >= 0) {
                        const int i = ids[q];
                        const uint32_t mi = (uint32_t)__builtin_amdgcn_readlane((int)m, i);
                        const uint64_t pi = readlane64(pos, i);
                        const uint32_t bi = (uint32_t)__builtin_amdgcn_readlane((int)b, i);
                        if ((uint32_t)lane < mi) {
                            keys[pi + lane] = v[q];
                            if (depth) depth[pi + lane] = bi + lane;
                        }
                    }
                }
            }
        }
        __builtin_amdgcn_wave_barrier();
        if (busy) {
            b += m;
            busy = b < nb;
        }
    }
}

}  // namespace pc

extern "C" {

size_t pc_hash_blocks_ws(uint32_t n_seqs) {
    (void)n_seqs;
    return pc::WS_HEADER + pc::WS_ALIGN;   // header + two work counters
}

pc_status pc_hash_blocks(const int32_t *tokens, uint64_t n_tokens, const uint64_t *tok_start,
                         const uint32_t *tok_len,
                         uint32_t n_seqs, uint32_t block_size, const uint64_t *parent, uint64_t root,
                         const uint64_t *blk_off, uint64_t n_blocks, uint64_t *keys, uint32_t *depth,
                         void *ws, size_t ws_bytes, void *stream) {
    if (block_size < 2 || block_size > 1024 || (block_size & 1)) return PC_ERR_INVALID;
    if (n_seqs >= 0x80000000u) return PC_ERR_TOO_LARGE;
    if (n_blocks >= (uint64_t)PC_NONE) return PC_ERR_TOO_LARGE;
    if (n_seqs > 0 && (!tokens || !tok_start || !tok_len || !blk_off)) return PC_ERR_INVALID;
    if (n_blocks > 0 && !keys) return PC_ERR_INVALID;
    if (!ws) return PC_ERR_WORKSPACE;
    if (ws_bytes < pc_hash_blocks_ws(n_seqs)) return PC_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    if (n_seqs == 0 || n_blocks == 0) return PC_OK;

    pc::Carver c{(char *)ws, 0};
    int32_t *hdr = c.take<int32_t>(pc::WS_HEADER / sizeof(int32_t));
    uint32_t *counters = c.take<uint32_t>(2);
    pc_status st = pc::fill_u32(reinterpret_cast<uint32_t *>(hdr), 0u, 1, s);
    if (st != PC_OK) return st;
    st = pc::fill_u32(counters, 0u, 2, s);
    if (st != PC_OK) return st;

    const int cus = pc::device_cus();
    // persistent grids: a few workgroups per CU, work handed out by counters
    uint64_t want = ((uint64_t)n_seqs * pc::WAVE + pc::HASH_THREADS - 1) / pc::HASH_THREADS;
    uint64_t cap = (uint64_t)cus * 8;
    unsigned grid = (unsigned)(want < cap ? want : cap);
    if (grid == 0) grid = 1;
    PC_LAUNCH(pc::K_HASH_DIGEST, pc::hash_digest_kernel, dim3(grid), dim3(pc::HASH_THREADS), 0, s,
              tokens, n_tokens, tok_start, tok_len, n_seqs, block_size, blk_off, n_blocks, keys,
              counters, hdr);
    want = ((uint64_t)n_seqs + pc::CHAIN_THREADS - 1) / pc::CHAIN_THREADS;
    cap = (uint64_t)cus * 8;
    grid = (unsigned)(want < cap ? want : cap);
    if (grid == 0) grid = 1;
    PC_LAUNCH(pc::K_HASH, pc::hash_chain_kernel, dim3(grid), dim3(pc::CHAIN_THREADS), 0, s, tok_len,
              n_seqs, block_size, parent, root, blk_off, n_blocks, keys, depth, counters + 1);
    return PC_OK;
}

}  // extern "C"
