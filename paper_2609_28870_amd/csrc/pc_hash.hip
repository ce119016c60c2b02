// Chained block hashing (pc_hash_blocks).
//
// Block identity is a function of the whole token prefix (a KV state is
// reusable only if everything before it matches, Sec. 2.2); blocks are 16
// tokens (Sec. 3.1).  The hash is fixed in pc.h: splitmix64's finalizer used
// as a step S(x, w) = mix64((x ^ w) + gamma), folded over the block's
// token-pair words from 0 (the digest) and chained block to block.
//
// GPU mapping.  The chain is serial inside a request, so one lane owns one
// request at a time and walks its blocks in order; the wave keeps all 64
// lanes busy by refilling a lane from a global request counter (one atomic
// per wave refill) as soon as its request ends, so long and short requests
// mix without leaving lanes idle.  A lane reads its block's 16 tokens as four
// 16-byte loads (one 64-byte segment) and writes the 8-byte key (and the
// depth) to the request's slice of the output.  The step is integer ALU work
// (two 64x64 multiplies per step, nine steps per 16-token block).
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
constexpr int HASH_CHUNK = 16;   // blocks a lane hashes between refills

__global__ __launch_bounds__(HASH_THREADS) void hash_blocks_kernel(
    const int32_t *__restrict__ tokens, uint64_t n_tokens, const uint64_t *__restrict__ tok_start,
    const uint32_t *__restrict__ tok_len, uint32_t n_seqs, uint32_t B,
    const uint64_t *__restrict__ parent, uint64_t root, const uint64_t *__restrict__ blk_off,
    uint64_t n_blocks, uint64_t *__restrict__ keys, uint32_t *__restrict__ depth,
    uint32_t *__restrict__ counter, int32_t *__restrict__ err) {
    const int lane = threadIdx.x & (WAVE - 1);
    bool done = false;
    bool busy = false;
    uint32_t b = 0, nb = 0;
    uint64_t key = 0, out = 0;
    const int32_t *tp = nullptr;
    bool fast = false;

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
                    const uint32_t len = tok_len[r];
                    const uint64_t st = tok_start[r];
                    nb = len / B;
                    b = 0;
                    key = parent ? parent[r] : root;
                    tp = tokens + st;
                    out = blk_off[r];
                    fast = (B == 16) && ((reinterpret_cast<uintptr_t>(tp) & 15) == 0);
                    busy = nb > 0;
                    // never touch memory outside the caller's arrays
                    if (st > n_tokens || len > n_tokens - st || out > n_blocks ||
                        nb > n_blocks - out) {
                        busy = false;
                        atomicOr(err, DEV_ERR_BAD_LAYOUT);
                    }
                }
            }
        }
        if (ballot(!done) == 0) break;
#pragma unroll 1
        for (int it = 0; it < HASH_CHUNK; ++it) {
            if (busy) {
                const int32_t *p = tp + (uint64_t)b * B;
                const uint64_t d = fast ? digest16(p) : digest_any(p, B);
                key = hstep(key, d);
                keys[out + b] = key;
                if (depth) depth[out + b] = b;
                ++b;
                busy = b < nb;
            }
        }
    }
}

}  // namespace pc

extern "C" {

size_t pc_hash_blocks_ws(uint32_t n_seqs) {
    (void)n_seqs;
    return pc::WS_HEADER + pc::WS_ALIGN;
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
    uint32_t *counter = c.take<uint32_t>(1);
    pc_status st = pc::fill_u32(reinterpret_cast<uint32_t *>(hdr), 0u, 1, s);
    if (st != PC_OK) return st;
    st = pc::fill_u32(counter, 0u, 1, s);
    if (st != PC_OK) return st;

    const int cus = pc::device_cus();
    // persistent grid: enough waves to fill every SIMD several times over
    uint64_t want = ((uint64_t)n_seqs + pc::HASH_THREADS - 1) / pc::HASH_THREADS;
    uint64_t cap = (uint64_t)cus * 8;
    unsigned grid = (unsigned)(want < cap ? want : cap);
    if (grid == 0) grid = 1;
    PC_LAUNCH(pc::K_HASH, pc::hash_blocks_kernel, dim3(grid), dim3(pc::HASH_THREADS), 0, s,
              tokens, n_tokens, tok_start, tok_len, n_seqs, block_size, parent, root, blk_off,
              n_blocks, keys, depth, counter, hdr);
    return PC_OK;
}

}  // extern "C"
