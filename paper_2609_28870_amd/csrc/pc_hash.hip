// Chained block hashing (pc_hash_blocks).
//
// Block identity is a function of the whole token prefix (a KV state is
// reusable only if everything before it matches, Sec. 2.2); blocks are 16
// tokens (Sec. 3.1).  The hash is fixed in pc.h: splitmix64's finalizer used
// as a step S(x, w) = mix64((x ^ w) + gamma), folded over the block's
// token-pair words from 0 (the digest) and chained block to block.
//
// GPU mapping: one kernel.  The chain is serial inside a request, so a lane
// owns a request and walks it in rounds of up to 32 blocks; the digests of a
// round are independent, so the whole wave computes them first (32 lanes per
// request, one block each, token loads of several requests in flight), puts
// them in an LDS tile with one row per request, and each lane then chains its
// own row.  Keys and depths leave one request at a time (coalesced).  Lanes
// whose request ended take the next one from a global counter, so long and
// short requests mix without idle lanes.  Per 16-token block the work is nine
// splitmix steps (two 64x64 multiplies each), 64 token bytes in and 12 bytes
// out.  The token reads bound it: every turn of a session re-reads the
// session's context, and the same kernel with a near-free digest runs only
// about 5% faster.  With a histogram pointer it also counts the low four
// bytes of every key it writes (LDS, then one global add per bin), which
// the sort takes instead of a counting pass of its own.
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

// any even block size, any 4-byte alignment
__device__ __forceinline__ uint64_t digest_any(const int32_t *p, uint32_t B) {
    uint64_t h = 0;
    for (uint32_t k = 0; k < B; k += 2) h = hstep(h, word((uint32_t)p[k], (uint32_t)p[k + 1]));
    return h;
}

// block sizes that are multiples of 16 from a 16-byte aligned start: the
// same words in the same order, 16 tokens per four 16-byte loads, the loads
// of the next 16 tokens issued before the current ones are folded
__device__ __forceinline__ uint64_t digest_vec16(const int32_t *p, uint32_t B) {
    const uint4 *q = reinterpret_cast<const uint4 *>(p);
    uint64_t h = 0;
    uint4 c0 = q[0], c1 = q[1], c2 = q[2], c3 = q[3];
    for (uint32_t g = 1; g <= B / 16; ++g) {
        uint4 n0 = c0, n1 = c1, n2 = c2, n3 = c3;
        if (g < B / 16) {
            n0 = q[4 * g];
            n1 = q[4 * g + 1];
            n2 = q[4 * g + 2];
            n3 = q[4 * g + 3];
        }
        h = hstep(h, word(c0.x, c0.y));
        h = hstep(h, word(c0.z, c0.w));
        h = hstep(h, word(c1.x, c1.y));
        h = hstep(h, word(c1.z, c1.w));
        h = hstep(h, word(c2.x, c2.y));
        h = hstep(h, word(c2.z, c2.w));
        h = hstep(h, word(c3.x, c3.y));
        h = hstep(h, word(c3.z, c3.w));
        c0 = n0;
        c1 = n1;
        c2 = n2;
        c3 = n3;
    }
    return h;
}

// true when every token and block of request r lies inside the arrays
__device__ __forceinline__ bool request_in_bounds(uint64_t st, uint32_t len, uint32_t nb, uint64_t out,
                                                  uint64_t n_tokens, uint64_t n_blocks) {
    return st <= n_tokens && len <= n_tokens - st && out <= n_blocks && nb <= n_blocks - out;
}


constexpr int GATHER_BATCH = 16;                         // requests per store round

// Both phases in one kernel: the chain kernel's lane-per-request rounds,
// with each round's digests computed in place of being read back from HBM.
// A sweep gives each request of FUSE_ROWS rows a group of FUSE_SPAN lanes
// (lane j of the group hashes block j of the round) and writes the digests
// into the LDS tile; the token loads of FUSE_SWEEPS sweeps are issued
// together.  The digests never touch HBM: a block costs its token bytes in and
// its key and depth out.
constexpr int FUSE_THREADS = 128;
constexpr int FUSE_WAVES = FUSE_THREADS / WAVE;
constexpr int FUSE_SPAN = 32;               // blocks per request per round
constexpr int FUSE_ROWS = WAVE / FUSE_SPAN; // requests per sweep
constexpr int FUSE_ROW = FUSE_SPAN + 1;     // padded LDS row
constexpr int FUSE_SWEEPS = 4;              // sweeps whose loads are in flight together
constexpr int HASH_WAVES_PER_CU = 32;       // waves per CU the request count is spread over

__device__ __forceinline__ uint64_t digest16_words(const uint4 (&q)[4]) {
    uint64_t h = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        h = hstep(h, word(q[i].x, q[i].y));
        h = hstep(h, word(q[i].z, q[i].w));
    }
    return h;
}

__global__ __launch_bounds__(FUSE_THREADS) void hash_fused_kernel(
    const int32_t *__restrict__ tokens, uint64_t n_tokens, const uint64_t *__restrict__ tok_start,
    const uint32_t *__restrict__ tok_len, uint32_t n_seqs, uint32_t B, const uint64_t *__restrict__ parent,
    uint64_t root, const uint64_t *__restrict__ blk_off, uint64_t n_blocks, uint64_t *__restrict__ keys,
    uint32_t *__restrict__ depth, uint32_t *__restrict__ key_hist, uint32_t flags, uint32_t *__restrict__ counter,
    int32_t *__restrict__ err, int lanes) {
    const bool deepest_first = (flags & PC_HASH_DEEPEST_FIRST) != 0;
    __shared__ uint64_t s_tile[FUSE_WAVES][WAVE * FUSE_ROW];
    __shared__ uint32_t s_hist[4 * 256];   // byte histograms of the keys written
    for (int i = threadIdx.x; i < 4 * 256; i += FUSE_THREADS) s_hist[i] = 0;
    __syncthreads();
    const int lane = threadIdx.x & (WAVE - 1);
    const int w = threadIdx.x / WAVE;
    const int grp = lane / FUSE_SPAN;
    const uint32_t jj = (uint32_t)(lane & (FUSE_SPAN - 1));
    uint64_t *tile = s_tile[w];
    // only the first `lanes` lanes take requests (all 64 still hash every
    // round's blocks)
    bool done = lane >= lanes, busy = false;
    uint32_t b = 0, nb = 0, fast = 0;
    uint64_t key = 0, out = 0, st = 0;
    while (true) {
        const bool need = !done && !busy;
        const uint64_t needmask = ballot(need);
        if (needmask) {
            const int leader = __ffsll((unsigned long long)needmask) - 1;
            uint32_t base = 0;
            if (lane == leader) base = atomicAdd(counter, (uint32_t)__popcll(needmask));
            base = __shfl(base, leader, WAVE);
            if (need) {
                // requests are taken last to first: contexts grow turn by
                // turn, so the longest chains start early instead of
                // finishing the kernel alone
                const uint32_t taken = base + mbcnt(needmask);
                const uint32_t r = n_seqs - 1 - taken;
                if (taken >= n_seqs) {
                    done = true;
                } else {
                    const uint32_t len = tok_len[r];
                    st = tok_start[r];
                    nb = len / B;
                    out = blk_off[r];
                    b = 0;
                    key = parent ? parent[r] : root;
                    // 1: B = 16, tokens preloaded; 2: B a multiple of 16, 16-byte loads
                    const bool al = (reinterpret_cast<uintptr_t>(tokens + st) & 15) == 0;
                    fast = (al && B == 16) ? 1u : (al && B % 16 == 0) ? 2u : 0u;
                    if (request_in_bounds(st, len, nb, out, n_tokens, n_blocks)) {
                        busy = nb > 0;
                    } else {
                        atomicOr(err, DEV_ERR_BAD_LAYOUT);
                    }
                }
            }
        }
        const uint64_t active = ballot(busy);
        if (active == 0) {
            if (ballot(!done) == 0) break;
            continue;
        }
        const uint32_t m = busy ? (nb - b < (uint32_t)FUSE_SPAN ? nb - b : (uint32_t)FUSE_SPAN) : 0u;
        // ---- digests of the round's blocks into the tile
        {
            uint64_t act = active;
            while (act) {
                int row[FUSE_SWEEPS];
                bool ok[FUSE_SWEEPS], fr[FUSE_SWEEPS], vq[FUSE_SWEEPS];
                uint64_t addr[FUSE_SWEEPS];
                uint4 tk[FUSE_SWEEPS][4];
#pragma unroll
                for (int q = 0; q < FUSE_SWEEPS; ++q) {
                    // the next FUSE_ROWS requests (wave-uniform); this lane's is number grp
                    int r = -1;
#pragma unroll
                    for (int g = 0; g < FUSE_ROWS; ++g) {
                        int rg = -1;
                        if (act) {
                            rg = __ffsll((unsigned long long)act) - 1;
                            act &= act - 1;
                        }
                        if (g == grp) r = rg;
                    }
                    const int src = r >= 0 ? r : 0;
                    const uint32_t mr = (uint32_t)__shfl((int)m, src, WAVE);
                    const uint32_t br = (uint32_t)__shfl((int)b, src, WAVE);
                    const uint32_t fq = (uint32_t)__shfl((int)fast, src, WAVE);
                    const uint64_t sr = (uint64_t)(uint32_t)__shfl((int)(uint32_t)st, src, WAVE) |
                                        ((uint64_t)(uint32_t)__shfl((int)(uint32_t)(st >> 32), src, WAVE) << 32);
                    row[q] = src;
                    ok[q] = r >= 0 && jj < mr;
                    fr[q] = fq == 1;
                    vq[q] = fq == 2;
                    addr[q] = sr + (uint64_t)(br + jj) * B;
                    if (ok[q] && fr[q]) {
                        const uint4 *p = reinterpret_cast<const uint4 *>(tokens + addr[q]);
                        tk[q][0] = p[0];
                        tk[q][1] = p[1];
                        tk[q][2] = p[2];
                        tk[q][3] = p[3];
                    }
                }
#pragma unroll
                for (int q = 0; q < FUSE_SWEEPS; ++q) {
                    if (ok[q]) {
                        const uint64_t d = fr[q]   ? digest16_words(tk[q])
                                           : vq[q] ? digest_vec16(tokens + addr[q], B)
                                                   : digest_any(tokens + addr[q], B);
                        tile[row[q] * FUSE_ROW + jj] = d;
                    }
                }
            }
        }
        __builtin_amdgcn_wave_barrier();
        // ---- the chain, one request per lane, from LDS
        if (busy) {
            uint64_t *rowp = tile + lane * FUSE_ROW;
            for (uint32_t q = 0; q < m; ++q) {
                key = hstep(key, rowp[q]);
                rowp[q] = key;
            }
        }
        __builtin_amdgcn_wave_barrier();
        // ---- keys and depths of row i back, coalesced per request
        {
            // output position of this round's first block (or, deepest
            // first, of its mirror image inside the request)
            const uint64_t pos = deepest_first ? out + nb - 1 - b : out + b;
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
                        v[q] = tile[i * FUSE_ROW + (lane < FUSE_SPAN ? lane : 0)];
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
                            const uint64_t at = deepest_first ? pi - lane : pi + lane;
                            keys[at] = v[q];
                            if (depth) depth[at] = bi + lane;
                            if (key_hist) {
                                const uint32_t lo = (uint32_t)v[q];
#pragma unroll
                                for (int p = 0; p < 4; ++p) atomicAdd(&s_hist[256 * p + ((lo >> (8 * p)) & 0xFF)], 1u);
                            }
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
    if (key_hist) {
        __syncthreads();
        for (int i = threadIdx.x; i < 4 * 256; i += FUSE_THREADS)
            if (s_hist[i]) atomicAdd(&key_hist[i], s_hist[i]);
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
                         uint32_t *key_hist, uint32_t flags, void *ws, size_t ws_bytes, void *stream) {
    if (block_size < 2 || block_size > 1024 || (block_size & 1)) return PC_ERR_INVALID;
    if (n_seqs >= 0x80000000u) return PC_ERR_TOO_LARGE;
    if (n_blocks >= (uint64_t)PC_NONE) return PC_ERR_TOO_LARGE;
    if (n_seqs > 0 && (!tokens || !tok_start || !tok_len || !blk_off)) return PC_ERR_INVALID;
    if (n_blocks > 0 && !keys) return PC_ERR_INVALID;
    if (!ws) return PC_ERR_WORKSPACE;
    if (ws_bytes < pc_hash_blocks_ws(n_seqs)) return PC_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    if (key_hist) {
        const pc_status hs = pc::fill_u32(key_hist, 0u, 4 * 256, s);
        if (hs != PC_OK) return hs;
    }
    if (n_seqs == 0 || n_blocks == 0) return PC_OK;

    pc::Carver c{(char *)ws, 0};
    int32_t *hdr = c.take<int32_t>(pc::WS_HEADER / sizeof(int32_t));
    uint32_t *counters = c.take<uint32_t>(2);
    pc_status st = pc::fill_u32(reinterpret_cast<uint32_t *>(hdr), 0u, 1, s);
    if (st != PC_OK) return st;
    st = pc::fill_u32(counters, 0u, 2, s);
    if (st != PC_OK) return st;

    const int cus = pc::device_cus();
    // Persistent grid: a few workgroups per CU, requests handed out by a
    // counter.  A wave's lanes advance their requests in lockstep rounds and
    // share the round's digest work, so a wave that holds many long requests
    // (the late turns of one large session arrive together) works for as
    // long as all of them take.  With few requests per resident wave, fewer
    // lanes per wave take requests (at least 8): the long ones spread over
    // more waves and the slowest wave finishes sooner.
    const uint64_t resident_waves = (uint64_t)cus * pc::HASH_WAVES_PER_CU;
    uint64_t lanes = ((uint64_t)n_seqs + resident_waves - 1) / resident_waves;
    lanes = lanes < 8 ? 8 : lanes > (uint64_t)pc::WAVE ? (uint64_t)pc::WAVE : lanes;
    const uint64_t per_wg = lanes * pc::FUSE_WAVES;
    uint64_t want = ((uint64_t)n_seqs + per_wg - 1) / per_wg;
    uint64_t cap = (uint64_t)cus * 8;
    unsigned grid = (unsigned)(want < cap ? want : cap);
    if (grid == 0) grid = 1;
    PC_LAUNCH(pc::K_HASH, pc::hash_fused_kernel, dim3(grid), dim3(pc::FUSE_THREADS), 0, s, tokens, n_tokens,
              tok_start, tok_len, n_seqs, block_size, parent, root, blk_off, n_blocks, keys, depth, key_hist,
              flags, counters, hdr, (int)lanes);
    return PC_OK;
}

}  // extern "C"
