// Hit-ratio and compute-savings histograms (pc_mrc_weighted).
//
// The block hit ratio counts every access, compulsory misses included
// (Sec. 3.2); the compute-savings ratio weights each hit by the recompute
// cost it avoids over the cost of all accesses (Sec. 5.2), with a cost that
// grows with the block's depth (Sec. 4.4; linear model in Appendix C):
// cost(t) = alpha + beta * depth[t].  Because LRU hits at capacity c exactly
// when D < c, binning D on the capacity edges gives every capacity at once.
//
// GPU mapping: each thread takes 8 consecutive accesses (16 when the depths
// come from the layout; 16-byte vector loads of dist / depth / next) and keeps the value range of the bin it is
// filling in registers, so an access that stays in that bin (neighbouring
// accesses of one request usually do) costs two compares; any other value
// finds its bin by an upper-bound search of the edges held in LDS.  Runs of
// equal bins are accumulated in registers, so one LDS atomic covers a run;
// each workgroup then adds its non-zero LDS bins to the outputs with global
// 64-bit atomics.  Up to 1024 edges sit in LDS at once; more are taken 1024
// at a time, one launch each, a launch counting only the accesses that fall
// between its edges.  Integer atomics make the result independent of
// scheduling order.  A last tiny kernel forms alpha*count + beta*depthsum
// exactly as 128-bit integers.
//
// pc_mrc_weighted_layout takes the depths from the request layout instead
// of an array: depth(t) = t - (start of t's request).  A map kernel writes a
// bitmap of every request start and, per 64 positions, the start of the
// request holding the first; a thread of the bins kernel finds its first
// access's request start from those (the last start bit at or below it in
// its 64-position word, else the word's entry) and follows the start bits
// across its accesses: 12 bytes of map per 64 accesses instead of 256 bytes
// of depth.  In the deepest-first layout (request-level residency)
// depth(t) = (last position of t's request) - t: the bitmap marks every
// request's last position and the table holds, per 64 positions, the last
// position of the request holding the word's last one; a thread looks up
// from its last access and follows the marks down.
#include "pc_internal.h"

namespace pc {

constexpr int MRC_THREADS = 256;

// number of edges <= x (edges non-decreasing)
__device__ __forceinline__ uint32_t upper_bound(const uint32_t *e, uint32_t m, uint32_t x) {
    uint32_t lo = 0, hi = m;
    while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if (e[mid] <= x) lo = mid + 1; else hi = mid;
    }
    return lo;
}

// consecutive accesses per thread: 8 with a depth array (32 registers of
// loads per lane keep eight waves per SIMD), 16 with depths from the layout
// (its map lookup per thread then covers twice the accesses: 4.6 -> 3.3 ms
// on the full trace)
template <bool LAYOUT> constexpr int mrc_per() { return LAYOUT ? 16 : 8; }
constexpr uint32_t MRC_EDGES = 1024;   // edges held in LDS by one launch

// Distances and gaps are 32-bit and NONE (no previous or next use) is the
// largest 32-bit value; edges are held clamped to it, min(edge, NONE).  A
// value x <= NONE - 1 is at or above an edge exactly when it is at or above
// the clamped edge, and NONE is at or above every clamped edge, so it lands
// in the last bin with no special case.
//
// The bin a value falls in and the range [lo, hi] of values that share it.
// With several launches (CHUNKED) a value outside this launch's edges gets
// the local bin K + 1, which is never written out: below `below` (the edge
// before this launch's first), or at or above its last edge while later
// edges remain.
struct BinRange {
    uint32_t lo, hi, bin;
};

__device__ __forceinline__ uint32_t clamp_edge(uint64_t e) { return e < NONE ? (uint32_t)e : NONE; }

template <bool CHUNKED>
__device__ __forceinline__ BinRange find_bin(const uint32_t *e, uint32_t K, uint32_t x, uint32_t below,
                                             bool last) {
    const uint32_t b = upper_bound(e, K, x);
    BinRange r{b ? e[b - 1] : 0u, b < K ? e[b] - 1 : NONE, b};
    if (CHUNKED) {
        if (b == 0 && x < below) r = BinRange{0u, below - 1, K + 1};
        else if (b == 0) r.lo = below;
        else if (b == K && !last) r.bin = K + 1;
    }
    return r;
}

// One launch covers bins k0 .. k0 + Kc of the n_caps + 1 (the last of them
// only when k0 + Kc == n_caps) with its Kc edges caps[k0 .. k0 + Kc) in LDS.
template <bool CHUNKED, bool LAYOUT>
__global__ __launch_bounds__(MRC_THREADS) void mrc_hist_kernel(
    const uint32_t *__restrict__ dist, const uint32_t *__restrict__ depth,
    const uint32_t *__restrict__ gstart, const uint8_t *__restrict__ startbits,
    const uint32_t *__restrict__ next, uint64_t n, const uint64_t *__restrict__ caps, uint32_t n_caps,
    uint32_t k0, uint32_t Kc, uint64_t *__restrict__ count, uint64_t *__restrict__ depthsum,
    uint64_t *__restrict__ nexthist, int desc, int32_t *__restrict__ err) {
    extern __shared__ uint64_t smem[];
    const uint32_t K = Kc;
    uint64_t *s_ds = smem;                    // K+2
    uint32_t *s_cnt = reinterpret_cast<uint32_t *>(s_ds + K + 2);   // K+2
    uint32_t *s_nh = s_cnt + K + 2;           // K+2
    uint32_t *s_caps = s_nh + K + 2;          // K, clamped to NONE
    const bool last = !CHUNKED || k0 + K == n_caps;
    const uint32_t below = CHUNKED && k0 ? clamp_edge(caps[k0 - 1]) : 0u;
    for (uint32_t i = threadIdx.x; i < K; i += blockDim.x) {
        s_caps[i] = clamp_edge(caps[k0 + i]);
        if (blockIdx.x == 0 && k0 + i + 1 < n_caps && caps[k0 + i] > caps[k0 + i + 1])
            atomicOr(err, DEV_ERR_BAD_CAPS);
    }
    for (uint32_t i = threadIdx.x; i < K + 2; i += blockDim.x) {
        s_ds[i] = 0;
        s_cnt[i] = 0;
        s_nh[i] = 0;
    }
    __syncthreads();
    constexpr int MRC_PER = mrc_per<LAYOUT>();
    const uint64_t chunks = (n + MRC_PER - 1) / MRC_PER;
    // vector loads only when every base pointer is 16-byte aligned
    const bool vec = ((reinterpret_cast<uintptr_t>(dist) | reinterpret_cast<uintptr_t>(depth) |
                       reinterpret_cast<uintptr_t>(next)) & 15) == 0;
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t ch = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; ch < chunks; ch += stride) {
        const uint64_t t0 = ch * MRC_PER;
        const bool full = t0 + MRC_PER <= n;
        uint32_t dv[MRC_PER], pv[MRC_PER], nv[MRC_PER];
        if (full && vec) {
#pragma unroll
            for (int q = 0; q < MRC_PER / 4; ++q) {
                const uint4 a = reinterpret_cast<const uint4 *>(dist + t0)[q];
                dv[4 * q] = a.x; dv[4 * q + 1] = a.y; dv[4 * q + 2] = a.z; dv[4 * q + 3] = a.w;
                if (depth) {
                    const uint4 b = reinterpret_cast<const uint4 *>(depth + t0)[q];
                    pv[4 * q] = b.x; pv[4 * q + 1] = b.y; pv[4 * q + 2] = b.z; pv[4 * q + 3] = b.w;
                }
                if (next) {
                    const uint4 c = reinterpret_cast<const uint4 *>(next + t0)[q];
                    nv[4 * q] = c.x; nv[4 * q + 1] = c.y; nv[4 * q + 2] = c.z; nv[4 * q + 3] = c.w;
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < MRC_PER; ++j) {
                const bool in = t0 + j < n;
                dv[j] = in ? dist[t0 + j] : 0u;
                pv[j] = (in && depth) ? depth[t0 + j] : 0u;
                nv[j] = (in && next) ? next[t0 + j] : 0u;
            }
        }
        if (LAYOUT) {
            const uint64_t wd = t0 >> 6;
            const uint64_t bits = reinterpret_cast<const uint64_t *>(startbits)[wd];
            const uint32_t sh = (uint32_t)(t0 & 63);   // a multiple of MRC_PER, at most 64 - MRC_PER
            const uint32_t sb = (uint32_t)(bits >> sh);
            if (!desc) {
                // the last request start at or below t0 (in the 64-position
                // word, else the word's entry), then the starts among the
                // thread's accesses
                const uint64_t upto = bits & ((2ull << sh) - 1);
                uint32_t st = upto ? (uint32_t)((wd << 6) + 63 - __builtin_clzll(upto)) : gstart[wd];
#pragma unroll
                for (int j = 0; j < MRC_PER; ++j) {
                    if (j && ((sb >> j) & 1u)) st = (uint32_t)(t0 + j);
                    pv[j] = (uint32_t)(t0 + j) - st;
                }
            } else {
                // the first request end at or above t0 + 7 (in the word, else
                // the word's entry), then the ends among the thread's accesses
                const uint64_t from = bits >> (sh + MRC_PER - 1);
                uint32_t en = from ? (uint32_t)((wd << 6) + sh + MRC_PER - 1 + __builtin_ctzll(from)) : gstart[wd];
#pragma unroll
                for (int j = MRC_PER - 1; j >= 0; --j) {
                    if (j < MRC_PER - 1 && ((sb >> j) & 1u)) en = (uint32_t)(t0 + j);
                    pv[j] = en - (uint32_t)(t0 + j);
                }
            }
        } else if (!depth) {
#pragma unroll
            for (int j = 0; j < MRC_PER; ++j) pv[j] = 0;
        }
        const int m = full ? MRC_PER : (int)(n - t0);
        // current bins (range empty at the start: lo > hi)
        BinRange cur{1u, 0u, K + 2}, ncur{1u, 0u, K + 2};
        uint32_t cnt = 0, ncnt = 0;
        uint64_t ds = 0;
        for (int j = 0; j < m; ++j) {
            const uint32_t d = dv[j];
            if (d < cur.lo || d > cur.hi) {
                if (cnt) {
                    atomicAdd(&s_cnt[cur.bin], cnt);
                    if (ds) atomicAdd(reinterpret_cast<unsigned long long *>(&s_ds[cur.bin]), (unsigned long long)ds);
                }
                cur = find_bin<CHUNKED>(s_caps, K, d, below, last);
                cnt = 0;
                ds = 0;
            }
            ++cnt;
            ds += pv[j];
            if (next) {
                const uint32_t q = nv[j];
                const uint32_t g = q == NONE ? NONE : q - (uint32_t)(t0 + j);
                if (g < ncur.lo || g > ncur.hi) {
                    if (ncnt) atomicAdd(&s_nh[ncur.bin], ncnt);
                    ncur = find_bin<CHUNKED>(s_caps, K, g, below, last);
                    ncnt = 0;
                }
                ++ncnt;
            }
        }
        if (cnt) {
            atomicAdd(&s_cnt[cur.bin], cnt);
            if (ds) atomicAdd(reinterpret_cast<unsigned long long *>(&s_ds[cur.bin]), (unsigned long long)ds);
        }
        if (ncnt) atomicAdd(&s_nh[ncur.bin], ncnt);
    }
    __syncthreads();
    for (uint32_t i = threadIdx.x; i <= K; i += blockDim.x) {
        if (s_cnt[i]) atomicAdd(reinterpret_cast<unsigned long long *>(&count[k0 + i]), (unsigned long long)s_cnt[i]);
        if (s_ds[i])
            atomicAdd(reinterpret_cast<unsigned long long *>(&depthsum[k0 + i]), (unsigned long long)s_ds[i]);
        if (next && s_nh[i])
            atomicAdd(reinterpret_cast<unsigned long long *>(&nexthist[k0 + i]), (unsigned long long)s_nh[i]);
    }
}

// The layout map, one thread per request: bit t of startbits set when a
// request starts at t (the bitmap is zeroed first), and gstart[w] = the
// start of the request holding position 64w; in the deepest-first layout
// (desc) bit t marks a request's last position and gstart[w] holds the last
// position of the request holding the word's last one.  Checks the layout as
// pc_prev_next_chained does.
__global__ __launch_bounds__(256) void mrc_map_kernel(const uint64_t *__restrict__ off, uint32_t n_seqs, uint64_t n,
                                                      int desc, uint32_t *__restrict__ gstart,
                                                      uint32_t *__restrict__ startbits, int32_t *__restrict__ err) {
    const uint64_t r = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= n_seqs) return;
    const uint64_t a = off[r], b = off[r + 1];
    bool ok = a <= b && b <= n;
    if (r == 0) ok = ok && a == 0;
    if (r + 1 == n_seqs) ok = ok && b == n;
    if (!ok) {
        atomicOr(err, DEV_ERR_BAD_LAYOUT);
        return;
    }
    if (a == b) return;
    if (!desc) {
        atomicOr(&startbits[a >> 5], 1u << (a & 31));
        for (uint64_t w = (a + 63) / 64; w * 64 < b; ++w) gstart[w] = (uint32_t)a;
    } else {
        const uint64_t e = b - 1, words = (n + 63) / 64;
        atomicOr(&startbits[e >> 5], 1u << (e & 31));
        // words whose last position (n - 1 for the last word) lies in [a, b)
        for (uint64_t w = a / 64; w < words; ++w) {
            const uint64_t last = 64 * w + 63 < n ? 64 * w + 63 : n - 1;
            if (last >= b) break;
            gstart[w] = (uint32_t)e;
        }
    }
}

// cost = alpha*count + beta*depthsum as a 128-bit integer (hi:lo), mod 2^128
__global__ void mrc_cost_kernel(const uint64_t *__restrict__ count, const uint64_t *__restrict__ depthsum,
                                uint32_t bins, uint64_t alpha, uint64_t beta, uint64_t *__restrict__ lo,
                                uint64_t *__restrict__ hi) {
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= bins) return;
    const uint64_t c = count[i], d = depthsum[i];
    const uint64_t a_lo = alpha * c, a_hi = __umul64hi(alpha, c);
    const uint64_t b_lo = beta * d, b_hi = __umul64hi(beta, d);
    const uint64_t s = a_lo + b_lo;
    lo[i] = s;
    hi[i] = a_hi + b_hi + (s < a_lo ? 1ull : 0ull);
}


// workspace of pc_mrc_weighted_layout: the header, gstart (one word per 64
// positions) and the start bitmap (one bit per position, whole 64-bit words)
struct MrcLayoutWs {
    int32_t *hdr;
    uint32_t *gstart, *startbits;
    size_t bytes;
};
static MrcLayoutWs mrc_layout_carve(void *ws, uint64_t n) {
    MrcLayoutWs w{};
    char *base = static_cast<char *>(ws);
    size_t off = 0;
    w.hdr = reinterpret_cast<int32_t *>(base);
    off += WS_HEADER;
    const uint64_t words = (n + 63) / 64;
    w.gstart = reinterpret_cast<uint32_t *>(base + off);
    off = align_up(off + words * sizeof(uint32_t));
    w.startbits = reinterpret_cast<uint32_t *>(base + off);
    off = align_up(off + words * sizeof(uint64_t));
    w.bytes = off;
    return w;
}

// both entry points: depths from `depth` (or none), or from the layout
// blk_off (then ws is a layout workspace)
static pc_status mrc_run(const uint32_t *dist, const uint32_t *depth, const uint64_t *blk_off, uint32_t n_seqs,
                         int desc, const uint32_t *next, uint64_t n, const uint64_t *caps, uint32_t n_caps, uint64_t alpha,
                         uint64_t beta, uint64_t *count, uint64_t *depthsum, uint64_t *cost_lo, uint64_t *cost_hi,
                         uint64_t *nextuse_hist, void *ws, size_t ws_bytes, hipStream_t s) {
    (void)ws_bytes;
    if (n >= (uint64_t)PC_NONE) return PC_ERR_TOO_LARGE;
    if (n_caps == 0 || n_caps > PC_MAX_CAPS) return PC_ERR_INVALID;
    if (!caps || !count || !depthsum || !cost_lo || !cost_hi) return PC_ERR_INVALID;
    if (n > 0 && !dist) return PC_ERR_INVALID;
    if (next && !nextuse_hist) return PC_ERR_INVALID;
    if (!ws) return PC_ERR_WORKSPACE;
    int32_t *hdr = reinterpret_cast<int32_t *>(ws);
    const uint32_t bins = n_caps + 1;
    pc_status st;
    if ((st = fill_u32(reinterpret_cast<uint32_t *>(hdr), 0u, 1, s)) != PC_OK) return st;
    if ((st = fill_u32(reinterpret_cast<uint32_t *>(count), 0u, 2 * (size_t)bins, s)) != PC_OK) return st;
    if ((st = fill_u32(reinterpret_cast<uint32_t *>(depthsum), 0u, 2 * (size_t)bins, s)) != PC_OK) return st;
    if (nextuse_hist && (st = fill_u32(reinterpret_cast<uint32_t *>(nextuse_hist), 0u, 2 * (size_t)bins, s)) != PC_OK)
        return st;

    const int cus = device_cus();
    const bool layout = blk_off != nullptr;
    const MrcLayoutWs lw = mrc_layout_carve(ws, n);
    if (layout && n > 0) {
        if (n_seqs == 0) return fill_u32(reinterpret_cast<uint32_t *>(hdr), (uint32_t)DEV_ERR_BAD_LAYOUT, 1, s);
        if ((st = fill_u32(lw.startbits, 0u, 2 * ((n + 63) / 64), s)) != PC_OK) return st;
        PC_LAUNCH(K_MRC_MAP, mrc_map_kernel, dim3((unsigned)(((uint64_t)n_seqs + 255) / 256)), dim3(256), 0, s,
                  blk_off, n_seqs, n, desc, lw.gstart, lw.startbits, hdr);
    }
    const uint32_t *gs = layout ? lw.gstart : nullptr;
    const uint8_t *sb = layout ? reinterpret_cast<const uint8_t *>(lw.startbits) : nullptr;
    const uint64_t per = layout ? mrc_per<true>() : mrc_per<false>();
    uint64_t grid = (n + MRC_THREADS * per - 1) / (MRC_THREADS * per);
    // up to 64 workgroups per CU: eight resident (32 registers of loads per
    // lane keep eight waves per SIMD) and the rest queued behind them, which
    // hid the load latency best; more make the final flush contend
    if (grid > (uint64_t)cus * 64) grid = (uint64_t)cus * 64;
    if (grid == 0) grid = 1;
    for (uint32_t k0 = 0; k0 < n_caps; k0 += MRC_EDGES) {
        const uint32_t Kc = n_caps - k0 < MRC_EDGES ? n_caps - k0 : MRC_EDGES;
        const size_t shmem = (size_t)(Kc + 2) * 16 + (size_t)Kc * 4;
        const bool chunked = n_caps > MRC_EDGES;
        if (!chunked && !layout)
            PC_LAUNCH(K_MRC_HIST, (mrc_hist_kernel<false, false>), dim3((unsigned)grid), dim3(MRC_THREADS), shmem,
                      s, dist, depth, gs, sb, next, n, caps, n_caps, k0, Kc, count, depthsum, nextuse_hist, desc, hdr);
        else if (!chunked)
            PC_LAUNCH(K_MRC_HIST, (mrc_hist_kernel<false, true>), dim3((unsigned)grid), dim3(MRC_THREADS), shmem,
                      s, dist, depth, gs, sb, next, n, caps, n_caps, k0, Kc, count, depthsum, nextuse_hist, desc, hdr);
        else if (!layout)
            PC_LAUNCH(K_MRC_HIST, (mrc_hist_kernel<true, false>), dim3((unsigned)grid), dim3(MRC_THREADS), shmem,
                      s, dist, depth, gs, sb, next, n, caps, n_caps, k0, Kc, count, depthsum, nextuse_hist, desc, hdr);
        else
            PC_LAUNCH(K_MRC_HIST, (mrc_hist_kernel<true, true>), dim3((unsigned)grid), dim3(MRC_THREADS), shmem,
                      s, dist, depth, gs, sb, next, n, caps, n_caps, k0, Kc, count, depthsum, nextuse_hist, desc, hdr);
    }
    PC_LAUNCH(K_MRC_COST, mrc_cost_kernel, dim3((bins + 255) / 256), dim3(256), 0, s, count, depthsum, bins, alpha,
              beta, cost_lo, cost_hi);
    return PC_OK;
}

}  // namespace pc

extern "C" {

size_t pc_mrc_weighted_ws(uint64_t n, uint32_t n_caps) {
    (void)n;
    (void)n_caps;
    return pc::WS_HEADER;
}

pc_status pc_mrc_weighted(const uint32_t *dist, const uint32_t *depth, const uint32_t *next, uint64_t n,
                          const uint64_t *caps, uint32_t n_caps, uint64_t alpha, uint64_t beta,
                          uint64_t *count, uint64_t *depthsum, uint64_t *cost_lo, uint64_t *cost_hi,
                          uint64_t *nextuse_hist, void *ws, size_t ws_bytes, void *stream) {
    if (n >= (uint64_t)PC_NONE) return PC_ERR_TOO_LARGE;
    if (ws && ws_bytes < pc_mrc_weighted_ws(n, n_caps)) return PC_ERR_WORKSPACE;
    return pc::mrc_run(dist, depth, nullptr, 0, 0, next, n, caps, n_caps, alpha, beta, count, depthsum, cost_lo, cost_hi,
                       nextuse_hist, ws, ws_bytes, (hipStream_t)stream);
}

size_t pc_mrc_weighted_layout_ws(uint64_t n, uint32_t n_caps) {
    (void)n_caps;
    return pc::mrc_layout_carve(nullptr, n).bytes;
}

pc_status pc_mrc_weighted_layout(const uint32_t *dist, const uint64_t *blk_off, uint32_t n_seqs, uint32_t flags,
                                 const uint32_t *next, uint64_t n, const uint64_t *caps, uint32_t n_caps,
                                 uint64_t alpha, uint64_t beta, uint64_t *count, uint64_t *depthsum, uint64_t *cost_lo,
                                 uint64_t *cost_hi, uint64_t *nextuse_hist, void *ws, size_t ws_bytes, void *stream) {
    if (n >= (uint64_t)PC_NONE) return PC_ERR_TOO_LARGE;
    if (n > 0 && !blk_off) return PC_ERR_INVALID;
    if (flags & ~PC_HASH_DEEPEST_FIRST) return PC_ERR_INVALID;
    if (ws && ws_bytes < pc_mrc_weighted_layout_ws(n, n_caps)) return PC_ERR_WORKSPACE;
    return pc::mrc_run(dist, nullptr, blk_off, n_seqs, (flags & PC_HASH_DEEPEST_FIRST) ? 1 : 0, next, n, caps, n_caps, alpha, beta, count, depthsum, cost_lo,
                       cost_hi, nextuse_hist, ws, ws_bytes, (hipStream_t)stream);
}

}  // extern "C"
