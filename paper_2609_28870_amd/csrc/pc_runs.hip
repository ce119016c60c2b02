// Exact LRU stack distance from the runs of the prev stream
// (pc_stack_distance_runs).  Same output as pc_stack_distance.
//
// The stack distance of an access is the number of distinct blocks used
// since the previous use of its block (Sec. 5; Appendix B).  With
// v(j) = prev(j) + 1 (0 when cold), #{j < t : v(j) < v(t)} = prev(t) + 1 + D(t),
// so D(t) = Z(t) + C'(t) - prev(t) - 1 with Z(t) the cold accesses before t
// and C'(t) the earlier warm accesses whose previous use is older than t's.
//
// Runs.  Call t a continuation when t - 1 and t are warm and
// prev(t) = prev(t - 1) + 1.  Then the window (prev(t), t) is the window of
// t - 1 without position prev(t) (whose block recurs only at t) and with
// position t - 1 (whose block last occurred at prev(t - 1), outside the new
// window): D(t) = D(t - 1).  A maximal chain of continuations is a run; its
// first access is its head.  Chained block keys make runs long (a request's
// reuse of an earlier request's prefix is one run), about one per request.
//
// Counting over runs.  The previous uses of a run's accesses form the range
// [p, p + len) of positions, p = prev(head); since prev is one-to-one, the
// ranges of different runs are disjoint, so every earlier run lies entirely
// below or above a head's previous use and C'(head of run r) is the sum of
// len(s) over the earlier runs s with p(s) < p(r).  That weighted dominance
// count over the runs is a bottom-up merge by p: at each level an element
// finds its rank in the sibling block by binary search, an element of a
// right block adds the sibling's prefix sum of len at that rank, and the
// merged prefix sums follow from the two blocks' own.
//
// Passes: count heads and cold accesses per 4096-position tile, keeping
// three bits per position (head, cold, last of a run); scan; read the number
// of runs back (the call synchronises once); compact the runs from those
// bits (head's prev, head position, end position, cold count before the
// head); merge levels; write D from the run list.  prev is streamed once.  With
// more runs than 1/16 of the accesses plus 1024 the call runs
// pc_stack_distance instead.
#include "pc_internal.h"

namespace pc {

constexpr int RUN_THREADS = 256;
constexpr int RUN_ITEMS = 16;
constexpr int RUN_TILE = RUN_THREADS * RUN_ITEMS;   // 4096 positions
constexpr int RSCAN_THREADS = 1024;
constexpr int RSCAN_TILE = RSCAN_THREADS * 4;

// header words of the runs workspace
constexpr int RW_STATUS = 0;
constexpr int RW_PATH = 1;    // 0 = runs, 1 = pc_stack_distance
constexpr int RW_RUNS = 2;    // number of runs
constexpr int RW_COLD = 3;    // number of cold accesses
constexpr int RW_RUNS_OK = 4; // 1 = the runs path runs (the gate of its kernels)

// the number of runs (written by the scan)
__device__ __forceinline__ uint64_t runs_of(const int32_t *hdr) { return (uint32_t)hdr[RW_RUNS]; }

// This thread's 16 consecutive prev values and the ones just before and
// after them (from the neighbouring lanes, or from memory across waves and
// tiles).
struct RunView {
    uint32_t p[RUN_ITEMS];
    uint32_t before;   // prev(t0 - 1), NONE at t = 0
    uint32_t after;    // prev(t0 + 16), NONE past the end
    uint64_t t0;
};

__device__ __forceinline__ void load_view(const uint32_t *__restrict__ prev, uint64_t n, RunView &v) {
    const uint64_t tile0 = (uint64_t)blockIdx.x * RUN_TILE;
    v.t0 = tile0 + (uint64_t)threadIdx.x * RUN_ITEMS;
    if (v.t0 + RUN_ITEMS <= n && (reinterpret_cast<uintptr_t>(prev) & 15) == 0) {
        const uint4 *q = reinterpret_cast<const uint4 *>(prev + v.t0);
#pragma unroll
        for (int k = 0; k < RUN_ITEMS / 4; ++k) {
            const uint4 x = q[k];
            v.p[4 * k] = x.x;
            v.p[4 * k + 1] = x.y;
            v.p[4 * k + 2] = x.z;
            v.p[4 * k + 3] = x.w;
        }
    } else {
#pragma unroll
        for (int k = 0; k < RUN_ITEMS; ++k) v.p[k] = v.t0 + k < n ? prev[v.t0 + k] : NONE;
    }
    // neighbours inside the wave by DPP, across waves and tiles from memory
    const int lane = threadIdx.x & (WAVE - 1);
    const uint32_t lo = from_lower(v.p[RUN_ITEMS - 1]);
    const uint32_t hi = from_upper(v.p[0]);
    v.before = lane ? lo : (v.t0 > 0 && v.t0 - 1 < n ? prev[v.t0 - 1] : NONE);
    v.after = lane != WAVE - 1 ? hi : (v.t0 + RUN_ITEMS < n ? prev[v.t0 + RUN_ITEMS] : NONE);
    if (v.t0 + RUN_ITEMS > n) v.after = NONE;
}

// warm t that does not continue t - 1's run
__device__ __forceinline__ bool is_head(uint32_t p, uint32_t before) {
    return p != NONE && (before == NONE || p != before + 1);
}

// Per 4096-position tile: the number of run heads and of cold accesses, and
// per thread (16 positions) three bit masks: heads and cold accesses
// (low / high half of .x) and last accesses of runs (.y).
__global__ __launch_bounds__(RUN_THREADS) void runs_count_kernel(const uint32_t *__restrict__ prev, uint64_t n,
                                                                 uint2 *__restrict__ counts,
                                                                 uint2 *__restrict__ marks) {
    __shared__ uint32_t tmp[RUN_THREADS / WAVE];
    RunView v;
    load_view(prev, n, v);
    uint32_t hm = 0, cm = 0, em = 0;
#pragma unroll
    for (int k = 0; k < RUN_ITEMS; ++k) {
        const uint64_t t = v.t0 + k;
        const uint32_t p = v.p[k];
        if (t < n) {
            if (p == NONE) {
                cm |= 1u << k;
            } else {
                if (is_head(p, k ? v.p[k - 1] : v.before)) hm |= 1u << k;
                // last access of its run: the next one is cold, a head, or past the end
                const uint32_t q = k + 1 < RUN_ITEMS ? v.p[k + 1] : v.after;
                if (t + 1 >= n || q == NONE || q != p + 1) em |= 1u << k;
            }
        }
    }
    marks[(uint64_t)blockIdx.x * RUN_THREADS + threadIdx.x] = make_uint2(hm | (cm << 16), em);
    uint32_t th = 0, tc = 0;
    block_excl_scan((uint32_t)__popc(hm), tmp, &th);
    block_excl_scan((uint32_t)__popc(cm), tmp, &tc);
    if (threadIdx.x == 0) counts[blockIdx.x] = make_uint2(th, tc);
}

// Exclusive scan of the per-tile (heads, cold) pairs: tile sums, one
// workgroup over them (writing the totals to the header), tiles again.
__global__ __launch_bounds__(RSCAN_THREADS) void runs_scan_tiles_kernel(const uint2 *__restrict__ c, uint64_t m,
                                                                        uint2 *__restrict__ tsum) {
    __shared__ uint32_t tmp[RSCAN_THREADS / WAVE];
    const uint64_t t0 = (uint64_t)blockIdx.x * RSCAN_TILE;
    uint32_t a = 0, b = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const uint64_t i = t0 + (uint64_t)k * RSCAN_THREADS + threadIdx.x;
        if (i < m) {
            a += c[i].x;
            b += c[i].y;
        }
    }
    uint32_t ta = 0, tb = 0;
    block_excl_scan(a, tmp, &ta);
    block_excl_scan(b, tmp, &tb);
    if (threadIdx.x == 0) tsum[blockIdx.x] = make_uint2(ta, tb);
}

__global__ __launch_bounds__(RSCAN_THREADS) void runs_scan_top_kernel(uint2 *__restrict__ tsum, uint64_t tiles,
                                                                      int32_t *__restrict__ hdr) {
    __shared__ uint32_t tmp[RSCAN_THREADS / WAVE];
    uint32_t ca = 0, cb = 0;
    for (uint64_t t0 = 0; t0 < tiles; t0 += RSCAN_THREADS) {
        const uint64_t i = t0 + threadIdx.x;
        const uint2 v = i < tiles ? tsum[i] : make_uint2(0u, 0u);
        uint32_t ta = 0, tb = 0;
        const uint32_t ea = block_excl_scan(v.x, tmp, &ta);
        const uint32_t eb = block_excl_scan(v.y, tmp, &tb);
        if (i < tiles) tsum[i] = make_uint2(ca + ea, cb + eb);
        ca += ta;
        cb += tb;
    }
    if (threadIdx.x == 0) {
        hdr[RW_RUNS] = (int32_t)ca;
        hdr[RW_COLD] = (int32_t)cb;
    }
}

__global__ __launch_bounds__(RSCAN_THREADS) void runs_scan_apply_kernel(const uint2 *__restrict__ c, uint64_t m,
                                                                        const uint2 *__restrict__ tsum,
                                                                        uint2 *__restrict__ out) {
    __shared__ uint32_t tmp[RSCAN_THREADS / WAVE];
    const uint64_t i0 = (uint64_t)blockIdx.x * RSCAN_TILE + (uint64_t)threadIdx.x * 4;
    uint2 v[4];
    uint32_t a = 0, b = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        v[k] = i0 + k < m ? c[i0 + k] : make_uint2(0u, 0u);
        a += v[k].x;
        b += v[k].y;
    }
    uint32_t ta = 0, tb = 0;
    uint32_t ra = tsum[blockIdx.x].x + block_excl_scan(a, tmp, &ta);
    uint32_t rb = tsum[blockIdx.x].y + block_excl_scan(b, tmp, &tb);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        if (i0 + k < m) out[i0 + k] = make_uint2(ra, rb);
        ra += v[k].x;
        rb += v[k].y;
    }
}

// Per run s (in time order): p[s] = prev(head), h[s] = head position,
// e[s] = last position, z[s] = cold accesses before the head; from the
// count pass's bit masks, reading prev only at the heads.
__global__ __launch_bounds__(RUN_THREADS) void runs_compact_kernel(const uint32_t *__restrict__ prev, uint64_t n,
                                                                   const uint2 *__restrict__ off,
                                                                   const uint2 *__restrict__ marks,
                                                                   uint32_t *__restrict__ rp, uint32_t *__restrict__ rh,
                                                                   uint32_t *__restrict__ re,
                                                                   uint32_t *__restrict__ rz, uint64_t tiles,
                                                                   const int32_t *__restrict__ hdr) {
    if (!hdr[RW_RUNS_OK]) return;
    __shared__ uint32_t tmp[RUN_THREADS / WAVE];
    for (uint64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
        const uint64_t t0 = tile * RUN_TILE + (uint64_t)threadIdx.x * RUN_ITEMS;
        const uint2 mk = marks[tile * RUN_THREADS + threadIdx.x];
        const uint32_t hm = mk.x & 0xFFFFu, cm = mk.x >> 16, em = mk.y;
        uint32_t th = 0, tc = 0;
        const uint2 o = off[tile];
        const uint32_t hs0 = o.x + block_excl_scan((uint32_t)__popc(hm), tmp, &th);   // runs started before t0
        const uint32_t cs0 = o.y + block_excl_scan((uint32_t)__popc(cm), tmp, &tc);
        // heads: one per set bit, numbered in position order
        for (uint32_t m = hm; m; m &= m - 1) {
            const int k = __builtin_ctz(m);
            const uint32_t below = (1u << k) - 1;
            const uint32_t s = hs0 + (uint32_t)__popc(hm & below);
            rp[s] = prev[t0 + k];
            rh[s] = (uint32_t)(t0 + k);
            rz[s] = cs0 + (uint32_t)__popc(cm & below);
        }
        // run ends: the run is the last one started at or before the position
        for (uint32_t m = em; m; m &= m - 1) {
            const int k = __builtin_ctz(m);
            const uint32_t upto = (k == 31) ? ~0u : (2u << k) - 1;
            re[hs0 + (uint32_t)__popc(hm & upto) - 1] = (uint32_t)(t0 + k);
        }
    }
}

// Level 0: keys p, weights len = e - h + 1 as one-element prefix sums.
__global__ __launch_bounds__(256) void runs_init_kernel(const uint32_t *__restrict__ rp, const uint32_t *__restrict__ rh,
                                                        const uint32_t *__restrict__ re,
                                                        uint32_t *__restrict__ key, uint32_t *__restrict__ pre,
                                                        uint32_t *__restrict__ idx, uint32_t *__restrict__ acc,
                                                        const int32_t *__restrict__ hdr) {
    if (!hdr[RW_RUNS_OK]) return;
    const uint64_t r = runs_of(hdr);
    for (uint64_t s = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; s < r; s += (uint64_t)gridDim.x * blockDim.x) {
        key[s] = rp[s];
        pre[s] = re[s] - rh[s] + 1;
        idx[s] = (uint32_t)s;
        acc[s] = 0;
    }
}

// One merge level: blocks of 2^lvl elements sorted by key with inclusive
// prefix sums of the weights become blocks of 2^(lvl+1).
__global__ __launch_bounds__(256) void runs_merge_kernel(const uint32_t *__restrict__ key, const uint32_t *__restrict__ pre,
                                                         const uint32_t *__restrict__ idx, int lvl,
                                                         uint32_t *__restrict__ key2, uint32_t *__restrict__ pre2,
                                                         uint32_t *__restrict__ idx2, uint32_t *__restrict__ acc,
                                                         const int32_t *__restrict__ hdr) {
    if (!hdr[RW_RUNS_OK]) return;
    const uint64_t r = runs_of(hdr);
    if ((1ull << lvl) >= r) return;   // the merge took fewer levels
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < r; i += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t blk = i >> lvl;
        const uint64_t sb = (blk ^ 1) << lvl;
        uint64_t se = sb + (1ull << lvl);
        if (se > r) se = r;
        const uint32_t k = key[i];
        uint64_t lo = sb, hi = sb < r ? se : sb;   // first sibling key >= k (keys are distinct)
        while (lo < hi) {
            const uint64_t mid = (lo + hi) >> 1;
            if (key[mid] < k) lo = mid + 1;
            else hi = mid;
        }
        const uint64_t rank = lo - sb;
        const uint32_t below = rank ? pre[lo - 1] : 0u;   // sibling weights with smaller keys
        if (blk & 1) acc[idx[i]] += below;                 // the sibling holds the earlier runs
        const uint64_t q = ((blk >> 1) << (lvl + 1)) + (i - (blk << lvl)) + rank;
        key2[q] = k;
        pre2[q] = pre[i] + below;
        idx2[q] = idx[i];
    }
}

// Distance of every run, in place of its cold count: z + acc - p - 1.
__global__ __launch_bounds__(256) void runs_dist_kernel(const uint32_t *__restrict__ rp,
                                                        const uint32_t *__restrict__ acc,
                                                        uint32_t *__restrict__ rz, const int32_t *__restrict__ hdr) {
    if (!hdr[RW_RUNS_OK]) return;
    const uint64_t r = runs_of(hdr);
    for (uint64_t s = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; s < r; s += (uint64_t)gridDim.x * blockDim.x)
        rz[s] = rz[s] + acc[s] - rp[s] - 1;
}

// D of every position from the run list alone: a warm position lies in
// exactly one run [h, e], every other position is cold.  The runs that can
// touch a tile are the one in progress at its start and those starting in
// it; a thread finds the run at its first position by binary search and
// walks on.
__global__ __launch_bounds__(RUN_THREADS) void runs_fill_kernel(uint64_t n, const uint2 *__restrict__ off,
                                                                uint64_t tiles, const uint32_t *__restrict__ rh,
                                                                const uint32_t *__restrict__ re,
                                                                const uint32_t *__restrict__ rd,
                                                                uint32_t *__restrict__ dist,
                                                                const int32_t *__restrict__ hdr) {
    if (!hdr[RW_RUNS_OK]) return;
    const uint64_t r = runs_of(hdr);
    for (uint64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
        // thread i holds positions tile0 + 1024 g + 4 i .. + 3 for g = 0..3
        // (increasing), so each 16-byte store covers 1 KB across the wave
        const uint64_t tile0 = tile * RUN_TILE;
        const uint64_t t0 = tile0 + (uint64_t)threadIdx.x * 4;
        const uint64_t first = off[tile].x;
        const int64_t lo = first ? (int64_t)first - 1 : 0;
        const int64_t hi = tile + 1 < tiles ? (int64_t)off[tile + 1].x : (int64_t)r;
        // last run in [lo, hi) with head <= t0, or lo - 1
        int64_t a = lo, b = hi;
        while (a < b) {
            const int64_t m = (a + b) >> 1;
            if (rh[m] <= t0) a = m + 1;
            else b = m;
        }
        int64_t s = a - 1;
        // the current run's end and distance and the next run's head, in
        // registers: loads only where a run starts
        bool in_run = s >= lo;
        uint64_t end = in_run ? re[s] : 0;
        uint32_t dv = in_run ? rd[s] : NONE;
        uint64_t next_head = s + 1 < hi ? rh[s + 1] : ~0ull;
        const bool vec = (reinterpret_cast<uintptr_t>(dist) & 15) == 0;
    #pragma unroll
        for (int g = 0; g < RUN_ITEMS / 4; ++g) {
            const uint64_t tg = t0 + (uint64_t)g * (RUN_THREADS * 4);
            uint32_t d[4];
    #pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint64_t t = tg + k;
                while (t >= next_head) {
                    ++s;
                    in_run = true;
                    end = re[s];
                    dv = rd[s];
                    next_head = s + 1 < hi ? rh[s + 1] : ~0ull;
                }
                d[k] = (in_run && end >= t) ? dv : NONE;
            }
            if (vec && tg + 4 <= n) {
                *reinterpret_cast<uint4 *>(dist + tg) = make_uint4(d[0], d[1], d[2], d[3]);
            } else {
    #pragma unroll
                for (int k = 0; k < 4; ++k)
                    if (tg + k < n) dist[tg + k] = d[k];
            }
        }
    }
}

__global__ void runs_status_kernel(const int32_t *__restrict__ nested, int32_t *__restrict__ hdr) {
    if (threadIdx.x == 0 && hdr[RW_PATH] && nested[0]) atomicOr(hdr + RW_STATUS, nested[0]);
}

// the path, decided from the number of runs: over runs, or the dominance
// count over accesses when there are more runs than the workspace holds
__global__ void runs_decide_kernel(int32_t *__restrict__ hdr, uint64_t rmax) {
    if (threadIdx.x != 0) return;
    const bool over = runs_of(hdr) > rmax;
    hdr[RW_PATH] = over ? 1 : 0;
    hdr[RW_RUNS_OK] = over ? 0 : 1;
}

static uint64_t runs_max(uint64_t n) { return n / 16 + 1024; }

struct RunsWs {
    int32_t *hdr;
    void *sd;   // pc_stack_distance workspace (the fallback); the arrays below live inside it
    size_t sd_bytes;
    uint2 *counts, *tsum, *off, *marks;
    uint32_t *rp, *rh, *re, *rz, *acc, *key[2], *pre[2], *idx[2];
    size_t bytes;
};

static RunsWs carve_runs(void *ws, uint64_t n) {
    Carver c{(char *)ws, 0};
    RunsWs w;
    w.hdr = c.take<int32_t>(WS_HEADER / sizeof(int32_t));
    w.sd_bytes = pc_stack_distance_ws(n);
    const size_t sd_at = c.off;
    const uint64_t tiles = (n + RUN_TILE - 1) / RUN_TILE;
    const uint64_t rm = runs_max(n);
    w.counts = c.take<uint2>(tiles);
    w.tsum = c.take<uint2>((tiles + RSCAN_TILE - 1) / RSCAN_TILE + 1);
    w.off = c.take<uint2>(tiles);
    w.marks = c.take<uint2>(tiles * RUN_THREADS);
    w.rp = c.take<uint32_t>(rm);
    w.rh = c.take<uint32_t>(rm);
    w.re = c.take<uint32_t>(rm);
    w.rz = c.take<uint32_t>(rm);
    w.acc = c.take<uint32_t>(rm);
    for (int i = 0; i < 2; ++i) {
        w.key[i] = c.take<uint32_t>(rm);
        w.pre[i] = c.take<uint32_t>(rm);
        w.idx[i] = c.take<uint32_t>(rm);
    }
    w.sd = ws ? (char *)ws + sd_at : nullptr;
    const size_t own = c.off;
    w.bytes = own > sd_at + w.sd_bytes ? own : sd_at + w.sd_bytes;
    return w;
}

}  // namespace pc

extern "C" {

size_t pc_stack_distance_runs_ws(uint64_t n) { return pc::carve_runs(nullptr, n).bytes; }

pc_status pc_stack_distance_runs(const uint32_t *prev, const uint32_t *next, uint64_t n, uint32_t *dist, void *ws,
                                 size_t ws_bytes, void *stream) {
    using namespace pc;
    if (n >= (uint64_t)PC_NONE) return PC_ERR_TOO_LARGE;
    if (n > 0 && (!prev || !next || !dist)) return PC_ERR_INVALID;
    if (!ws) return PC_ERR_WORKSPACE;
    if (ws_bytes < pc_stack_distance_runs_ws(n)) return PC_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    const RunsWs w = carve_runs(ws, n);
    pc_status st = fill_u32(reinterpret_cast<uint32_t *>(w.hdr), 0u, 8, s);
    if (st != PC_OK || n == 0) return st;
    const uint64_t tiles = (n + RUN_TILE - 1) / RUN_TILE;
    const uint64_t stiles = (tiles + RSCAN_TILE - 1) / RSCAN_TILE;
    PC_LAUNCH(K_RUNS_COUNT, runs_count_kernel, dim3((unsigned)tiles), dim3(RUN_THREADS), 0, s, prev, n, w.counts,
              w.marks);
    PC_LAUNCH(K_RUNS_SCAN, runs_scan_tiles_kernel, dim3((unsigned)stiles), dim3(RSCAN_THREADS), 0, s,
              (const uint2 *)w.counts, tiles, w.tsum);
    PC_LAUNCH(K_RUNS_SCAN, runs_scan_top_kernel, dim3(1), dim3(RSCAN_THREADS), 0, s, w.tsum, stiles, w.hdr);
    PC_LAUNCH(K_RUNS_SCAN, runs_scan_apply_kernel, dim3((unsigned)stiles), dim3(RSCAN_THREADS), 0, s,
              (const uint2 *)w.counts, tiles, (const uint2 *)w.tsum, w.off);
    // the path is decided on the device, so nothing here waits for the GPU:
    // every later launch is gated on the decision, and the launches of the
    // path not taken return at once (grids capped per compute unit)
    const uint64_t rm = runs_max(n);
    PC_LAUNCH(K_RUNS_SCAN, runs_decide_kernel, dim3(1), dim3(64), 0, s, w.hdr, rm);
    if ((st = stack_distance_gated(prev, next, n, dist, w.sd, s, w.hdr + RW_PATH)) != PC_OK) return st;
    PC_LAUNCH(K_FILL32, runs_status_kernel, dim3(1), dim3(64), 0, s, (const int32_t *)w.sd, w.hdr);
    const int32_t *ok = w.hdr;
    PC_LAUNCH(K_RUNS_COMPACT, runs_compact_kernel, dim3(capped(tiles, 16)), dim3(RUN_THREADS), 0, s, prev, n,
              (const uint2 *)w.off, (const uint2 *)w.marks, w.rp, w.rh, w.re, w.rz, tiles, ok);
    const unsigned rg = capped((rm + 255) / 256, 16);
    PC_LAUNCH(K_RUNS_MERGE, runs_init_kernel, dim3(rg), dim3(256), 0, s, (const uint32_t *)w.rp,
              (const uint32_t *)w.rh, (const uint32_t *)w.re, w.key[0], w.pre[0], w.idx[0], w.acc, ok);
    // one launch per level the largest run count needs; the levels past the
    // actual count return at once
    int cur = 0;
    for (int lvl = 0; (1ull << lvl) < rm; ++lvl) {
        PC_LAUNCH(K_RUNS_MERGE, runs_merge_kernel, dim3(rg), dim3(256), 0, s, (const uint32_t *)w.key[cur],
                  (const uint32_t *)w.pre[cur], (const uint32_t *)w.idx[cur], lvl, w.key[cur ^ 1], w.pre[cur ^ 1],
                  w.idx[cur ^ 1], w.acc, ok);
        cur ^= 1;
    }
    PC_LAUNCH(K_RUNS_MERGE, runs_dist_kernel, dim3(rg), dim3(256), 0, s, (const uint32_t *)w.rp,
              (const uint32_t *)w.acc, w.rz, ok);
    PC_LAUNCH(K_RUNS_FILL, runs_fill_kernel, dim3(capped(tiles, 16)), dim3(RUN_THREADS), 0, s, n,
              (const uint2 *)w.off, tiles, (const uint32_t *)w.rh, (const uint32_t *)w.re, (const uint32_t *)w.rz,
              dist, ok);
    return PC_OK;
}

}  // extern "C"
