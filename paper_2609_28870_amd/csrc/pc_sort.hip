// Previous / next use of every access (pc_prev_next_use).
//
// prev[t] = last earlier position with the same key, next[t] = first later
// one.  The paper's offline analysis ranks blocks by time until next access
// (Sec. 3.2 Belady; Sec. 5.2 BeladyCompute); prev == none marks a compulsory
// miss (Sec. 4.6).
//
// GPU mapping: a stable LSD radix sort of (key, t) groups equal keys with t
// ascending; neighbours in sorted order are exactly the (prev, next) links.
// Keys are 64-bit hashes, so sorting by their low 32 bits already makes
// equal keys contiguous except where different keys share those bits; the
// link step resolves such short "mixed" runs by scanning them, and when a
// run is too long to scan it flags the four passes over the high bits and a
// second link (then the full 64-bit sort makes equal keys adjacent).
//   * the four 8-bit digit histograms of a group of passes come from the
//     caller (the hash kernel counts them while it writes the keys) or from
//     one counting pass (LDS-privatised, then global atomics); one workgroup
//     scans them into digit bases;
//   * each of the eight sort passes is a single "onesweep" kernel: a
//     workgroup takes the next tile from an atomic counter (so every tile it
//     waits on is already running), ranks its 8192 elements by digit with
//     wave ballots (stable: lanes in order, waves in order), publishes its
//     per-digit counts and reads its predecessors' with a decoupled
//     look-back, then writes the tile out through LDS so each digit run is a
//     contiguous burst;
//   * the link + partition kernels read sorted neighbours into (t, prev,
//     next) triples and move them back to time order (see below).
// Waits in the look-back are bounded: after the spin limit the kernel
// records an error in the workspace header instead of hanging.
//
// Inside the library the same kernels also serve a count the GPU wrote
// (n_dev: the chained prev/next sorts the accesses it left unresolved, a
// number it only knows on the device): grids are sized for the host bound n,
// workgroups past the device count return at once, and every launch can be
// gated on a device word, so no call ever waits for the GPU.
#include "pc_internal.h"

namespace pc {

constexpr int RADIX = 256;
constexpr int SORT_THREADS = 512;
constexpr int SORT_WAVES = SORT_THREADS / WAVE;
constexpr int SORT_ITEMS = 16;
constexpr int SORT_TILE = SORT_THREADS * SORT_ITEMS;   // 8192
constexpr int SORT_PASSES = 8;
constexpr uint64_t FLAG_AGG = 1ull << 32;
constexpr uint64_t FLAG_INC = 1ull << 33;
constexpr uint32_t SPIN_LIMIT = 1u << 22;

// Histograms of the four byte digits p0 .. p0+3 (one group of passes) in one
// read of the keys; the group over the high bytes runs only when asked.
constexpr int HIST_DIGITS = SORT_PASSES / 2;
__global__ __launch_bounds__(256) void sort_hist_kernel(const uint64_t *__restrict__ keys, uint64_t n, int p0,
                                                        uint32_t *__restrict__ hist,
                                                        const int32_t *__restrict__ only_if,
                                                        const uint32_t *__restrict__ n_dev,
                                                        const int32_t *__restrict__ gate) {
    if ((only_if && *only_if == 0) || gated_off(gate)) return;
    n = dev_count(n, n_dev);
    __shared__ uint32_t h[HIST_DIGITS][RADIX];
    for (int i = threadIdx.x; i < HIST_DIGITS * RADIX; i += blockDim.x) (&h[0][0])[i] = 0;
    __syncthreads();
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        const uint32_t k = (uint32_t)(keys[i] >> (8 * p0));
#pragma unroll
        for (int p = 0; p < HIST_DIGITS; ++p) atomicAdd(&h[p][(k >> (8 * p)) & 0xFF], 1u);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < HIST_DIGITS * RADIX; i += blockDim.x) {
        const uint32_t v = (&h[0][0])[i];
        if (v) atomicAdd(&hist[p0 * RADIX + i], v);
    }
}

// exclusive scan of each pass's 256-bin histogram -> digit bases; hist
// holds the group's rows (p0 .. p0+3) at rows 0..3; a row that does not sum
// to n (a histogram handed in by the caller) is reported
__global__ __launch_bounds__(RADIX) void sort_scan_kernel(const uint32_t *__restrict__ hist, int p0,
                                                          uint32_t *__restrict__ start, uint64_t n,
                                                          int32_t *__restrict__ err,
                                                          const int32_t *__restrict__ only_if,
                                                          const uint32_t *__restrict__ n_dev,
                                                          const int32_t *__restrict__ gate) {
    if ((only_if && *only_if == 0) || gated_off(gate)) return;
    n = dev_count(n, n_dev);
    __shared__ uint32_t tmp[RADIX / WAVE];
    for (int p = 0; p < HIST_DIGITS; ++p) {
        uint32_t total;
        const uint32_t e = block_excl_scan(hist[p * RADIX + threadIdx.x], tmp, &total);
        start[(p0 + p) * RADIX + threadIdx.x] = e;
        if (threadIdx.x == 0 && (uint64_t)total != n) atomicOr(err, DEV_ERR_BAD_HIST);
    }
}

// Large tiles make each digit's run in the output long (about 32 elements
// of 8192), so the scattered writes are mostly whole lines; the tile is
// staged twice through one buffer (keys, then values) and the per-wave digit
// counters are 16-bit (a tile holds at most 8192 elements), which keeps two
// workgroups on a CU
struct SortLds {
    uint64_t stage[SORT_TILE];
    uint16_t wcnt[SORT_WAVES][RADIX];
    uint32_t lstart[RADIX];
    uint32_t gbase[RADIX];
    uint32_t tmp[SORT_WAVES];
    uint32_t tile;
};

// One tile of a pass: the workgroup takes the next tile from the counter
// (tiles are handed out in order, so every tile a look-back waits on belongs
// to a workgroup already running it); false when none is left.
__device__ __forceinline__ bool sort_tile(SortLds &L, const uint64_t *__restrict__ keys_in,
                                          const uint32_t *__restrict__ vals_in, uint64_t *__restrict__ keys_out,
                                          uint32_t *__restrict__ vals_out, uint64_t n, int shift,
                                          const uint32_t *__restrict__ start, uint64_t *__restrict__ status,
                                          uint32_t *__restrict__ counter, uint32_t epoch, int32_t *__restrict__ err) {
    const int tid = threadIdx.x;
    const int lane = tid & (WAVE - 1);
    const int w = tid / WAVE;
    if (tid == 0) L.tile = atomicAdd(counter, 1u);
    for (int i = tid; i < SORT_WAVES * RADIX / 2; i += SORT_THREADS) reinterpret_cast<uint32_t *>(&L.wcnt[0][0])[i] = 0;
    __syncthreads();
    const uint32_t tile = L.tile;
    const uint64_t base = (uint64_t)tile * SORT_TILE;
    if (base >= n) return false;

    uint64_t k[SORT_ITEMS];
    uint32_t v[SORT_ITEMS];
    uint32_t pos[SORT_ITEMS];
    bool ok[SORT_ITEMS];
#pragma unroll
    for (int j = 0; j < SORT_ITEMS; ++j) {
        const uint64_t idx = base + (uint64_t)(w * SORT_ITEMS + j) * WAVE + lane;
        ok[j] = idx < n;
        k[j] = ok[j] ? keys_in[idx] : 0ull;
        v[j] = ok[j] ? (vals_in ? vals_in[idx] : (uint32_t)idx) : 0u;
    }
    // stable rank inside the wave: lanes with the same digit are matched by
    // eight ballots; a per-wave running count orders the wave's chunks
#pragma unroll
    for (int j = 0; j < SORT_ITEMS; ++j) {
        const uint32_t d = (uint32_t)(k[j] >> shift) & 0xFF;
        const uint64_t m = match_digit<8>(d, ballot(ok[j]));
        const uint32_t before = mbcnt(m);
        uint32_t cur = 0;
        if (ok[j]) cur = L.wcnt[w][d];
        pos[j] = cur + before;
        if (ok[j] && before == 0) L.wcnt[w][d] = (uint16_t)(cur + (uint32_t)__popcll(m));
    }
    __syncthreads();
    uint32_t cnt = 0;
    if (tid < RADIX) {
        for (int x = 0; x < SORT_WAVES; ++x) {
            const uint32_t c = L.wcnt[x][tid];
            L.wcnt[x][tid] = (uint16_t)cnt;
            cnt += c;
        }
    }
    uint32_t total;
    const uint32_t lst = block_excl_scan(tid < RADIX ? cnt : 0u, L.tmp, &total);
    if (tid < RADIX) L.lstart[tid] = lst;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < SORT_ITEMS; ++j) {
        if (ok[j]) {
            const uint32_t d = (uint32_t)(k[j] >> shift) & 0xFF;
            pos[j] += L.lstart[d] + L.wcnt[w][d];
            L.stage[pos[j]] = k[j];
        }
    }
    // decoupled look-back over the per-digit counts of earlier tiles
    if (tid < RADIX) {
        const uint64_t ep = (uint64_t)epoch << 34;
        uint64_t *mine = status + (uint64_t)tile * RADIX + tid;
        uint32_t excl = 0;
        if (tile == 0) {
            st_status64(mine, ep | FLAG_INC | cnt);
        } else {
            st_status64(mine, ep | FLAG_AGG | cnt);
            int64_t j = (int64_t)tile - 1;
            uint32_t spins = 0;
            while (j >= 0) {
                const uint64_t x = ld_status64(status + (uint64_t)j * RADIX + tid);
                if ((x >> 34) != epoch || (x & (FLAG_AGG | FLAG_INC)) == 0) {
                    if (++spins > SPIN_LIMIT) {
                        atomicOr(err, DEV_ERR_LOOKBACK_TIMEOUT);
                        break;
                    }
                    __builtin_amdgcn_s_sleep(1);
                    continue;
                }
                excl += (uint32_t)x;
                if (x & FLAG_INC) break;
                --j;
            }
            st_status64(mine, ep | FLAG_INC | (uint32_t)(excl + cnt));
        }
        L.gbase[tid] = start[tid] + excl - lst;
        // the last tile holds every digit's total: it must fill the digit's
        // range exactly (a caller's histogram that does not match the keys)
        if ((uint64_t)(tile + 1) * SORT_TILE >= n) {
            const uint32_t hi = tid + 1 < RADIX ? start[tid + 1] : (uint32_t)n;
            if (start[tid] + excl + cnt != hi) atomicOr(err, DEV_ERR_BAD_HIST);
        }
    }
    __syncthreads();
    const uint64_t left = n - base;
    const uint32_t n_tile = left < (uint64_t)SORT_TILE ? (uint32_t)left : (uint32_t)SORT_TILE;
    // keys out, remembering each slot's destination for the values (a
    // histogram that does not match the keys cannot send a write outside)
    uint32_t dst[SORT_ITEMS];
#pragma unroll
    for (int r = 0; r < SORT_ITEMS; ++r) {
        const uint32_t i = (uint32_t)(tid + r * SORT_THREADS);
        dst[r] = NONE;
        if (i < n_tile) {
            const uint64_t kk = L.stage[i];
            dst[r] = L.gbase[(uint32_t)(kk >> shift) & 0xFF] + i;
            if (dst[r] < n) keys_out[dst[r]] = kk;
        }
    }
    __syncthreads();
    uint32_t *s_val = reinterpret_cast<uint32_t *>(L.stage);
#pragma unroll
    for (int j = 0; j < SORT_ITEMS; ++j)
        if (ok[j]) s_val[pos[j]] = v[j];
    __syncthreads();
#pragma unroll
    for (int r = 0; r < SORT_ITEMS; ++r) {
        const uint32_t i = (uint32_t)(tid + r * SORT_THREADS);
        if (i < n_tile && dst[r] < n) vals_out[dst[r]] = s_val[i];
    }
    return true;
}

__global__ __launch_bounds__(SORT_THREADS, 4) void sort_pass_kernel(
    const uint64_t *__restrict__ keys_in, const uint32_t *__restrict__ vals_in,
    uint64_t *__restrict__ keys_out, uint32_t *__restrict__ vals_out, uint64_t n, int shift,
    const uint32_t *__restrict__ start, uint64_t *__restrict__ status, uint32_t *__restrict__ counter,
    uint32_t epoch, int32_t *__restrict__ err, const int32_t *__restrict__ only_if,
    const uint32_t *__restrict__ n_dev, const int32_t *__restrict__ gate) {
    // passes over the high key bits run only when the link step needs them
    if ((only_if && *only_if == 0) || gated_off(gate)) return;
    n = dev_count(n, n_dev);
    // Workgroups past the tile count take no tile (the counter then hands
    // out exactly the tiles there are) and leave at once: a grid sized for a
    // bound well above a device count costs little.
    if ((uint64_t)blockIdx.x * SORT_TILE >= n) return;
    __shared__ SortLds L;
    sort_tile(L, keys_in, vals_in, keys_out, vals_out, n, shift, start, status, counter, epoch, err);
}

// The same pass from a small persistent grid (each workgroup takes tiles
// until none are left), for launches that seldom do work: gated off, such a
// launch costs a few hundred workgroups instead of one per tile.  When it
// does run it is slower (11.0 against 7.5 ms for four passes over 2.1e9
// keys), since one tile per workgroup overlaps one tile's tail with the next
// one's loads.
__global__ __launch_bounds__(SORT_THREADS, 4) void sort_pass_persistent_kernel(
    const uint64_t *__restrict__ keys_in, const uint32_t *__restrict__ vals_in,
    uint64_t *__restrict__ keys_out, uint32_t *__restrict__ vals_out, uint64_t n, int shift,
    const uint32_t *__restrict__ start, uint64_t *__restrict__ status, uint32_t *__restrict__ counter,
    uint32_t epoch, int32_t *__restrict__ err, const int32_t *__restrict__ only_if,
    const uint32_t *__restrict__ n_dev, const int32_t *__restrict__ gate) {
    if ((only_if && *only_if == 0) || gated_off(gate)) return;
    n = dev_count(n, n_dev);
    __shared__ SortLds L;
    while (sort_tile(L, keys_in, vals_in, keys_out, vals_out, n, shift, start, status, counter, epoch, err))
        __syncthreads();   // the tile has left the LDS before the next one comes in
}

// ---- links, and the way back to time order -------------------------------
// Equal neighbours in (key, t) order are consecutive uses of one key, giving
// the triple (t, prev(t), next(t)).  t is a permutation of [0, n), so the
// triples with t in [a, b) fill exactly positions [a, b) once they are
// partitioned by the top bits of t; the order inside a range does not matter
// because the last step places every triple at its own t.  Each partition
// pass therefore reserves its output runs with global atomics on per-bucket
// cursors (per workgroup chunk in the link, per tile later; see below)
// instead of a look-back, stages each tile digit-sorted in LDS and writes
// each run contiguously.
constexpr int LINK_THREADS = 256;
constexpr int LINK_ITEMS = 8;                          // link: 2048-element tiles
constexpr int LINK_TILE = LINK_THREADS * LINK_ITEMS;
constexpr int PART_THREADS = 512;
constexpr int PART_ITEMS = 16;                         // plain partition: 8192-element tiles
constexpr int PERM_TILE = PART_THREADS * PART_ITEMS;   // the larger tile
constexpr int PERM_RADIX = 1024;   // digits of a later pass (a chunk spans two earlier buckets)
constexpr int LINK_RADIX = 256;    // digits of the first pass: at most 256 buckets
constexpr int PERM_LOCAL_BITS = 14;
constexpr uint64_t PERM_CHUNK_MAX = 1ull << 20;   // elements per workgroup, later passes
constexpr uint64_t LINK_CHUNK_MAX = 1ull << 16;   // elements per workgroup, link

// Work per workgroup: later passes take chunks of up to 2^20 elements (they
// reserve per tile, so the chunk only spreads the work).  The link reserves
// per chunk and its chunks are smaller: the runs that its workgroups in
// flight append to then lie closer together, and the link, which waits on
// more loads per element than the plain partition, gains from that.  About
// two chunks per CU; the same on the host (grids) and the device (a count
// the GPU wrote).
__host__ __device__ inline uint64_t chunk_elems(uint64_t n, int cus, uint64_t cap, uint64_t tile) {
    uint64_t c = (n + (uint64_t)cus * 2 - 1) / ((uint64_t)cus * 2);
    c = (c + tile - 1) / tile * tile;
    if (c > cap) c = cap;
    return c < tile ? tile : c;
}
// the most chunks any count up to n splits into (the grid of a pass)
static uint64_t max_chunks(uint64_t n, int cus, uint64_t cap, uint64_t tile) {
    const uint64_t by_cap = (n + cap - 1) / cap;
    const uint64_t by_cus = (uint64_t)cus * 2 + 1;
    const uint64_t at_n = (n + chunk_elems(n, cus, cap, tile) - 1) / chunk_elems(n, cus, cap, tile);
    uint64_t g = by_cap > by_cus ? by_cap : by_cus;
    if (at_n > g) g = at_n;
    return g ? g : 1;
}

// After the four passes over the low 32 key bits, equal keys are contiguous
// unless different keys share those bits ("mixed" runs, a few percent of the
// accesses for 64-bit hashes).  The link step resolves them by scanning the
// run: an element inside a block of equal keys finds its neighbour in one
// step, while a block boundary scans back (or forward) to the previous (next)
// block of its key or the run's end.  The scans of a workgroup share a budget
// of twice its element count; running out of it (adversarial keys: many keys
// sharing low bits) raises a flag that switches on the four passes over the
// high bits and a second link over the fully sorted keys, where equal keys
// are adjacent and no scan is needed.
__device__ __forceinline__ bool same_low(uint64_t a, uint64_t b) { return (uint32_t)a == (uint32_t)b; }

// Scan from position `from` (inclusive) in direction dir (-1 / +1) over
// elements sharing k's low bits; stop at k (found), at the run's end, or
// after `limit` steps.  Keys are read 8 at a time so a long scan costs one
// memory latency per 8 elements.  Returns false when the limit was reached
// first; *hit = position of k or UINT64_MAX.
constexpr int SCAN_BATCH = 8;
constexpr uint32_t LINK_SCAN_LIMIT = 64;   // memory steps a lane takes alone
__device__ __forceinline__ bool scan_run(const uint64_t *__restrict__ sk, uint64_t n, uint64_t k, uint64_t from,
                                         int dir, uint32_t limit, uint64_t *hit) {
    *hit = ~0ull;
    int64_t j = (int64_t)from;
    for (uint32_t steps = 0; steps < limit; steps += SCAN_BATCH) {
        uint64_t kb[SCAN_BATCH];
#pragma unroll
        for (int q = 0; q < SCAN_BATCH; ++q) {
            const int64_t x = j + dir * q;
            kb[q] = (x >= 0 && (uint64_t)x < n) ? sk[x] : ~k;   // ~k: differs from k in the low bits
        }
#pragma unroll
        for (int q = 0; q < SCAN_BATCH; ++q) {
            if (kb[q] == k) {
                *hit = (uint64_t)(j + dir * q);
                return true;
            }
            if (!same_low(kb[q], k)) return true;
        }
        j += dir * SCAN_BATCH;
    }
    return false;
}

// Previous (dir = -1) or next (dir = +1) element with the same full key as
// sorted position i, whose adjacent element shares the low key bits but not
// the key.  Lanes resolve such requests independently: each scans a few
// batches on its own; a lane still unresolved after that (a long run, e.g. a
// hot key sharing its low bits with another key) is taken over by the whole
// wave, 64 positions per step.  The wave steps are charged to the
// workgroup's budget (*budget, in positions); when it runs out the lane gives
// up and *overflow is raised, which switches on the passes over the high key
// bits and a second link.  All lanes of the wave must call this together.
__device__ __forceinline__ uint32_t resolve_mixed(const uint64_t *__restrict__ sk, const uint32_t *__restrict__ st,
                                                  uint64_t n, bool active, uint64_t i, int dir, int lane,
                                                  int32_t *budget, int32_t *__restrict__ overflow) {
    uint32_t res = NONE;
    uint64_t k = 0;
    int64_t cont = 0;
    bool need = false;
    if (active) {
        k = sk[i];
        const int64_t from = (int64_t)i + 2 * dir;   // i + dir is the known different key
        if (from >= 0 && (uint64_t)from < n) {
            uint64_t hit;
            if (scan_run(sk, n, k, (uint64_t)from, dir, LINK_SCAN_LIMIT, &hit)) {
                if (hit != ~0ull) res = st[hit];
            } else {
                need = true;
                cont = from + dir * (int64_t)LINK_SCAN_LIMIT;
            }
        }
    }
    for (uint64_t pending = ballot(need); pending; pending &= pending - 1) {
        const int L = __builtin_ctzll(pending);
        const uint64_t kL = shfl64(k, L);
        const int dL = __shfl(dir, L, WAVE);
        int64_t pos = (int64_t)shfl64((uint64_t)cont, L);
        uint32_t found = NONE;
        for (;;) {
            int32_t left = 0;
            if (lane == 0) left = atomicAdd(budget, -WAVE);
            left = __shfl(left, 0, WAVE);
            if (left < WAVE) {
                if (lane == 0) atomicOr(overflow, 1);
                break;
            }
            const int64_t x = pos + dL * lane;
            const uint64_t kk = (x >= 0 && (uint64_t)x < n) ? sk[x] : ~kL;
            const uint64_t hitm = ballot(kk == kL);
            const uint64_t ev = hitm | ballot(!same_low(kk, kL));
            if (ev) {
                const int f = __builtin_ctzll(ev);
                if ((hitm >> f) & 1) found = st[pos + dL * f];
                break;
            }
            pos += dL * WAVE;
        }
        if (lane == L) res = found;
    }
    return res;
}

// One workgroup owns a contiguous chunk of the input and streams it tile by
// tile: LDS counters give each element its slot inside its digit, the tile
// is staged digit-sorted in LDS (times, then (prev, next) pairs, through a
// single buffer), and each digit's part is appended to a run reserved in the
// bucket's output range.  The link reserves once per chunk: it first counts
// the chunk's digits and takes one run per digit with a single global atomic,
// so each bucket cursor sees one atomic per workgroup and the runs a
// workgroup appends to stay few and long.  Later passes skip that extra read
// of t and reserve per tile (their tiles are four times larger, so the runs
// stay long enough).  Longer tiles give longer runs per digit, hence fewer
// partially written lines; the link keeps 2048 because it holds keys and
// neighbours per element and waits on more loads: four small workgroups per
// CU overlap those waits better than two large.  A tile or chunk of a later
// pass spans at most 1024 consecutive buckets (see the plan), so digit =
// bucket mod 1024 names them without collision; the first pass has at most
// 256.
template <int TILE, int THREADS, int RADIX_N>
struct PermLds {
    uint64_t stage[TILE];   // bucket names while counting; per tile: times (as u32), then (prev, next) pairs
    uint32_t cnt[RADIX_N];
    uint32_t lstart[RADIX_N];
    uint32_t cur[RADIX_N];
    uint32_t tmp[THREADS / WAVE];
    int32_t budget;   // positions the link may still scan for long mixed runs
    uint32_t nmixed;  // mixed-run requests of the current tile (the list lives in `stage`)
};

template <bool FROM_SORT, int PERM_THREADS, int ITEMS, int RADIX_N, bool PER_TILE>
__device__ __forceinline__ void perm_partition_body(
    PermLds<PERM_THREADS * ITEMS, PERM_THREADS, RADIX_N> &L, const uint64_t *__restrict__ sk, const uint32_t *__restrict__ in_t,
    const uint64_t *__restrict__ in_pn, uint64_t n, int s, uint64_t per_wg, uint32_t *__restrict__ cursor,
    uint32_t *__restrict__ out_t, uint64_t *__restrict__ out_pn, bool full, int32_t *__restrict__ overflow) {
    uint32_t *s_stage = reinterpret_cast<uint32_t *>(L.stage), *s_cnt = L.cnt, *s_lstart = L.lstart,
             *s_cur = L.cur, *s_bucket = reinterpret_cast<uint32_t *>(L.stage), *s_tmp = L.tmp;
    static_assert(RADIX_N % PERM_THREADS == 0 || PERM_THREADS % RADIX_N == 0, "whole digits per thread");
    // per-tile bucket names live in the stage buffer, which the link's
    // mixed-run list also uses
    static_assert(!(PER_TILE && FROM_SORT), "the link reserves per chunk");
    // digits per thread; with fewer digits than threads, threads below
    // RADIX_N own one digit each
    constexpr int DPT = RADIX_N >= PERM_THREADS ? RADIX_N / PERM_THREADS : 1;
    const bool owner = (int)threadIdx.x * DPT < RADIX_N;
    // positions fit 32 bits (n < 2^32 - 1); offsets from a tile's base are
    // compared against what is left, so nothing wraps near the end
    if ((uint64_t)blockIdx.x * per_wg >= n) return;
    const int tid0 = threadIdx.x;   // the tile loop below takes its own copy
    const uint32_t lo = (uint32_t)((uint64_t)blockIdx.x * per_wg);
    const uint32_t hi = (uint64_t)lo + per_wg < n ? (uint32_t)(lo + per_wg) : (uint32_t)n;

    // ---- (per chunk) count the chunk's digits and reserve one run per digit
    for (int i = tid0; i < RADIX_N; i += PERM_THREADS) s_cnt[i] = 0;
    if (tid0 == 0) L.budget = (int32_t)(2 * (hi - lo) + 4096);
    __syncthreads();
    if constexpr (!PER_TILE) {
    // eight loads in flight per thread before their LDS updates
    for (uint32_t b0 = lo; b0 < hi; b0 += 8 * PERM_THREADS) {
        const uint32_t left = hi - b0;
        uint32_t tt[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const uint32_t o = (uint32_t)(q * PERM_THREADS + tid0);
            tt[q] = o < left ? (in_t + b0)[o] : 0u;
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            // (a time outside [0, n) can only come from inconsistent input;
            // it reserves nothing and its element is not written)
            if ((uint32_t)(q * PERM_THREADS + tid0) < left && tt[q] < n) {
                const uint32_t d = (tt[q] >> s) & (RADIX_N - 1);
                atomicAdd(&s_cnt[d], 1u);
                s_bucket[d] = tt[q] >> s;   // every writer of digit d writes the same bucket
            }
        }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < DPT && owner; ++q) {
        const int d = tid0 * DPT + q;
        const uint32_t c = s_cnt[d];
        if (c) s_cur[d] = atomicAdd(&cursor[s_bucket[d]], c);
    }
    __syncthreads();
    }

    // ---- stream the chunk tile by tile
    constexpr int TILE = PERM_THREADS * ITEMS;
    for (uint32_t base = lo; base < hi; base += TILE) {
        const uint32_t left = hi - base;
        // an opaque copy of the thread index: values derived from it are
        // recomputed per tile instead of being held (and spilled) across the loop
        int tid = threadIdx.x;
        __asm__ volatile("" : "+v"(tid));
        const int lane = tid & (WAVE - 1);
        for (int i = tid; i < RADIX_N; i += PERM_THREADS) s_cnt[i] = 0;
        if (tid == 0) L.nmixed = 0;
        __syncthreads();
        // per-tile base pointers keep the per-lane offsets 32-bit.  Every
        // load of the tile is issued before the first use, so a tile costs
        // one memory latency, not one per item.
        const uint32_t *tb = in_t + base;
        uint32_t t[ITEMS], pos[ITEMS];
        uint64_t pn[ITEMS];   // prev | next << 32
        bool ok[ITEMS];
        if (FROM_SORT) {
            const uint64_t *kb = sk + base;
            const int w = tid / WAVE;
            uint64_t k[ITEMS];
#pragma unroll
            for (int j = 0; j < ITEMS; ++j) {
                const uint32_t o = (uint32_t)(j * PERM_THREADS + tid);
                ok[j] = o < left;
                const uint32_t oc = ok[j] ? o : 0u;
                t[j] = tb[oc];
                k[j] = kb[oc];
            }
            // the elements just outside each item's wave: lane j loads the
            // one before item j's first lane, lane 8 + j the one after its
            // last valid lane
            uint64_t ek = 0;
            uint32_t et = 0;
            {
                const int j = lane & 7;
                const uint32_t w0 = (uint32_t)(j * PERM_THREADS + w * WAVE);   // wave's first offset
                const uint32_t lastj = w0 < left ? (left - 1 - w0 < (uint32_t)(WAVE - 1) ? left - 1 - w0 : WAVE - 1) : 0u;
                const uint64_t gp = lane < 8 ? (uint64_t)base + w0 - 1 : (uint64_t)base + w0 + lastj + 1;
                const bool want = lane < 16 && w0 < left && (lane < 8 ? (uint64_t)base + w0 > 0 : gp < n);
                if (want) {
                    ek = sk[gp];
                    et = in_t[gp];
                }
            }
            // fast links from neighbours; a lane whose neighbour shares the
            // low bits but not the key appends a request (offset, direction)
            // to the tile's list, resolved below by the whole workgroup
            uint32_t *mlist = reinterpret_cast<uint32_t *>(L.stage);   // 2 * TILE entries
            uint32_t mixbits = 0;   // bit 2j: item j's prev is in the list, bit 2j+1: its next
#pragma unroll
            for (int j = 0; j < ITEMS; ++j) {
                const uint32_t o = (uint32_t)(j * PERM_THREADS + tid);
                const uint64_t i = (uint64_t)base + o;
                // consecutive lanes hold consecutive sorted positions: the
                // neighbours' keys and times come from the adjacent lanes
                const uint32_t w0 = o - (uint32_t)lane;
                const int last = w0 < left ? (int)(left - 1 - w0 < (uint32_t)(WAVE - 1) ? left - 1 - w0 : WAVE - 1)
                                           : -1;
                uint64_t kp = from_lower64(k[j]), kn = from_upper64(k[j]);
                uint32_t tp = from_lower(t[j]);
                uint32_t tn = from_upper(t[j]);
                const uint64_t ekp = readlane64(ek, j), ekn = readlane64(ek, 8 + j);
                const uint32_t etp = (uint32_t)__builtin_amdgcn_readlane((int)et, j);
                const uint32_t etn = (uint32_t)__builtin_amdgcn_readlane((int)et, 8 + j);
                bool mp = false, mn = false;
                uint32_t pv = NONE, nx = NONE;
                if (ok[j]) {
                    const bool has_next = i + 1 < n;
                    if (lane == 0) { kp = ekp; tp = etp; }
                    if (lane == last) { kn = ekn; tn = etn; }
                    if (i > 0 && kp == k[j]) pv = tp;
                    else mp = i > 0 && !full && same_low(kp, k[j]);
                    if (has_next && kn == k[j]) nx = tn;
                    else mn = has_next && !full && same_low(kn, k[j]);
                }
                const uint64_t mpm = ballot(mp), mnm = ballot(mn);
                if (mpm | mnm) {
                    const uint32_t cnt = (uint32_t)__popcll(mpm) + (uint32_t)__popcll(mnm);
                    uint32_t e0 = 0;
                    if (lane == 0) e0 = atomicAdd(&L.nmixed, cnt);
                    e0 = (uint32_t)__shfl((int)e0, 0, WAVE);
                    if (mp) {
                        const uint32_t e = e0 + mbcnt(mpm);
                        mlist[e] = o << 1;
                        pv = e;
                        mixbits |= 1u << (2 * j);
                    }
                    if (mn) {
                        const uint32_t e = e0 + (uint32_t)__popcll(mpm) + mbcnt(mnm);
                        mlist[e] = (o << 1) | 1u;
                        nx = e;
                        mixbits |= 2u << (2 * j);
                    }
                }
                pn[j] = (uint64_t)pv | ((uint64_t)nx << 32);
            }
            __syncthreads();
            const uint32_t nm = L.nmixed;
            if (nm) {
                // resolve the list in place (entry -> time of the neighbour)
                for (uint32_t e0 = 0; e0 < nm; e0 += PERM_THREADS) {
                    const uint32_t e = e0 + tid;
                    const bool act = e < nm;
                    const uint32_t code = act ? mlist[e] : 0u;
                    const uint32_t res = resolve_mixed(sk, in_t, n, act, (uint64_t)base + (code >> 1),
                                                       (code & 1) ? 1 : -1, lane, &L.budget, overflow);
                    if (act) mlist[e] = res;
                }
                __syncthreads();
#pragma unroll
                for (int j = 0; j < ITEMS; ++j) {
                    if (mixbits & (3u << (2 * j))) {
                        uint32_t pv = (uint32_t)pn[j], nx = (uint32_t)(pn[j] >> 32);
                        if (mixbits & (1u << (2 * j))) pv = mlist[pv];
                        if (mixbits & (2u << (2 * j))) nx = mlist[nx];
                        pn[j] = (uint64_t)pv | ((uint64_t)nx << 32);
                    }
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < ITEMS; ++j) {
                const uint32_t o = (uint32_t)(j * PERM_THREADS + tid);
                ok[j] = o < left;
                const uint32_t oc = ok[j] ? o : 0u;
                t[j] = tb[oc];
                pn[j] = (in_pn + base)[oc];
            }
        }
#pragma unroll
        for (int j = 0; j < ITEMS; ++j) {
            // (per tile: a time outside [0, n), from inconsistent input,
            // reserves nothing and is not written)
            if (PER_TILE) ok[j] = ok[j] && t[j] < n;
            if (ok[j]) {
                pos[j] = atomicAdd(&s_cnt[(t[j] >> s) & (RADIX_N - 1)], 1u);
                if (PER_TILE) s_bucket[(t[j] >> s) & (RADIX_N - 1)] = t[j] >> s;
            }
        }
        __syncthreads();
        uint32_t c[DPT], mine = 0, total;
#pragma unroll
        for (int q = 0; q < DPT; ++q) {
            c[q] = owner ? s_cnt[tid * DPT + q] : 0u;
            mine += c[q];
        }
        uint32_t run = block_excl_scan(mine, s_tmp, &total);
#pragma unroll
        for (int q = 0; q < DPT && owner; ++q) {
            s_lstart[tid * DPT + q] = run;
            run += c[q];
            if (PER_TILE && c[q]) s_cur[tid * DPT + q] = atomicAdd(&cursor[s_bucket[tid * DPT + q]], c[q]);
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < ITEMS; ++j) {
            if (!ok[j]) continue;
            pos[j] += s_lstart[(t[j] >> s) & (RADIX_N - 1)];
            s_stage[pos[j]] = t[j];
        }
        __syncthreads();
        // times out, remembering each slot's destination for the (prev, next) pairs
        uint32_t dst[ITEMS];
#pragma unroll
        for (int r = 0; r < ITEMS; ++r) {
            const uint32_t slot = (uint32_t)(tid + r * PERM_THREADS);
            dst[r] = ~0u;
            if (slot < total) {
                const uint32_t tt = s_stage[slot];
                const uint32_t d = (tt >> s) & (RADIX_N - 1);
                dst[r] = s_cur[d] + (slot - s_lstart[d]);
                if (dst[r] < n) out_t[dst[r]] = tt;
            }
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < ITEMS; ++j)
            if (ok[j]) L.stage[pos[j]] = pn[j];
        __syncthreads();
#pragma unroll
        for (int r = 0; r < ITEMS; ++r)
            if (dst[r] < n) out_pn[dst[r]] = L.stage[tid + r * PERM_THREADS];
        if (!PER_TILE)
#pragma unroll
            for (int q = 0; q < DPT; ++q)
                if (owner) s_cur[tid * DPT + q] += c[q];
        __syncthreads();
    }
}

// The link variant holds more state per element (keys and neighbours): four
// 256-thread workgroups per CU; the plain partition runs two of 512.  The first link
// (over keys sorted by their low 32 bits) raises *flag when a mixed run is too
// long to scan; the second one runs only then (only_if = flag), over fully
// sorted keys.
__global__ __launch_bounds__(LINK_THREADS, 4) void link_partition_kernel(
    const uint64_t *__restrict__ sk, const uint32_t *__restrict__ in_t, uint64_t n, int s, int cus,
    uint32_t *__restrict__ cursor, uint32_t *__restrict__ out_t, uint64_t *__restrict__ out_pn,
    const int32_t *__restrict__ only_if, int32_t *__restrict__ flag, const uint32_t *__restrict__ n_dev,
    const int32_t *__restrict__ gate) {
    if ((only_if && *only_if == 0) || gated_off(gate)) return;
    n = dev_count(n, n_dev);
    const uint64_t per_wg = chunk_elems(n, cus, LINK_CHUNK_MAX, LINK_TILE);
    __shared__ PermLds<LINK_TILE, LINK_THREADS, LINK_RADIX> L;
    perm_partition_body<true, LINK_THREADS, LINK_ITEMS, LINK_RADIX, false>(L, sk, in_t, nullptr, n, s, per_wg, cursor, out_t, out_pn, only_if != nullptr,
                              flag);
}

__global__ __launch_bounds__(PART_THREADS, 4) void perm_partition_kernel(
    const uint32_t *__restrict__ in_t, const uint64_t *__restrict__ in_pn, uint64_t n, int s, int cus,
    uint32_t *__restrict__ cursor, uint32_t *__restrict__ out_t, uint64_t *__restrict__ out_pn,
    const uint32_t *__restrict__ n_dev, const int32_t *__restrict__ gate) {
    if (gated_off(gate)) return;
    n = dev_count(n, n_dev);
    const uint64_t per_wg = chunk_elems(n, cus, PERM_CHUNK_MAX, PERM_TILE);
    __shared__ PermLds<PERM_TILE, PART_THREADS, PERM_RADIX> L;
    perm_partition_body<false, PART_THREADS, PART_ITEMS, PERM_RADIX, true>(L, nullptr, in_t, in_pn, n, s, per_wg, cursor, out_t, out_pn, true, nullptr);
}

// cursor[b] = b << s: each bucket's output run starts at its first t
__global__ void perm_cursor_kernel(uint32_t *__restrict__ cursor, uint64_t nb, int s, const int32_t *__restrict__ gate) {
    if (gated_off(gate)) return;
    const uint64_t b = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b < nb) cursor[b] = (uint32_t)(b << s);
}

// every 16384-range of t holds exactly its own triples: place the (prev,
// next) pairs by t in LDS (128 KB, one 1024-thread workgroup per CU) and
// write prev / next in time order
constexpr int LOCAL_THREADS = 1024;
__global__ __launch_bounds__(LOCAL_THREADS) void perm_local_kernel(const uint32_t *__restrict__ in_t,
                                                                   const uint64_t *__restrict__ in_pn,
                                                                   uint64_t n, uint32_t *__restrict__ prev,
                                                                   uint32_t *__restrict__ next,
                                                                   const uint32_t *__restrict__ n_dev,
                                                                   const int32_t *__restrict__ gate) {
    constexpr uint32_t SPAN = 1u << PERM_LOCAL_BITS;
    constexpr int PER = SPAN / LOCAL_THREADS;
    __shared__ uint64_t s_pn[SPAN];
    if (gated_off(gate)) return;
    n = dev_count(n, n_dev);
    // one range per workgroup, or several from a capped grid
    for (uint64_t r0 = (uint64_t)blockIdx.x * SPAN; r0 < n; r0 += (uint64_t)gridDim.x * SPAN) {
        const uint32_t cnt = n - r0 < SPAN ? (uint32_t)(n - r0) : SPAN;
        const uint32_t *tb = in_t + r0;
        const uint64_t *pb = in_pn + r0;
        uint32_t tt[PER];
        uint64_t v[PER];
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const uint32_t j = threadIdx.x + q * LOCAL_THREADS;
            const uint32_t jc = j < cnt ? j : 0u;
            tt[q] = tb[jc];
            v[q] = pb[jc];
        }
#pragma unroll
        for (int q = 0; q < PER; ++q)
            if (threadIdx.x + q * LOCAL_THREADS < cnt) s_pn[(uint32_t)(tt[q] - r0) & (SPAN - 1)] = v[q];
        __syncthreads();
        for (uint32_t j = threadIdx.x; j < cnt; j += LOCAL_THREADS) {
            const uint64_t x = s_pn[j];
            prev[r0 + j] = (uint32_t)x;
            next[r0 + j] = (uint32_t)(x >> 32);
        }
        __syncthreads();   // the range has left the LDS before the next one comes in
    }
}

struct SortWs {
    int32_t *hdr;
    uint32_t *hist, *start, *counters;
    uint64_t *k1, *k2;   // sort ping-pong; afterwards (prev, next) pairs
    uint32_t *v1, *v2;   // sort ping-pong; afterwards times t
    uint64_t *status;
    uint32_t *cursor;
    size_t bytes;
};

// Partition plan for the way back to time order.  The last step uses
// 16384-ranges of t.  The link splits into at most 256 buckets, later passes
// into at most 512 per earlier bucket.  Every bucket is at least 16384 wide,
// so a tile of a later pass (8192 elements) spans at most two earlier
// buckets, i.e. at most 1024 consecutive buckets of its own pass, and
// (bucket mod 1024) names them without collision inside the tile.
struct PermPlan {
    int passes;
    int s[4];
    uint64_t buckets[4];
    uint64_t max_buckets;
};

static PermPlan plan_perm(uint64_t n) {
    PermPlan p{};
    int nbits = 0;
    while (nbits < 64 && (1ull << nbits) < n) ++nbits;
    int hi = nbits;   // bits above PERM_LOCAL_BITS still to split
    int cur = nbits;
    int shifts[4], k = 0;
    // 8 bits in the link (its tiles are small), up to 9 in later passes:
    // longer runs per tile and bucket than 10
    int width = 8;
    while (cur > PERM_LOCAL_BITS && k < 4) {
        int next_s = cur - width > PERM_LOCAL_BITS ? cur - width : PERM_LOCAL_BITS;
        shifts[k++] = next_s;
        cur = next_s;
        width = 9;
    }
    (void)hi;
    if (k == 0) shifts[k++] = PERM_LOCAL_BITS;
    p.passes = k;
    p.max_buckets = 1;
    for (int i = 0; i < k; ++i) {
        p.s[i] = shifts[i];
        p.buckets[i] = (n + (1ull << shifts[i]) - 1) >> shifts[i];
        if (p.buckets[i] > p.max_buckets) p.max_buckets = p.buckets[i];
    }
    return p;
}

static SortWs carve_sort(void *ws, uint64_t n) {
    Carver c{(char *)ws, 0};
    SortWs w;
    const uint64_t tiles = (n + SORT_TILE - 1) / SORT_TILE;
    w.hdr = c.take<int32_t>(WS_HEADER / sizeof(int32_t));
    w.hist = c.take<uint32_t>(SORT_PASSES * RADIX);
    w.start = c.take<uint32_t>(SORT_PASSES * RADIX);
    w.counters = c.take<uint32_t>(SORT_PASSES);
    w.k1 = c.take<uint64_t>(n);
    w.k2 = c.take<uint64_t>(n);
    w.v1 = c.take<uint32_t>(n);
    w.v2 = c.take<uint32_t>(n);
    w.status = c.take<uint64_t>(tiles * RADIX);
    w.cursor = c.take<uint32_t>(plan_perm(n).max_buckets + 1);
    w.bytes = c.off;
    return w;
}


pc_status prev_next_core(const uint64_t *keys, uint64_t n, const uint32_t *n_dev, uint32_t *prev, uint32_t *next,
                         const uint32_t *key_hist, void *ws, hipStream_t s, const int32_t *gate, bool rare) {
    SortWs w = carve_sort(ws, n);
    pc_status st = fill_u32_gated(reinterpret_cast<uint32_t *>(w.hdr), 0u, 1, s, gate);
    if (st != PC_OK || n == 0) return st;

    const uint64_t tiles = (n + SORT_TILE - 1) / SORT_TILE;
    if ((st = fill_u32_gated(w.hist, 0u, SORT_PASSES * RADIX, s, gate)) != PC_OK) return st;
    if ((st = fill_u32_gated(w.counters, 0u, SORT_PASSES, s, gate)) != PC_OK) return st;
    if ((st = fill_u32_gated(reinterpret_cast<uint32_t *>(w.status), 0u, tiles * RADIX * 2, s, gate)) != PC_OK)
        return st;

    const int cus = device_cus();
    uint64_t hg = (n + 4095) / 4096;
    if (hg > (uint64_t)cus * 4) hg = (uint64_t)cus * 4;
    // flag (header word 1): the first link met a mixed run too long to scan,
    // so the high-byte passes and a second link run
    int32_t *need_high = w.hdr + 1;
    if ((st = fill_u32_gated(reinterpret_cast<uint32_t *>(need_high), 0u, 1, s, gate)) != PC_OK) return st;
    // the low bytes' histograms: handed in by the hash, or counted here
    if (!key_hist)
        PC_LAUNCH(K_SORT_HIST, sort_hist_kernel, dim3((unsigned)hg), dim3(256), 0, s, keys, n, 0, w.hist,
                  (const int32_t *)nullptr, n_dev, gate);
    PC_LAUNCH(K_SORT_SCAN, sort_scan_kernel, dim3(1), dim3(RADIX), 0, s, key_hist ? key_hist : w.hist, 0, w.start, n,
              w.hdr, (const int32_t *)nullptr, n_dev, gate);

    // Links + partition back to time order.  The sort leaves (key, t) in
    // (k2, v2) after four passes and again after eight; the triples ping-pong
    // between the first sort buffers ((prev, next) pairs in k1, t in v1) and,
    // once the sorted keys have been consumed, the second ones (k2, v2).
    // The plan is made for the bound n: with fewer elements its later
    // buckets stay empty.
    const PermPlan pp = plan_perm(n);
    if (pp.buckets[0] > (uint64_t)LINK_RADIX) return PC_ERR_TOO_LARGE;   // the plan never splits wider
    uint32_t *bt[2] = {w.v1, w.v2};
    uint64_t *bpn[2] = {w.k1, w.k2};
    const unsigned ptiles = (unsigned)max_chunks(n, cus, PERM_CHUNK_MAX, PERM_TILE);
    const unsigned ltiles = (unsigned)max_chunks(n, cus, LINK_CHUNK_MAX, LINK_TILE);
    const unsigned cg0 = (unsigned)((pp.buckets[0] + 255) / 256);

    const uint64_t *kin = keys;
    const uint32_t *vin = nullptr;
    for (int p = 0; p < SORT_PASSES; ++p) {
        if (p == SORT_PASSES / 2) {
            // first link, over keys sorted by their low 32 bits
            PC_LAUNCH(K_FILL32, perm_cursor_kernel, dim3(cg0), dim3(256), 0, s, w.cursor, pp.buckets[0], pp.s[0],
                      gate);
            PC_LAUNCH(K_LINK, link_partition_kernel, dim3(ltiles), dim3(LINK_THREADS), 0, s, kin, vin, n, pp.s[0],
                      cus, w.cursor, bt[0], bpn[0], (const int32_t *)nullptr, need_high, n_dev, gate);
            PC_LAUNCH(K_SORT_HIST, sort_hist_kernel, dim3((unsigned)hg), dim3(256), 0, s, keys, n, SORT_PASSES / 2,
                      w.hist, (const int32_t *)need_high, n_dev, gate);
            PC_LAUNCH(K_SORT_SCAN, sort_scan_kernel, dim3(1), dim3(RADIX), 0, s, w.hist + SORT_PASSES / 2 * RADIX,
                      SORT_PASSES / 2, w.start, n, w.hdr, (const int32_t *)need_high, n_dev, gate);
        }
        uint64_t *kout = (p & 1) ? w.k2 : w.k1;
        uint32_t *vout = (p & 1) ? w.v2 : w.v1;
        // the passes over the high bits, and every pass of a call that
        // seldom runs, take the persistent grid
        const int32_t *high = p >= SORT_PASSES / 2 ? (const int32_t *)need_high : nullptr;
        if (high || rare)
            PC_LAUNCH(K_SORT_PASS, sort_pass_persistent_kernel, dim3(capped(tiles, 2)), dim3(SORT_THREADS), 0, s,
                      kin, vin, kout, vout, n, 8 * p, w.start + p * RADIX, w.status, w.counters + p,
                      (uint32_t)(p + 1), w.hdr, high, n_dev, gate);
        else
            PC_LAUNCH(K_SORT_PASS, sort_pass_kernel, dim3((unsigned)tiles), dim3(SORT_THREADS), 0, s, kin, vin,
                      kout, vout, n, 8 * p, w.start + p * RADIX, w.status, w.counters + p, (uint32_t)(p + 1),
                      w.hdr, high, n_dev, gate);
        kin = kout;
        vin = vout;
    }
    // second link, over fully sorted keys, only if the first one gave up
    PC_LAUNCH(K_FILL32, perm_cursor_kernel, dim3(cg0), dim3(256), 0, s, w.cursor, pp.buckets[0], pp.s[0], gate);
    PC_LAUNCH(K_LINK, link_partition_kernel, dim3(ltiles), dim3(LINK_THREADS), 0, s, kin, vin, n, pp.s[0], cus,
              w.cursor, bt[0], bpn[0], (const int32_t *)need_high, (int32_t *)nullptr, n_dev, gate);
    int cur = 0;
    for (int i = 1; i < pp.passes; ++i) {
        const unsigned cg = (unsigned)((pp.buckets[i] + 255) / 256);
        PC_LAUNCH(K_FILL32, perm_cursor_kernel, dim3(cg), dim3(256), 0, s, w.cursor, pp.buckets[i], pp.s[i], gate);
        const int nxt = cur ^ 1;
        PC_LAUNCH(K_PERM, perm_partition_kernel, dim3(ptiles), dim3(PART_THREADS), 0, s, bt[cur], bpn[cur], n,
                  pp.s[i], cus, w.cursor, bt[nxt], bpn[nxt], n_dev, gate);
        cur = nxt;
    }
    const uint64_t span = 1ull << PERM_LOCAL_BITS;
    const uint64_t ranges = (n + span - 1) / span;
    PC_LAUNCH(K_PERM_LOCAL, perm_local_kernel, dim3(rare ? capped(ranges, 1) : (unsigned)ranges), dim3(LOCAL_THREADS),
              0, s, bt[cur], bpn[cur], n, prev, next, n_dev, gate);
    return PC_OK;
}

}  // namespace pc

extern "C" {

size_t pc_prev_next_use_ws(uint64_t n) { return pc::carve_sort(nullptr, n).bytes; }

pc_status pc_prev_next_use(const uint64_t *keys, uint64_t n, uint32_t *prev, uint32_t *next,
                           const uint32_t *key_hist, void *ws, size_t ws_bytes, void *stream) {
    if (n >= (uint64_t)PC_NONE) return PC_ERR_TOO_LARGE;
    if (n > 0 && (!keys || !prev || !next)) return PC_ERR_INVALID;
    if (!ws) return PC_ERR_WORKSPACE;
    if (ws_bytes < pc_prev_next_use_ws(n)) return PC_ERR_WORKSPACE;
    return pc::prev_next_core(keys, n, nullptr, prev, next, key_hist, ws, (hipStream_t)stream, nullptr, false);
}

}  // extern "C"
