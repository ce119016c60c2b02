// Exact LRU stack distance (pc_stack_distance).
//
// Definition: D(t) = #{ i in (prev(t), t) : next(i) > t }, the number of
// distinct blocks touched since the previous use; an LRU cache of c blocks
// hits exactly when D < c (LRU is a stack algorithm; Sec. 5 "LRU as a
// bedrock", Appendix B "stack distance between reuses").
//
// Reformulation used here.  With v(j) = prev(j) + 1 (0 for a cold access),
// the number of j < t with v(j) < v(t) is prev(t) + 1 + D(t): every i <=
// prev(t) qualifies, and in the window (prev(t), t) exactly the first use of
// each distinct block does.  Non-cold v are distinct, so with Z(t) = number of
// cold accesses before t and C'(t) = #{ non-cold j < t : v(j) < v(t) }:
//        D(t) = Z(t) + C'(t) - v(t).
// C' is a two-dimensional dominance count.  The non-cold accesses are taken in
// v order -- that is just next[] read in index order, since next[p] = t
// exactly when v(t) = p + 1 -- and partitioned by the bits of t from the top
// (MSD radix).  At every level an element adds the number of elements that
// precede it in v order, sit in the same bucket (same higher bits of t) and
// carry a smaller digit.  Summed over all levels this is exactly C'(t), and
// the last level leaves every element at its own t.
//
// Buckets are ranges of t, so their sizes are known in advance from the
// per-4096 prefix of cold counts: #non-cold t < X = X - Z(X).
//   * sd_cold_count + a three-step scan -> Z at every multiple of 4096
//   * per level (1-3 levels of 8-bit digits above bit 12), over tiles of 1024
//     elements: sd_count (per-tile digit counts), a segmented scan of those
//     counts over the tiles of each bucket (sd_seg: reduce, carry, scan --
//     no waiting on other workgroups), then sd_dominance_pass: one ballot
//     per digit bit gives every lane the earlier lanes of its 64-lane chunk
//     with a smaller / equal digit, a 2-D prefix over
//     (chunk, digit) in LDS extends that to the tile, the scanned counts
//     extend it across tiles, and the tile is written out digit-partitioned
//     through LDS.
//   * sd_local_finish -> one workgroup per 4096-range of t: two in-LDS levels
//     of 6 bits finish the count, then D is written in t order with the cold
//     prefix from a block scan.
#include "pc_internal.h"

namespace pc {

constexpr int LOCAL_BITS = 12;
constexpr uint32_t LOCAL_SPAN = 1u << LOCAL_BITS;   // 4096
constexpr int DOM_THREADS = 512;
constexpr int DOM_WAVES = DOM_THREADS / WAVE;
constexpr int DOM_CHUNKS_PER_WAVE = 4;
constexpr int DOM_CHUNKS = DOM_WAVES * DOM_CHUNKS_PER_WAVE;   // 32
constexpr int DOM_TILE = DOM_CHUNKS * WAVE;                    // 2048
constexpr int DOM_RADIX = 256;
static_assert(DOM_THREADS == 2 * DOM_RADIX, "the column prefix splits the chunks in two halves");
constexpr int LOC_THREADS = 512;
constexpr int LOC_WAVES = LOC_THREADS / WAVE;
constexpr int LOC_CHUNKS = LOCAL_SPAN / WAVE;                  // 64
constexpr int LOC_CPW = LOC_CHUNKS / LOC_WAVES;                // 8
constexpr int LOC_PARTS = LOC_THREADS / 64;                    // column-prefix parts per digit
constexpr int SCAN_THREADS = 1024;

// number of non-cold accesses t < X (X a multiple of 4096, or X = n)
__device__ __forceinline__ uint64_t cnt_lt(uint64_t X, const uint32_t *__restrict__ Zc) {
    return X - Zc[(X + LOCAL_SPAN - 1) >> LOCAL_BITS];
}

__global__ __launch_bounds__(256) void sd_cold_count_kernel(const uint32_t *__restrict__ prev,
                                                            uint64_t n, uint32_t *__restrict__ cnt,
                                                            const int32_t *gate) {
    if (gated_off(gate)) return;
    __shared__ uint32_t tmp[4];
    constexpr int PER = LOCAL_SPAN / 256;   // 16 consecutive values per thread
    const uint64_t nchunks = (n + LOCAL_SPAN - 1) / LOCAL_SPAN;
    for (uint64_t chunk = blockIdx.x; chunk < nchunks; chunk += gridDim.x) {
    const uint64_t base = chunk * LOCAL_SPAN + (uint64_t)threadIdx.x * PER;
    uint32_t c = 0;
    if (base + PER <= n && (reinterpret_cast<uintptr_t>(prev) & 15) == 0) {
        const uint4 *p = reinterpret_cast<const uint4 *>(prev + base);   // four 16-byte loads in flight
        uint4 v[PER / 4];
#pragma unroll
        for (int q = 0; q < PER / 4; ++q) v[q] = p[q];
#pragma unroll
        for (int q = 0; q < PER / 4; ++q)
            c += (v[q].x == NONE) + (v[q].y == NONE) + (v[q].z == NONE) + (v[q].w == NONE);
    } else {
        for (int j = 0; j < PER; ++j) c += (base + j < n && prev[base + j] == NONE) ? 1u : 0u;
    }
    uint32_t total;
    block_excl_scan(c, tmp, &total);
    if (threadIdx.x == 0) cnt[chunk] = total;
    }
}

// exclusive scan of m values (one workgroup); out[m] = total
__global__ __launch_bounds__(SCAN_THREADS) void sd_scan_kernel(const uint32_t *__restrict__ in,
                                                               uint64_t m,
                                                               uint32_t *__restrict__ out,
                                                               const int32_t *gate) {
    if (gated_off(gate)) return;
    __shared__ uint32_t tmp[SCAN_THREADS / WAVE];
    const uint64_t seg = (m + SCAN_THREADS - 1) / SCAN_THREADS;
    const uint64_t lo = threadIdx.x * seg;
    const uint64_t hi = lo + seg < m ? lo + seg : m;
    uint32_t s = 0;
    for (uint64_t i = lo; i < hi; ++i) s += in[i];
    uint32_t total;
    uint32_t run = block_excl_scan(s, tmp, &total);
    for (uint64_t i = lo; i < hi; ++i) {
        const uint32_t x = in[i];
        out[i] = run;
        run += x;
    }
    if (threadIdx.x == 0) out[m] = total;
}

// Exclusive scan of m values over many workgroups (the per-4096 cold counts
// number n / 4096): block sums, one workgroup scans the sums, every block
// scans itself on top of its offset.  out[m] = total.
constexpr int SCAN_BLOCK = SCAN_THREADS * 4;
__global__ __launch_bounds__(SCAN_THREADS) void sd_scan_reduce_kernel(const uint32_t *__restrict__ in, uint64_t m,
                                                                      uint32_t *__restrict__ part,
                                                                      const int32_t *gate) {
    if (gated_off(gate)) return;
    __shared__ uint32_t tmp[SCAN_THREADS / WAVE];
    const uint64_t i0 = (uint64_t)blockIdx.x * SCAN_BLOCK + (uint64_t)threadIdx.x * 4;
    uint32_t x = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) x += i0 + q < m ? in[i0 + q] : 0u;
    uint32_t total;
    block_excl_scan(x, tmp, &total);
    if (threadIdx.x == 0) part[blockIdx.x] = total;
}

__global__ __launch_bounds__(SCAN_THREADS) void sd_scan_apply_kernel(const uint32_t *__restrict__ in, uint64_t m,
                                                                     const uint32_t *__restrict__ part_ex,
                                                                     uint64_t nblocks, uint32_t *__restrict__ out,
                                                                     const int32_t *gate) {
    if (gated_off(gate)) return;
    __shared__ uint32_t tmp[SCAN_THREADS / WAVE];
    const uint64_t i0 = (uint64_t)blockIdx.x * SCAN_BLOCK + (uint64_t)threadIdx.x * 4;
    uint32_t v[4], x = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        v[q] = i0 + q < m ? in[i0 + q] : 0u;
        x += v[q];
    }
    uint32_t total;
    uint32_t run = part_ex[blockIdx.x] + block_excl_scan(x, tmp, &total);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        if (i0 + q < m) out[i0 + q] = run;
        run += v[q];
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) out[m] = part_ex[nblocks];
}

// tiles per bucket of a dominance pass (bucket = t >> S)
__global__ void sd_tile_count_kernel(const uint32_t *__restrict__ Zc, uint64_t n, int S,
                                     uint64_t nbuckets, uint32_t *__restrict__ tcount, const int32_t *gate) {
    if (gated_off(gate)) return;
    const uint64_t b = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= nbuckets) return;
    uint64_t lo = b << S, hi = (b + 1) << S;
    lo = lo < n ? lo : n;
    hi = hi < n ? hi : n;
    const uint64_t size = cnt_lt(hi, Zc) - cnt_lt(lo, Zc);
    tcount[b] = (uint32_t)((size + DOM_TILE - 1) / DOM_TILE);
}

// ---- one MSD level of the dominance count (8-bit digits of t) -----------
// Tiles: FIRST reads next[] in index order (= v order) in fixed index ranges,
// one bucket; later levels read the previous level's output with tiles that
// never straddle a bucket (bucket = t >> (s + k)), located through tfirst.
struct TileLoc {
    uint64_t bucket, e0, e1, first_tile;
    bool valid;
};

// tile -> bucket of a level (largest b with tfirst[b] <= tile), computed
// once per level so the level's kernels need one load instead of a search
__global__ void sd_tile_bucket_kernel(const uint32_t *__restrict__ tfirst, uint64_t nbuckets, uint64_t max_tiles,
                                      uint32_t *__restrict__ tile_bucket, const int32_t *gate) {
    if (gated_off(gate)) return;
    const uint64_t tile = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (tile >= max_tiles || tile >= tfirst[nbuckets]) return;
    uint64_t lo = 0, hi = nbuckets;
    while (hi - lo > 1) {
        const uint64_t mid = (lo + hi) >> 1;
        if (tfirst[mid] <= tile) lo = mid; else hi = mid;
    }
    tile_bucket[tile] = (uint32_t)lo;
}

template <bool FIRST>
__device__ __forceinline__ TileLoc locate_tile(uint64_t tile, uint64_t n, const uint32_t *__restrict__ Zc,
                                               int S, const uint32_t *__restrict__ tfirst, uint64_t nbuckets,
                                               const uint32_t *__restrict__ tile_bucket) {
    TileLoc L{0, 0, 0, 0, true};
    if (FIRST) {
        const uint64_t tiles = (n + DOM_TILE - 1) / DOM_TILE;
        if (tile >= tiles) { L.valid = false; return L; }
        L.e0 = tile * DOM_TILE;
        L.e1 = L.e0 + DOM_TILE < n ? L.e0 + DOM_TILE : n;
        return L;
    }
    if (tile >= tfirst[nbuckets]) { L.valid = false; return L; }
    const uint64_t lo = tile_bucket[tile];
    L.bucket = lo;
    L.first_tile = tfirst[lo];
    uint64_t blo = lo << S, bhi = (lo + 1) << S;
    blo = blo < n ? blo : n;
    bhi = bhi < n ? bhi : n;
    const uint64_t bs = cnt_lt(blo, Zc), be = cnt_lt(bhi, Zc);
    L.e0 = bs + (tile - L.first_tile) * DOM_TILE;
    L.e1 = L.e0 + DOM_TILE < be ? L.e0 + DOM_TILE : be;
    return L;
}

template <bool FIRST>
__device__ __forceinline__ void load_tile(const TileLoc &L, const uint32_t *__restrict__ in_t,
                                          const uint32_t *__restrict__ in_acc, int w, int lane,
                                          uint32_t (&t)[DOM_CHUNKS_PER_WAVE], uint32_t (&acc)[DOM_CHUNKS_PER_WAVE],
                                          bool (&ok)[DOM_CHUNKS_PER_WAVE], bool want_acc) {
#pragma unroll
    for (int i = 0; i < DOM_CHUNKS_PER_WAVE; ++i) {
        const uint64_t e = L.e0 + (uint64_t)(w * DOM_CHUNKS_PER_WAVE + i) * WAVE + lane;
        if (FIRST) {
            const uint32_t x = e < L.e1 ? in_t[e] : NONE;
            ok[i] = x != NONE;
            t[i] = x;
            acc[i] = 0;
        } else {
            ok[i] = e < L.e1;
            t[i] = ok[i] ? in_t[e] : 0u;
            acc[i] = (ok[i] && want_acc) ? in_acc[e] : 0u;
        }
    }
}

// Per-tile digit counts (and whether the tile starts a bucket), the input of
// the segmented scan over tiles.  Only counts are needed here, so instead of
// ranking lanes each run of equal digits in a 64-lane chunk (runs are long at
// the top levels, where t grows with v) adds its length with one LDS atomic.
// A workgroup takes COUNT_TPW consecutive tiles and issues every lookup and
// load of all of them before counting: one tile's work is too short to
// cover the chain of dependent loads (tile -> bucket -> range -> elements).
constexpr int COUNT_TPW = 4;
template <bool FIRST>
__global__ __launch_bounds__(DOM_THREADS) void sd_count_kernel(
    const uint32_t *__restrict__ in_t, uint64_t n, const uint32_t *__restrict__ Zc, int s, int k,
    const uint32_t *__restrict__ tfirst, uint64_t nbuckets, const uint32_t *__restrict__ tile_bucket,
    uint16_t *__restrict__ cnt, uint8_t *__restrict__ seg, uint64_t groups, const int32_t *gate) {
    if (gated_off(gate)) return;
    __shared__ uint32_t s_cnt[COUNT_TPW][DOM_RADIX];
    const int tid = threadIdx.x, lane = tid & (WAVE - 1), w = tid / WAVE;
    for (uint64_t grp = blockIdx.x; grp < groups; grp += gridDim.x) {
    __syncthreads();   // the previous group's counts are written out
    const uint64_t tile0 = grp * COUNT_TPW;
    // an invalid tile (past the level's last) has an empty range: it loads
    // nothing, and every later tile is invalid too
    TileLoc L[COUNT_TPW];
#pragma unroll
    for (int q = 0; q < COUNT_TPW; ++q)
        L[q] = locate_tile<FIRST>(tile0 + q, n, Zc, s + k, tfirst, nbuckets, tile_bucket);
    if (!L[0].valid) break;   // every later group is past the level's last tile too
    for (int i = tid; i < COUNT_TPW * DOM_RADIX; i += DOM_THREADS) (&s_cnt[0][0])[i] = 0;
    uint32_t t[COUNT_TPW][DOM_CHUNKS_PER_WAVE], acc[DOM_CHUNKS_PER_WAVE];
    bool ok[COUNT_TPW][DOM_CHUNKS_PER_WAVE];
#pragma unroll
    for (int q = 0; q < COUNT_TPW; ++q) load_tile<FIRST>(L[q], in_t, nullptr, w, lane, t[q], acc, ok[q], false);
    __syncthreads();
    const uint32_t dmask = (1u << k) - 1u;
#pragma unroll
    for (int q = 0; q < COUNT_TPW; ++q) {
#pragma unroll
        for (int i = 0; i < DOM_CHUNKS_PER_WAVE; ++i) {
            // invalid lanes take digit RADIX (never counted) so they end runs
            const uint32_t d = ok[q][i] ? (t[q][i] >> s) & dmask : (uint32_t)DOM_RADIX;
            const uint32_t dl = from_lower(d);   // lane 0 keeps its own and is a head anyway
            const bool head = lane == 0 || dl != d;
            const uint64_t heads = ballot(head);
            // next head above this lane (or 64): the run is [lane, next)
            const uint64_t above = lane == WAVE - 1 ? 0ull : heads & (~0ull << (lane + 1));
            const uint32_t next = above ? (uint32_t)__builtin_ctzll(above) : (uint32_t)WAVE;
            if (head && d < (uint32_t)DOM_RADIX) atomicAdd(&s_cnt[q][d], next - (uint32_t)lane);
        }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < COUNT_TPW; ++q) {
        if (!L[q].valid) break;
        const uint64_t tile = tile0 + q;
        if (tid < DOM_RADIX) cnt[tile * DOM_RADIX + tid] = (uint16_t)s_cnt[q][tid];
        if (tid == 0) seg[tile] = FIRST ? (tile == 0) : (tile == L[q].first_tile);
    }
    }
}

// Segmented exclusive scan over tiles, per digit (a bucket's first tile
// restarts the sum), in three steps over groups of SEG_GROUP tiles.
constexpr int SEG_GROUP = 256;
constexpr int SEG_BATCH = 16;

__device__ __forceinline__ uint64_t total_tiles(const uint32_t *tfirst_end, uint64_t fixed) {
    return tfirst_end ? (uint64_t)*tfirst_end : fixed;
}

// A: per group, the sum after its last bucket start, and whether it has one
__global__ __launch_bounds__(DOM_RADIX) void sd_seg_reduce_kernel(const uint16_t *__restrict__ cnt,
                                                                  const uint8_t *__restrict__ seg,
                                                                  const uint32_t *tfirst_end, uint64_t fixed,
                                                                  uint32_t *__restrict__ gsum,
                                                                  uint8_t *__restrict__ ghas, const int32_t *gate) {
    if (gated_off(gate)) return;
    const uint64_t rows = total_tiles(tfirst_end, fixed);
    const uint64_t r0 = (uint64_t)blockIdx.x * SEG_GROUP;
    if (r0 >= rows) return;
    const uint64_t r1 = r0 + SEG_GROUP < rows ? r0 + SEG_GROUP : rows;
    const int d = threadIdx.x;
    uint32_t tail = 0;
    bool has = false;
    for (uint64_t r = r0; r < r1; r += SEG_BATCH) {
        uint32_t c[SEG_BATCH];
        bool f[SEG_BATCH];
#pragma unroll
        for (int q = 0; q < SEG_BATCH; ++q) {
            const bool in = r + q < r1;
            c[q] = in ? cnt[(r + q) * DOM_RADIX + d] : 0u;
            f[q] = in && seg[r + q];
        }
#pragma unroll
        for (int q = 0; q < SEG_BATCH; ++q) {
            if (f[q]) { tail = 0; has = true; }
            tail += c[q];
        }
    }
    gsum[blockIdx.x * DOM_RADIX + d] = tail;
    if (d == 0) ghas[blockIdx.x] = has;
}

// B: carry into every group: per digit (one workgroup each), a segmented
// scan over the groups where a group holding a bucket start restarts the
// sum.  Inside a wave: the plain prefix sum minus the sum before the last
// start at or below the lane (found with a ballot); across the waves of a
// 1024-group chunk and across chunks: a short serial carry.
constexpr int CARRY_THREADS = 1024;
__global__ __launch_bounds__(CARRY_THREADS) void sd_seg_carry_kernel(const uint32_t *__restrict__ gsum,
                                                                     const uint8_t *__restrict__ ghas,
                                                                     const uint32_t *tfirst_end, uint64_t fixed,
                                                                     uint32_t *__restrict__ gin, const int32_t *gate) {
    if (gated_off(gate)) return;
    __shared__ uint32_t s_val[CARRY_THREADS / WAVE];
    __shared__ uint32_t s_has[CARRY_THREADS / WAVE];
    const uint64_t rows = total_tiles(tfirst_end, fixed);
    const uint64_t groups = (rows + SEG_GROUP - 1) / SEG_GROUP;
    const int d = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & (WAVE - 1), w = tid / WAVE;
    uint32_t carry = 0;   // carry into the current chunk
    for (uint64_t g0 = 0; g0 < groups; g0 += CARRY_THREADS) {
        const uint64_t g = g0 + tid;
        const bool in = g < groups;
        const bool f = in && ghas[g];
        const uint32_t v = in ? gsum[g * DOM_RADIX + d] : 0u;
        const uint32_t S = wave_incl_scan(v);
        const uint64_t fm = ballot(f);
        const uint64_t le = fm & (lane == WAVE - 1 ? ~0ull : ((2ull << lane) - 1));   // starts at or below me
        const int last = le ? 63 - __builtin_clzll(le) : -1;
        const uint32_t before = (uint32_t)__shfl((int)S, last > 0 ? last - 1 : 0, WAVE);
        const uint32_t seg = last > 0 ? S - before : S;   // sum since the last start (or since lane 0)
        if (lane == WAVE - 1) {
            s_val[w] = seg;
            s_has[w] = fm != 0;
        }
        __syncthreads();
        uint32_t cin = carry;   // carry into this wave
        for (int x = 0; x < w; ++x) cin = s_has[x] ? s_val[x] : cin + s_val[x];
        uint32_t chunk_out = cin;
        for (int x = w; x < CARRY_THREADS / WAVE; ++x) chunk_out = s_has[x] ? s_val[x] : chunk_out + s_val[x];
        const uint32_t incl = last >= 0 ? seg : cin + seg;   // carry after group g
        const uint32_t prev = (uint32_t)__shfl_up((int)incl, 1, WAVE);
        if (in) gin[g * DOM_RADIX + d] = lane == 0 ? cin : prev;
        carry = chunk_out;
        __syncthreads();
    }
}

// C: per group, the exclusive prefix of every tile
__global__ __launch_bounds__(DOM_RADIX) void sd_seg_scan_kernel(const uint16_t *__restrict__ cnt,
                                                                const uint8_t *__restrict__ seg,
                                                                const uint32_t *tfirst_end, uint64_t fixed,
                                                                const uint32_t *__restrict__ gin,
                                                                uint32_t *__restrict__ pre, const int32_t *gate) {
    if (gated_off(gate)) return;
    const uint64_t rows = total_tiles(tfirst_end, fixed);
    const uint64_t r0 = (uint64_t)blockIdx.x * SEG_GROUP;
    if (r0 >= rows) return;
    const uint64_t r1 = r0 + SEG_GROUP < rows ? r0 + SEG_GROUP : rows;
    const int d = threadIdx.x;
    uint32_t run = gin[blockIdx.x * DOM_RADIX + d];
    for (uint64_t r = r0; r < r1; r += SEG_BATCH) {
        uint32_t c[SEG_BATCH];
        bool f[SEG_BATCH];
#pragma unroll
        for (int q = 0; q < SEG_BATCH; ++q) {
            const bool in = r + q < r1;
            c[q] = in ? cnt[(r + q) * DOM_RADIX + d] : 0u;
            f[q] = in && seg[r + q];
        }
#pragma unroll
        for (int q = 0; q < SEG_BATCH; ++q) {
            if (r + q < r1) {
                if (f[q]) run = 0;
                pre[(r + q) * DOM_RADIX + d] = run;
                run += c[q];
            }
        }
    }
}

// The level itself: per tile, every element adds the number of earlier
// elements of its bucket (in v order) with a smaller digit -- from earlier
// tiles (the scanned counts), earlier chunks of the tile (2-D prefix over
// (chunk, digit) in LDS) and earlier lanes of its chunk (ballot masks) --
// and the tile is written out digit-partitioned through LDS.
template <bool FIRST>
__global__ __launch_bounds__(DOM_THREADS) void sd_dominance_kernel(
    const uint32_t *__restrict__ in_t, const uint32_t *__restrict__ in_acc,
    uint32_t *__restrict__ out_t, uint32_t *__restrict__ out_acc, uint64_t n,
    const uint32_t *__restrict__ Zc, int s, int k, const uint32_t *__restrict__ tfirst,
    uint64_t nbuckets, const uint32_t *__restrict__ tile_bucket, const uint32_t *__restrict__ pre,
    int32_t *__restrict__ err, uint64_t ntiles, const int32_t *gate) {
    if (gated_off(gate)) return;
    // chunk histograms -> column prefix; once every position is known, the
    // staged tile (t, then acc) in the same space: 36 KB of LDS in all, so
    // four workgroups share a CU
    __shared__ uint16_t s_h[DOM_CHUNKS][DOM_RADIX];
    __shared__ uint16_t s_pl[DOM_CHUNKS][DOM_RADIX];    // 2-D prefix (earlier chunks, smaller digit)
    static_assert(sizeof(s_h) >= 2 * DOM_TILE * sizeof(uint32_t), "the stage fits the histograms");
    uint32_t *s_st = reinterpret_cast<uint32_t *>(&s_h[0][0]);   // staged t
    uint32_t *s_sa = s_st + DOM_TILE;                           // staged acc
    // per-digit tile starts and smaller-digit counts; before that, the two
    // half sums of the column prefix
    __shared__ uint32_t s_part[2][DOM_RADIX];
    uint32_t *s_lstart = s_part[0], *s_gl = s_part[1];
    __shared__ uint32_t s_base[DOM_RADIX];
    __shared__ uint32_t s_tmp[DOM_WAVES];

    const int tid = threadIdx.x;
    const int lane = tid & (WAVE - 1);
    const int w = tid / WAVE;
    const uint32_t dmask = (1u << k) - 1u;
    for (uint64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    __syncthreads();   // the previous tile has left the LDS
    const TileLoc L = locate_tile<FIRST>(tile, n, Zc, s + k, tfirst, nbuckets, tile_bucket);
    if (!L.valid) break;   // every later tile is past the level's last too
    // same digit, earlier tiles of the bucket (threads below RADIX own a digit)
    const uint32_t G = tid < DOM_RADIX ? pre[tile * DOM_RADIX + tid] : 0u;
    {
        uint64_t *z = reinterpret_cast<uint64_t *>(&s_h[0][0]);
        for (int i = tid; i < DOM_CHUNKS * DOM_RADIX / 4; i += DOM_THREADS) z[i] = 0;
    }
    uint32_t t[DOM_CHUNKS_PER_WAVE], acc[DOM_CHUNKS_PER_WAVE];
    bool ok[DOM_CHUNKS_PER_WAVE];
    load_tile<FIRST>(L, in_t, in_acc, w, lane, t, acc, ok, true);
    __syncthreads();

    // ---- rank inside each 64-lane chunk
    uint16_t q_ic[DOM_CHUNKS_PER_WAVE], l_ic[DOM_CHUNKS_PER_WAVE];
#pragma unroll
    for (int i = 0; i < DOM_CHUNKS_PER_WAVE; ++i) {
        const int c = w * DOM_CHUNKS_PER_WAVE + i;
        const uint32_t d = (t[i] >> s) & dmask;
        uint32_t lt;
        // the top level often has few digit bits (8 buckets at 2^31 accesses)
        const uint64_t eq = k <= 4 ? rank_digit<4>(d, ballot(ok[i]), &lt) : rank_digit<8>(d, ballot(ok[i]), &lt);
        q_ic[i] = ok[i] ? (uint16_t)mbcnt(eq) : 0;
        l_ic[i] = ok[i] ? (uint16_t)lt : 0;
        if (ok[i] && q_ic[i] == 0) s_h[c][d] = (uint16_t)__popcll(eq);
    }
    __syncthreads();

    // ---- column prefix over chunks (thread = digit, two halves of the
    // chunks) and tile totals; all loads are issued before any store
    uint32_t tot = 0;
    {
        constexpr int HALF = DOM_CHUNKS / 2;
        const int d = tid & (DOM_RADIX - 1), c0 = (tid / DOM_RADIX) * HALF;
        uint16_t h[HALF];
        uint32_t sum = 0;
#pragma unroll
        for (int c = 0; c < HALF; ++c) {
            h[c] = s_h[c0 + c][d];
            sum += h[c];
        }
        s_part[tid / DOM_RADIX][d] = sum;
        __syncthreads();
        uint32_t run = c0 ? s_part[0][d] : 0u;
        tot = tid < DOM_RADIX ? s_part[0][d] + s_part[1][d] : 0u;
#pragma unroll
        for (int c = 0; c < HALF; ++c) {
            s_h[c0 + c][d] = (uint16_t)run;
            run += h[c];
        }
    }
    __syncthreads();
    // ---- row prefix over digits: s_pl[c][d] = sum_{d' < d} s_h[c][d']
    for (int c = w * (DOM_CHUNKS / DOM_WAVES); c < (w + 1) * (DOM_CHUNKS / DOM_WAVES); ++c) {
        const uint32_t a0 = s_h[c][4 * lane + 0], a1 = s_h[c][4 * lane + 1];
        const uint32_t a2 = s_h[c][4 * lane + 2], a3 = s_h[c][4 * lane + 3];
        const uint32_t x = wave_excl_scan(a0 + a1 + a2 + a3);
        s_pl[c][4 * lane + 0] = (uint16_t)x;
        s_pl[c][4 * lane + 1] = (uint16_t)(x + a0);
        s_pl[c][4 * lane + 2] = (uint16_t)(x + a0 + a1);
        s_pl[c][4 * lane + 3] = (uint16_t)(x + a0 + a1 + a2);
    }
    uint32_t n_valid;
    const uint32_t lst = block_excl_scan(tot, s_tmp, &n_valid);
    uint32_t gsum;
    const uint32_t GL = block_excl_scan(G, s_tmp, &gsum);   // smaller digit, earlier tiles
    if (tid < DOM_RADIX) {
        const uint64_t X = ((L.bucket << k) + (uint64_t)tid) << s;
        const uint64_t sub = cnt_lt(X < n ? X : n, Zc);
        s_lstart[tid] = lst;
        s_gl[tid] = GL;
        s_base[tid] = (uint32_t)(sub + G - lst);   // wraps mod 2^32 like positions
    }
    __syncthreads();

    // ---- stage the tile digit-partitioned, with the level's count added
    uint32_t pj[DOM_CHUNKS_PER_WAVE];
#pragma unroll
    for (int i = 0; i < DOM_CHUNKS_PER_WAVE; ++i) {
        if (ok[i]) {
            const int c = w * DOM_CHUNKS_PER_WAVE + i;
            const uint32_t d = (t[i] >> s) & dmask;
            pj[i] = s_lstart[d] + s_h[c][d] + q_ic[i];
            acc[i] += s_gl[d] + s_pl[c][d] + l_ic[i];
        }
    }
    __syncthreads();   // the histograms are read: their space becomes the stage
#pragma unroll
    for (int i = 0; i < DOM_CHUNKS_PER_WAVE; ++i) {
        if (ok[i]) {
            s_st[pj[i]] = t[i];
            s_sa[pj[i]] = acc[i];
        }
    }
    __syncthreads();
    for (uint32_t j = tid; j < n_valid; j += DOM_THREADS) {
        const uint32_t tt = s_st[j];
        const uint32_t d = (tt >> s) & dmask;
        const uint32_t dst = s_base[d] + j;
        // consistent prev/next always land inside; inconsistent input is
        // reported instead of written out of bounds
        if (dst < n) {
            out_t[dst] = tt;
            out_acc[dst] = s_sa[j];
        } else {
            atomicOr(err, DEV_ERR_BAD_LAYOUT);
        }
    }
    }
}

// Last 12 bits, one workgroup per 4096-range of t, then D in t order.  The
// level-A counts go straight into a slot per t (acc included), so only the
// six low bits of t are staged for level B, and the prev values needed at the
// end are loaded up front; LDS stays under 40 KB (four workgroups per CU).
__global__ __launch_bounds__(LOC_THREADS, 6) void sd_local_kernel(
    const uint32_t *__restrict__ in_t, const uint32_t *__restrict__ in_acc,
    const uint32_t *__restrict__ prev, uint64_t n, const uint32_t *__restrict__ Zc,
    uint32_t *__restrict__ dist, const int32_t *gate) {
    if (gated_off(gate)) return;
    __shared__ uint32_t slot[LOCAL_SPAN];           // by t: acc + counts; first the column-prefix sums
    __shared__ uint16_t s_h[LOC_CHUNKS][64];        // chunk histograms -> column prefix
    __shared__ uint16_t s_pl[LOC_CHUNKS][64];       // 2-D prefix (earlier chunks, smaller digit)
    __shared__ uint8_t s_low[LOCAL_SPAN];           // bits 0..5 of t, grouped by bits 6..11
    __shared__ uint32_t s_lstart[65];
    __shared__ uint32_t s_tmp[LOC_WAVES];
    uint32_t(*s_part)[64] = reinterpret_cast<uint32_t(*)[64]>(slot);   // [LOC_PARTS][64]

    const int tid = threadIdx.x;
    const int lane = tid & (WAVE - 1);
    const int w = tid / WAVE;
    const uint64_t nchunks = (n + LOCAL_SPAN - 1) / LOCAL_SPAN;
    for (uint64_t chunk = blockIdx.x; chunk < nchunks; chunk += gridDim.x) {
    __syncthreads();   // the previous range has left the LDS
    const uint64_t r0 = chunk * LOCAL_SPAN;
    const uint64_t r1 = r0 + LOCAL_SPAN < n ? r0 + LOCAL_SPAN : n;
    const uint64_t e0 = cnt_lt(r0, Zc), e1 = cnt_lt(r1, Zc);
    for (int i = tid; i < LOC_CHUNKS * 64 / 2; i += LOC_THREADS) reinterpret_cast<uint32_t *>(&s_h[0][0])[i] = 0;

    // ---- loads: the range's elements (v order) and its prev values (t order)
    constexpr int PER = LOCAL_SPAN / LOC_THREADS;   // 8
    // (32-bit offsets from per-range base pointers)
    uint32_t t[LOC_CPW], acc[LOC_CPW], p[PER];
    bool ok[LOC_CPW];
    const uint32_t ne = (uint32_t)(e1 - e0), nt = (uint32_t)(r1 - r0);
    const uint32_t *tb = in_t + e0, *ab = in_acc + e0, *pb = prev + r0;
#pragma unroll
    for (int i = 0; i < LOC_CPW; ++i) {
        const uint32_t o = (uint32_t)((w * LOC_CPW + i) * WAVE + lane);
        ok[i] = o < ne;
        const uint32_t oc = ok[i] ? o : 0u;
        t[i] = tb[oc];
        acc[i] = ab[oc];
    }
    const uint32_t tofs = (uint32_t)tid * PER;
    const uint64_t tbase = r0 + tofs;
    // a full range with aligned bases moves prev and D as two 16-byte
    // vectors per thread
    const bool vec = nt == LOCAL_SPAN && ((reinterpret_cast<uintptr_t>(pb) | reinterpret_cast<uintptr_t>(dist + r0)) & 15) == 0;
    static_assert(PER == 8, "two 16-byte vectors per thread");
    if (vec) {
        const uint4 a = reinterpret_cast<const uint4 *>(pb + tofs)[0];
        const uint4 b = reinterpret_cast<const uint4 *>(pb + tofs)[1];
        p[0] = a.x; p[1] = a.y; p[2] = a.z; p[3] = a.w;
        p[4] = b.x; p[5] = b.y; p[6] = b.z; p[7] = b.w;
    } else {
#pragma unroll
        for (int j = 0; j < PER; ++j) p[j] = pb[tofs + j < nt ? tofs + j : 0u];
    }
    __syncthreads();   // chunk histograms zeroed

    // ---- level A: digit = bits 6..11 of t, chunks of 64 in v order
    uint8_t qa[LOC_CPW], la[LOC_CPW];
#pragma unroll
    for (int i = 0; i < LOC_CPW; ++i) {
        const int c = w * LOC_CPW + i;
        const uint32_t d = (t[i] >> 6) & 63;
        uint32_t lt;
        const uint64_t eq = rank_digit<6>(d, ballot(ok[i]), &lt);
        qa[i] = ok[i] ? (uint8_t)mbcnt(eq) : 0;
        la[i] = ok[i] ? (uint8_t)lt : 0;
        if (ok[i] && qa[i] == 0) s_h[c][d] = (uint16_t)__popcll(eq);
    }
    __syncthreads();
    // column prefix: thread (digit d, part q) scans LOC_CHUNKS / LOC_PARTS
    // chunks, then the part sums are combined
    {
        constexpr int CP = LOC_CHUNKS / LOC_PARTS;
        const int d = tid & 63, q = tid >> 6;
        uint16_t h[CP];
        uint32_t sum = 0;
#pragma unroll
        for (int c = 0; c < CP; ++c) {
            h[c] = s_h[q * CP + c][d];
            sum += h[c];
        }
        s_part[q][d] = sum;
        __syncthreads();
        uint32_t run = 0, tot = 0;
#pragma unroll
        for (int x = 0; x < LOC_PARTS; ++x) {
            const uint32_t v = s_part[x][d];
            if (x < q) run += v;
            tot += v;
        }
#pragma unroll
        for (int c = 0; c < CP; ++c) {
            s_h[q * CP + c][d] = (uint16_t)run;
            run += h[c];
        }
        if (q == 0) {
            const uint32_t incl = wave_incl_scan(tot);
            s_lstart[d] = incl - tot;
            if (d == 63) s_lstart[64] = incl;
        }
    }
    __syncthreads();
    for (int c = w * LOC_CPW; c < (w + 1) * LOC_CPW; ++c) s_pl[c][lane] = (uint16_t)wave_excl_scan(s_h[c][lane]);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < LOC_CPW; ++i) {
        if (ok[i]) {
            const int c = w * LOC_CPW + i;
            const uint32_t d = (t[i] >> 6) & 63;
            s_low[s_lstart[d] + s_h[c][d] + qa[i]] = (uint8_t)(t[i] & 63);
            slot[t[i] & (LOCAL_SPAN - 1)] = acc[i] + s_pl[c][d] + la[i];
        }
    }
    __syncthreads();

    // ---- level B: bits 0..5 inside each 64-range (at most 64 elements,
    // all with different t, so their six low bits are distinct)
    for (int g = w; g < 64; g += LOC_WAVES) {
        const uint32_t base = s_lstart[g];
        const bool okb = (uint32_t)lane < s_lstart[g + 1] - base;
        const uint32_t lb = okb ? s_low[base + lane] : 0u;
        const uint32_t lt = count_smaller_distinct6(lb, okb);
        if (okb) slot[g * 64 + lb] += lt;
    }
    __syncthreads();

    // ---- D in t order: Z(t) from a block scan of cold flags
    uint32_t cold = 0;
#pragma unroll
    for (int j = 0; j < PER; ++j) cold += (tbase + j < n && p[j] == NONE) ? 1u : 0u;
    uint32_t allcold;
    uint32_t z = Zc[chunk] + block_excl_scan(cold, s_tmp, &allcold);
    uint32_t dv[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        if (p[j] == NONE) {
            dv[j] = NONE;
            ++z;
        } else {
            dv[j] = z + slot[(tofs + j) & (LOCAL_SPAN - 1)] - (p[j] + 1u);
        }
    }
    if (vec) {
        reinterpret_cast<uint4 *>(dist + tbase)[0] = make_uint4(dv[0], dv[1], dv[2], dv[3]);
        reinterpret_cast<uint4 *>(dist + tbase)[1] = make_uint4(dv[4], dv[5], dv[6], dv[7]);
    } else {
#pragma unroll
        for (int j = 0; j < PER; ++j)
            if (tbase + j < n) dist[tbase + j] = dv[j];
    }
    }
}

// ---- request-level residency --------------------------------------------
// Request-level distance from the per-access distance of the request-ordered
// stream.  With v = prev + 1 (0 for a cold access) and t in request [s, e):
//     dist_req(t) = dist(t) - #{ j in [s, t) : v(j) < v(t) }.
// When v(t) exceeds every earlier v of its request the count is t - s.  That
// is always so for chained prefix keys: a block's last use is no later than
// the last use of any shallower block of its chain, and each request lists
// its shallower blocks after its deeper ones.  Other key streams take a
// direct count over [s, t) for the accesses that break the order.
// One wave per request (grid-stride), REQ_ITEMS x 64 accesses per step.
constexpr int REQ_ITEMS = 8;

__global__ __launch_bounds__(256) void req_dist_kernel(const uint32_t *__restrict__ prev,
                                                       const uint32_t *__restrict__ dist,
                                                       const uint64_t *__restrict__ blk_off, uint32_t n_seqs,
                                                       uint64_t n, uint32_t *__restrict__ dist_req,
                                                       int32_t *__restrict__ err) {
    const int lane = threadIdx.x & (WAVE - 1);
    const uint32_t waves = gridDim.x * (blockDim.x / WAVE);
    const uint32_t w0 = __builtin_amdgcn_readfirstlane(blockIdx.x * (blockDim.x / WAVE) + threadIdx.x / WAVE);
    if (w0 == 0 && lane == 0 && (blk_off[0] != 0 || blk_off[n_seqs] != n)) atomicOr(err, DEV_ERR_BAD_LAYOUT);
    for (uint32_t r = w0; r < n_seqs; r += waves) {
        const uint64_t s = blk_off[r], e = blk_off[r + 1];
        if (s > e || e > n) {
            if (lane == 0) atomicOr(err, DEV_ERR_BAD_LAYOUT);
            continue;
        }
        uint32_t carry = 0;   // max v over the request's accesses before this step
        for (uint64_t base = s; base < e; base += REQ_ITEMS * WAVE) {
            uint32_t v[REQ_ITEMS], d[REQ_ITEMS];
#pragma unroll
            for (int i = 0; i < REQ_ITEMS; ++i) {
                const uint64_t t = base + i * WAVE + lane;
                const bool ok = t < e;
                v[i] = ok ? prev[t] + 1u : 0u;
                d[i] = ok ? dist[t] : 0u;
            }
#pragma unroll
            for (int i = 0; i < REQ_ITEMS; ++i) {
                const uint64_t t = base + i * WAVE + lane;
                // v(t) is above every earlier v iff it is the prefix max and
                // above the carry (earlier non-zero v are distinct from it)
                const uint32_t incl = wave_incl_max(v[i]);
                const bool top = v[i] == incl && v[i] > carry;
                carry = max(carry, (uint32_t)__builtin_amdgcn_readlane((int)incl, WAVE - 1));
                if (t >= e) continue;
                if (v[i] == 0u) {
                    dist_req[t] = NONE;
                } else if (top) {
                    dist_req[t] = d[i] - (uint32_t)(t - s);
                } else {
                    uint32_t c = 0;
                    for (uint64_t j = s; j < t; ++j) c += (prev[j] + 1u < v[i]) ? 1u : 0u;
                    dist_req[t] = d[i] - c;
                }
            }
        }
    }
}

// Each request's accesses in reverse (deepest block first): the recency
// order of request-level residency.  One wave per request, grid-stride.
__global__ __launch_bounds__(256) void req_order_kernel(const uint64_t *__restrict__ keys,
                                                        const uint32_t *__restrict__ depth,
                                                        const uint64_t *__restrict__ blk_off, uint32_t n_seqs,
                                                        uint64_t n, uint64_t *__restrict__ keys_out,
                                                        uint32_t *__restrict__ depth_out,
                                                        int32_t *__restrict__ err) {
    const int lane = threadIdx.x & (WAVE - 1);
    const uint64_t waves = (uint64_t)gridDim.x * (blockDim.x / WAVE);
    for (uint64_t r = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) / WAVE; r < n_seqs; r += waves) {
        const uint64_t a = blk_off[r], b = blk_off[r + 1];
        if (a > b || b > n) {
            if (lane == 0) atomicOr(err, DEV_ERR_BAD_LAYOUT);
            continue;
        }
        const uint64_t m = b - a;
        for (uint64_t j = lane; j < m; j += WAVE) {
            keys_out[b - 1 - j] = keys[a + j];
            if (depth) depth_out[b - 1 - j] = depth[a + j];
        }
    }
}

struct SdPlan {
    int passes;
    int s[4], k[4];
    uint64_t nbuckets[4];
    uint64_t grid[4];
    uint64_t max_buckets, max_grid;
};

static SdPlan plan_sd(uint64_t n) {
    SdPlan p{};
    int nbits = 0;
    while (nbits < 64 && (1ull << nbits) < n) ++nbits;   // bits of n-1
    const int g = nbits > LOCAL_BITS ? nbits - LOCAL_BITS : 0;
    p.passes = g == 0 ? 1 : (g + 7) / 8;
    if (g == 0) {
        p.k[0] = 1;
    } else {
        p.k[0] = g - 8 * (p.passes - 1);
        for (int i = 1; i < p.passes; ++i) p.k[i] = 8;
    }
    p.s[p.passes - 1] = LOCAL_BITS;
    for (int i = p.passes - 2; i >= 0; --i) p.s[i] = p.s[i + 1] + p.k[i + 1];
    p.max_buckets = 1;
    p.max_grid = 1;
    for (int i = 0; i < p.passes; ++i) {
        const int S = p.s[i] + p.k[i];
        p.nbuckets[i] = S >= 64 ? 1 : (n + (1ull << S) - 1) >> S;
        if (p.nbuckets[i] == 0) p.nbuckets[i] = 1;
        p.grid[i] = (n + DOM_TILE - 1) / DOM_TILE + (i == 0 ? 0 : p.nbuckets[i]);
        if (p.grid[i] == 0) p.grid[i] = 1;
        if (p.nbuckets[i] > p.max_buckets) p.max_buckets = p.nbuckets[i];
        if (p.grid[i] > p.max_grid) p.max_grid = p.grid[i];
    }
    return p;
}


struct SdWs {
    int32_t *hdr;
    uint32_t *cold, *Zc, *tcount, *tfirst, *part, *part_ex;
    uint32_t *at, *aa, *bt, *ba;
    uint16_t *cnt;
    uint8_t *seg, *ghas;
    uint32_t *gsum, *gin, *pre, *tile_bucket;
    size_t bytes;
};

// workspace of one call
static SdWs carve_sd(void *ws, uint64_t n, const SdPlan &p) {
    Carver c{(char *)ws, 0};
    SdWs w;
    const uint64_t nchunks = (n + LOCAL_SPAN - 1) / LOCAL_SPAN;
    const uint64_t groups = (p.max_grid + SEG_GROUP - 1) / SEG_GROUP;
    w.hdr = c.take<int32_t>(WS_HEADER / sizeof(int32_t));
    w.cold = c.take<uint32_t>(nchunks + 1);
    w.Zc = c.take<uint32_t>(nchunks + 2);
    const uint64_t nblocks = (nchunks + SCAN_BLOCK - 1) / SCAN_BLOCK;
    w.part = c.take<uint32_t>(nblocks + 1);
    w.part_ex = c.take<uint32_t>(nblocks + 2);
    w.tcount = c.take<uint32_t>(p.max_buckets + 1);
    w.tfirst = c.take<uint32_t>(p.max_buckets + 2);
    w.at = c.take<uint32_t>(n);
    w.aa = c.take<uint32_t>(n);
    w.bt = c.take<uint32_t>(n);
    w.ba = c.take<uint32_t>(n);
    w.cnt = c.take<uint16_t>(p.max_grid * DOM_RADIX);
    w.seg = c.take<uint8_t>(p.max_grid);
    w.ghas = c.take<uint8_t>(groups);
    w.gsum = c.take<uint32_t>(groups * DOM_RADIX);
    w.gin = c.take<uint32_t>(groups * DOM_RADIX);
    w.pre = c.take<uint32_t>(p.max_grid * DOM_RADIX);
    w.tile_bucket = c.take<uint32_t>(p.max_grid);
    w.bytes = c.off;
    return w;
}

// Workgroups per CU of the loops over tiles: enough that each takes only a
// few tiles (one tile per workgroup balances best: a static share of many
// tiles ran the dominance passes 25% slower), few enough that a launch gated
// off costs little.
constexpr int SD_GRID_PER_CU = 64;

// Z at every multiple of 4096 from the cold (prev = none) flags
static pc_status sd_cold_prefix(const uint32_t *prev, uint64_t n, SdWs &w, hipStream_t s, const int32_t *gate) {
    const uint64_t nchunks = (n + LOCAL_SPAN - 1) / LOCAL_SPAN;
    PC_LAUNCH(K_SD_COLD, sd_cold_count_kernel, dim3(capped(nchunks, SD_GRID_PER_CU)), dim3(256), 0, s, prev, n,
              w.cold, gate);
    const uint64_t nblocks = (nchunks + SCAN_BLOCK - 1) / SCAN_BLOCK;
    PC_LAUNCH(K_SD_SCAN, sd_scan_reduce_kernel, dim3((unsigned)nblocks), dim3(SCAN_THREADS), 0, s, w.cold, nchunks,
              w.part, gate);
    PC_LAUNCH(K_SD_SCAN, sd_scan_kernel, dim3(1), dim3(SCAN_THREADS), 0, s, w.part, nblocks, w.part_ex, gate);
    PC_LAUNCH(K_SD_SCAN, sd_scan_apply_kernel, dim3((unsigned)nblocks), dim3(SCAN_THREADS), 0, s, w.cold, nchunks,
              w.part_ex, nblocks, w.Zc, gate);
    return PC_OK;
}

// The MSD dominance levels over the elements listed in `first` (time t of
// each element, PC_NONE for a slot without one), in the order whose
// dominance count is wanted.  Leaves (t, acc) partitioned by t's 4096-range.
static pc_status sd_levels(const uint32_t *first, uint64_t n, const SdPlan &p, SdWs &w, hipStream_t s,
                           uint32_t **out_t, uint32_t **out_a, const int32_t *gate) {
    uint32_t *src_t = nullptr, *src_a = nullptr;
    for (int i = 0; i < p.passes; ++i) {
        uint32_t *dt = (i & 1) ? w.bt : w.at;
        uint32_t *da = (i & 1) ? w.ba : w.aa;
        const int S = p.s[i] + p.k[i];
        const uint64_t ntiles = p.grid[i];
        const uint64_t cgroups = (p.grid[i] + COUNT_TPW - 1) / COUNT_TPW;
        const unsigned groups = (unsigned)((p.grid[i] + SEG_GROUP - 1) / SEG_GROUP);
        const unsigned grid = capped(ntiles, SD_GRID_PER_CU), cgrid = capped(cgroups, SD_GRID_PER_CU);
        const uint64_t fixed = (n + DOM_TILE - 1) / DOM_TILE;
        if (i == 0) {
            PC_LAUNCH(K_SD_COUNT, sd_count_kernel<true>, dim3(cgrid), dim3(DOM_THREADS), 0, s, first, n, w.Zc,
                      p.s[i], p.k[i], (const uint32_t *)nullptr, (uint64_t)1, (const uint32_t *)nullptr, w.cnt, w.seg,
                      cgroups, gate);
        } else {
            const uint64_t nb = p.nbuckets[i];
            PC_LAUNCH(K_SD_TILES, sd_tile_count_kernel, dim3((unsigned)((nb + 255) / 256)), dim3(256), 0, s, w.Zc,
                      n, S, nb, w.tcount, gate);
            PC_LAUNCH(K_SD_SCAN, sd_scan_kernel, dim3(1), dim3(SCAN_THREADS), 0, s, w.tcount, nb, w.tfirst, gate);
            PC_LAUNCH(K_SD_TILES, sd_tile_bucket_kernel, dim3((unsigned)((p.grid[i] + 255) / 256)), dim3(256), 0,
                      s, w.tfirst, nb, p.grid[i], w.tile_bucket, gate);
            PC_LAUNCH(K_SD_COUNT, sd_count_kernel<false>, dim3(cgrid), dim3(DOM_THREADS), 0, s, src_t, n, w.Zc,
                      p.s[i], p.k[i], w.tfirst, nb, w.tile_bucket, w.cnt, w.seg, cgroups, gate);
        }
        const uint32_t *tend = i == 0 ? nullptr : w.tfirst + p.nbuckets[i];
        PC_LAUNCH(K_SD_SEG, sd_seg_reduce_kernel, dim3(groups), dim3(DOM_RADIX), 0, s, w.cnt, w.seg, tend, fixed,
                  w.gsum, w.ghas, gate);
        PC_LAUNCH(K_SD_SEG, sd_seg_carry_kernel, dim3(DOM_RADIX), dim3(CARRY_THREADS), 0, s, w.gsum, w.ghas, tend,
                  fixed, w.gin, gate);
        PC_LAUNCH(K_SD_SEG, sd_seg_scan_kernel, dim3(groups), dim3(DOM_RADIX), 0, s, w.cnt, w.seg, tend, fixed,
                  w.gin, w.pre, gate);
        if (i == 0) {
            PC_LAUNCH(K_SD_PASS, sd_dominance_kernel<true>, dim3(grid), dim3(DOM_THREADS), 0, s, first,
                      (const uint32_t *)nullptr, dt, da, n, w.Zc, p.s[i], p.k[i], (const uint32_t *)nullptr,
                      (uint64_t)1, (const uint32_t *)nullptr, w.pre, w.hdr, ntiles, gate);
        } else {
            PC_LAUNCH(K_SD_PASS, sd_dominance_kernel<false>, dim3(grid), dim3(DOM_THREADS), 0, s, src_t, src_a, dt,
                      da, n, w.Zc, p.s[i], p.k[i], w.tfirst, p.nbuckets[i], w.tile_bucket, w.pre, w.hdr, ntiles, gate);
        }
        src_t = dt;
        src_a = da;
    }
    *out_t = src_t;
    *out_a = src_a;
    return PC_OK;
}

// The whole dominance count; with a gate, every launch is skipped on the
// device unless the gate word is non-zero.
pc_status stack_distance_gated(const uint32_t *prev, const uint32_t *next, uint64_t n, uint32_t *dist, void *ws,
                               hipStream_t s, const int32_t *gate) {
    const SdPlan p = plan_sd(n);
    SdWs w = carve_sd(ws, n, p);
    pc_status st = fill_u32_gated(reinterpret_cast<uint32_t *>(w.hdr), 0u, 1, s, gate);
    if (st != PC_OK || n == 0) return st;
    if ((st = sd_cold_prefix(prev, n, w, s, gate)) != PC_OK) return st;
    uint32_t *lt, *la;
    if ((st = sd_levels(next, n, p, w, s, &lt, &la, gate)) != PC_OK) return st;
    const uint64_t nchunks = (n + LOCAL_SPAN - 1) / LOCAL_SPAN;
    PC_LAUNCH(K_SD_LOCAL, sd_local_kernel, dim3(capped(nchunks, SD_GRID_PER_CU)), dim3(LOC_THREADS), 0, s, lt, la,
              prev, n, w.Zc, dist, gate);
    return PC_OK;
}

}  // namespace pc

extern "C" {

size_t pc_stack_distance_ws(uint64_t n) {
    const pc::SdPlan p = pc::plan_sd(n);
    return pc::carve_sd(nullptr, n, p).bytes;
}

pc_status pc_stack_distance(const uint32_t *prev, const uint32_t *next, uint64_t n, uint32_t *dist,
                            void *ws, size_t ws_bytes, void *stream) {
    if (n >= (uint64_t)PC_NONE) return PC_ERR_TOO_LARGE;
    if (n > 0 && (!prev || !next || !dist)) return PC_ERR_INVALID;
    if (!ws) return PC_ERR_WORKSPACE;
    if (ws_bytes < pc_stack_distance_ws(n)) return PC_ERR_WORKSPACE;
    return pc::stack_distance_gated(prev, next, n, dist, ws, (hipStream_t)stream, nullptr);
}

size_t pc_request_order_ws(void) { return pc::WS_HEADER; }

pc_status pc_request_order(const uint64_t *keys, const uint32_t *depth, const uint64_t *blk_off, uint32_t n_seqs,
                           uint64_t n, uint64_t *keys_out, uint32_t *depth_out, void *ws, size_t ws_bytes,
                           void *stream) {
    if (n >= (uint64_t)PC_NONE) return PC_ERR_TOO_LARGE;
    if (n > 0 && (!keys || !keys_out || !blk_off)) return PC_ERR_INVALID;
    if ((depth == nullptr) != (depth_out == nullptr)) return PC_ERR_INVALID;
    if ((n > 0 && keys == keys_out) || (depth && depth == depth_out)) return PC_ERR_INVALID;
    if (!ws) return PC_ERR_WORKSPACE;
    if (ws_bytes < pc_request_order_ws()) return PC_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    int32_t *hdr = reinterpret_cast<int32_t *>(ws);
    pc_status st = pc::fill_u32(reinterpret_cast<uint32_t *>(hdr), 0u, 1, s);
    if (st != PC_OK || n == 0 || n_seqs == 0) return st;
    const int cus = pc::device_cus();
    uint64_t grid = ((uint64_t)n_seqs + 3) / 4;
    if (grid > (uint64_t)cus * 8) grid = (uint64_t)cus * 8;
    PC_LAUNCH(pc::K_REQ_ORDER, pc::req_order_kernel, dim3((unsigned)grid), dim3(256), 0, s, keys, depth, blk_off,
              n_seqs, n, keys_out, depth_out, hdr);
    return PC_OK;
}

size_t pc_stack_distance_req_ws(void) { return pc::WS_HEADER; }

pc_status pc_stack_distance_req(const uint32_t *prev, const uint32_t *dist, const uint64_t *blk_off, uint32_t n_seqs,
                                uint64_t n, uint32_t *dist_req, void *ws, size_t ws_bytes, void *stream) {
    if (n >= (uint64_t)PC_NONE) return PC_ERR_TOO_LARGE;
    if (n > 0 && (!prev || !dist || !dist_req || !blk_off || n_seqs == 0)) return PC_ERR_INVALID;
    if (n_seqs >= 0x80000000u) return PC_ERR_TOO_LARGE;
    if (!ws) return PC_ERR_WORKSPACE;
    if (ws_bytes < pc_stack_distance_req_ws()) return PC_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    int32_t *hdr = reinterpret_cast<int32_t *>(ws);
    pc_status st = pc::fill_u32(reinterpret_cast<uint32_t *>(hdr), 0u, 1, s);
    if (st != PC_OK || n == 0) return st;
    const int cus = pc::device_cus();
    uint64_t grid = ((uint64_t)n_seqs + 3) / 4;
    if (grid > (uint64_t)cus * 64) grid = (uint64_t)cus * 64;   // 64 per CU: 7.44 -> 7.15 ms on the full trace
    PC_LAUNCH(pc::K_REQ_DIST, pc::req_dist_kernel, dim3((unsigned)grid), dim3(256), 0, s, prev, dist, blk_off, n_seqs,
              n, dist_req, hdr);
    return PC_OK;
}

}  // extern "C"
