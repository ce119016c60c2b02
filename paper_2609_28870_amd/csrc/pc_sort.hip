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
// link step resolves such short "mixed" runs by scanning them, and a device
// check switches on the four passes over the high bits when a mixed run could
// be long (then the full 64-bit sort makes equal keys adjacent).
//   * one pass computes all eight 8-bit digit histograms (LDS-privatised,
//     then global atomics), one workgroup scans them into digit bases;
//   * each of the eight sort passes is a single "onesweep" kernel: a
//     workgroup takes the next tile from an atomic counter (so every tile it
//     waits on is already running), ranks its 4096 elements by digit with
//     wave ballots (stable: lanes in order, waves in order), publishes its
//     per-digit counts and reads its predecessors' with a decoupled
//     look-back, then writes the tile out through LDS so each digit run is a
//     contiguous burst;
//   * the link + partition kernels read sorted neighbours into (t, prev,
//     next) triples and move them back to time order (see below).
// Waits in the look-back are bounded: after the spin limit the kernel
// records an error in the workspace header instead of hanging.
#include "pc_internal.h"

namespace pc {

constexpr int RADIX = 256;
constexpr int SORT_THREADS = 512;
constexpr int SORT_WAVES = SORT_THREADS / WAVE;
constexpr int SORT_ITEMS = 8;
constexpr int SORT_TILE = SORT_THREADS * SORT_ITEMS;   // 4096
constexpr int SORT_PASSES = 8;
constexpr uint64_t FLAG_AGG = 1ull << 32;
constexpr uint64_t FLAG_INC = 1ull << 33;
constexpr uint32_t SPIN_LIMIT = 1u << 22;

__global__ __launch_bounds__(256) void sort_hist_kernel(const uint64_t *__restrict__ keys,
                                                        uint64_t n, uint32_t *__restrict__ hist) {
    __shared__ uint32_t h[SORT_PASSES][RADIX];
    for (int i = threadIdx.x; i < SORT_PASSES * RADIX; i += blockDim.x) (&h[0][0])[i] = 0;
    __syncthreads();
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        const uint64_t k = keys[i];
#pragma unroll
        for (int p = 0; p < SORT_PASSES; ++p) atomicAdd(&h[p][(k >> (8 * p)) & 0xFF], 1u);
    }
    __syncthreads();
    for (int i = threadIdx.x; i < SORT_PASSES * RADIX; i += blockDim.x) {
        const uint32_t v = (&h[0][0])[i];
        if (v) atomicAdd(&hist[i], v);
    }
}

// exclusive scan of each pass's 256-bin histogram -> digit bases
__global__ __launch_bounds__(RADIX) void sort_scan_kernel(const uint32_t *__restrict__ hist,
                                                          uint32_t *__restrict__ start) {
    __shared__ uint32_t tmp[RADIX / WAVE];
    for (int p = 0; p < SORT_PASSES; ++p) {
        uint32_t total;
        const uint32_t e = block_excl_scan(hist[p * RADIX + threadIdx.x], tmp, &total);
        start[p * RADIX + threadIdx.x] = e;
    }
}

__global__ __launch_bounds__(SORT_THREADS) void sort_pass_kernel(
    const uint64_t *__restrict__ keys_in, const uint32_t *__restrict__ vals_in,
    uint64_t *__restrict__ keys_out, uint32_t *__restrict__ vals_out, uint64_t n, int shift,
    const uint32_t *__restrict__ start, uint64_t *__restrict__ status, uint32_t *__restrict__ counter,
    uint32_t epoch, int32_t *__restrict__ err, const int32_t *__restrict__ only_if) {
    // passes over the high key bits run only when the link step needs them
    if (only_if && *only_if == 0) return;
    __shared__ uint64_t s_key[SORT_TILE];
    __shared__ uint32_t s_val[SORT_TILE];
    __shared__ uint32_t s_wcnt[SORT_WAVES][RADIX];
    __shared__ uint32_t s_lstart[RADIX];
    __shared__ uint32_t s_gbase[RADIX];
    __shared__ uint32_t s_tmp[SORT_WAVES];
    __shared__ uint32_t s_tile;

    const int tid = threadIdx.x;
    const int lane = tid & (WAVE - 1);
    const int w = tid / WAVE;
    if (tid == 0) s_tile = atomicAdd(counter, 1u);
    for (int i = tid; i < SORT_WAVES * RADIX; i += SORT_THREADS) (&s_wcnt[0][0])[i] = 0;
    __syncthreads();
    const uint32_t tile = s_tile;
    const uint64_t base = (uint64_t)tile * SORT_TILE;

    uint64_t k[SORT_ITEMS];
    uint32_t v[SORT_ITEMS];
    uint32_t rank[SORT_ITEMS];
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
        uint64_t m = ballot(ok[j]);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const bool bit = (d >> b) & 1;
            const uint64_t B = ballot(ok[j] && bit);
            m &= bit ? B : ~B;
        }
        const uint32_t before = mbcnt(m);
        uint32_t cur = 0;
        if (ok[j]) cur = s_wcnt[w][d];
        rank[j] = cur + before;
        if (ok[j] && before == 0) s_wcnt[w][d] = cur + (uint32_t)__popcll(m);
    }
    __syncthreads();
    uint32_t cnt = 0;
    if (tid < RADIX) {
        for (int x = 0; x < SORT_WAVES; ++x) {
            const uint32_t c = s_wcnt[x][tid];
            s_wcnt[x][tid] = cnt;
            cnt += c;
        }
    }
    uint32_t total;
    const uint32_t lst = block_excl_scan(tid < RADIX ? cnt : 0u, s_tmp, &total);
    if (tid < RADIX) s_lstart[tid] = lst;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < SORT_ITEMS; ++j) {
        if (ok[j]) {
            const uint32_t d = (uint32_t)(k[j] >> shift) & 0xFF;
            const uint32_t pos = s_lstart[d] + s_wcnt[w][d] + rank[j];
            s_key[pos] = k[j];
            s_val[pos] = v[j];
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
        s_gbase[tid] = start[tid] + excl - lst;
    }
    __syncthreads();
    const uint64_t left = n - base;
    const uint32_t n_tile = left < (uint64_t)SORT_TILE ? (uint32_t)left : (uint32_t)SORT_TILE;
    for (uint32_t i = tid; i < n_tile; i += SORT_THREADS) {
        const uint64_t kk = s_key[i];
        const uint32_t d = (uint32_t)(kk >> shift) & 0xFF;
        const uint32_t dst = s_gbase[d] + i;
        keys_out[dst] = kk;
        vals_out[dst] = s_val[i];
    }
}

// ---- links, and the way back to time order -------------------------------
// Equal neighbours in (key, t) order are consecutive uses of one key, giving
// the triple (t, prev(t), next(t)).  t is a permutation of [0, n), so the
// triples with t in [a, b) fill exactly positions [a, b) once they are
// partitioned by the top bits of t; the order inside a range does not matter
// because the last step places every triple at its own t.  Each partition
// pass therefore reserves its output runs with one global atomic per
// (workgroup, digit) instead of a look-back, stages each tile digit-sorted
// in LDS and writes each run contiguously.
constexpr int PERM_THREADS = 512;
constexpr int PERM_ITEMS = 8;
constexpr int PERM_TILE = PERM_THREADS * PERM_ITEMS;   // 4096
constexpr int PERM_RADIX = 1024;
constexpr int PERM_LOCAL_BITS = 12;

// After the four passes over the low 32 key bits, equal keys are contiguous
// unless different keys share those bits ("mixed" runs, a few percent of the
// accesses for 64-bit hashes).  The link step resolves them by scanning the
// run: an element inside a block of equal keys finds its neighbour in one
// step, while a block boundary scans back (or forward) to the previous (next)
// block of its key or the run's end.  This check bounds the total of those
// boundary scans from above (short runs are charged their probe length,
// long ones are scanned); when the total exceeds a budget (adversarial keys:
// many keys sharing low bits) it switches on the four passes over the high
// bits, after which equal keys are adjacent and every scan is one step.
__device__ __forceinline__ bool same_low(uint64_t a, uint64_t b) { return (uint32_t)a == (uint32_t)b; }

// Scan from position `from` (inclusive) in direction dir (-1 / +1) over
// elements sharing k's low bits; stop at k (found), at the run's end, or
// after `limit` steps.  Keys are read 8 at a time so a long scan costs one
// memory latency per 8 elements.  Returns the number of elements examined;
// *hit = position of k or UINT64_MAX.
constexpr int SCAN_BATCH = 8;
__device__ __forceinline__ uint64_t scan_run(const uint64_t *__restrict__ sk, uint64_t n, uint64_t k,
                                             uint64_t from, int dir, uint64_t limit, uint64_t *hit) {
    uint64_t steps = 0;
    *hit = ~0ull;
    int64_t j = (int64_t)from;
    while (steps < limit) {
        uint64_t kb[SCAN_BATCH];
#pragma unroll
        for (int q = 0; q < SCAN_BATCH; ++q) {
            const int64_t x = j + dir * q;
            kb[q] = (x >= 0 && (uint64_t)x < n) ? sk[x] : ~k;   // ~k: differs from k in the low bits
        }
#pragma unroll
        for (int q = 0; q < SCAN_BATCH; ++q) {
            ++steps;
            if (kb[q] == k) {
                *hit = (uint64_t)(j + dir * q);
                return steps;
            }
            if (!same_low(kb[q], k)) return steps;
        }
        j += dir * SCAN_BATCH;
    }
    return steps;
}

__global__ __launch_bounds__(256) void sort_mix_check_kernel(const uint64_t *__restrict__ sk, uint64_t n,
                                                             uint64_t budget,
                                                             unsigned long long *__restrict__ work,
                                                             int32_t *__restrict__ need_high) {
    __shared__ uint32_t s_tmp[256 / WAVE];
    // When the run ends within PROBE positions (one probe load), charge PROBE
    // without scanning: the total stays an upper bound.
    constexpr uint64_t PROBE = 32;
    uint64_t cost = 0;
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n && cost <= budget; i += stride) {
        const uint64_t k = sk[i];
        uint64_t hit;
        if (i > 0) {
            const uint64_t kp = sk[i - 1];
            if (same_low(kp, k) && kp != k) {
                if (i < PROBE || !same_low(sk[i - PROBE], k)) cost += PROBE;
                else cost += scan_run(sk, n, k, i - 1, -1, budget + 1, &hit);
            }
        }
        if (i + 1 < n) {
            const uint64_t kn = sk[i + 1];
            if (same_low(kn, k) && kn != k) {
                if (i + PROBE >= n || !same_low(sk[i + PROBE], k)) cost += PROBE;
                else cost += scan_run(sk, n, k, i + 1, +1, budget + 1, &hit);
            }
        }
    }
    // one atomic per workgroup
    const uint32_t c32 = cost > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)cost;
    uint32_t total32;
    block_excl_scan(c32, s_tmp, &total32);
    if (threadIdx.x == 0 && total32) {
        const uint64_t total = atomicAdd(work, (unsigned long long)total32) + total32;
        if (total > budget || total32 == 0xFFFFFFFFu) atomicOr(need_high, 1);
    }
}

// previous / next element with the same full key inside a mixed run (total
// work bounded by the check above)
__device__ __forceinline__ void link_prev(const uint64_t *__restrict__ sk, const uint32_t *__restrict__ sv,
                                          uint64_t n, uint64_t i, uint32_t &p) {
    uint64_t hit;
    scan_run(sk, n, sk[i], i - 1, -1, ~0ull, &hit);
    p = hit != ~0ull ? sv[hit] : NONE;
}
__device__ __forceinline__ void link_next(const uint64_t *__restrict__ sk, const uint32_t *__restrict__ sv,
                                          uint64_t n, uint64_t i, uint32_t &q) {
    uint64_t hit;
    scan_run(sk, n, sk[i], i + 1, +1, ~0ull, &hit);
    q = hit != ~0ull ? sv[hit] : NONE;
}

__device__ __forceinline__ uint64_t shfl_up64(uint64_t v) {
    const uint32_t lo = (uint32_t)__shfl_up((int)(uint32_t)v, 1, WAVE);
    const uint32_t hi = (uint32_t)__shfl_up((int)(uint32_t)(v >> 32), 1, WAVE);
    return (uint64_t)lo | ((uint64_t)hi << 32);
}
__device__ __forceinline__ uint64_t shfl_down64(uint64_t v) {
    const uint32_t lo = (uint32_t)__shfl_down((int)(uint32_t)v, 1, WAVE);
    const uint32_t hi = (uint32_t)__shfl_down((int)(uint32_t)(v >> 32), 1, WAVE);
    return (uint64_t)lo | ((uint64_t)hi << 32);
}

// One workgroup owns a contiguous chunk of the input.  It first counts the
// chunk's digits, reserves one run per digit in the bucket's output range with
// a single global atomic (so each bucket cursor sees one atomic per workgroup,
// not per tile), then streams the chunk tile by tile: LDS counters give each
// element its slot inside its digit, the tile is staged digit-sorted in LDS,
// and each digit's part is appended to the workgroup's run.  A chunk spans at
// most 1024 consecutive buckets (see the plan), so digit = bucket mod 1024
// names them without collision.
template <bool FROM_SORT>
__global__ __launch_bounds__(PERM_THREADS) void perm_partition_kernel(
    const uint64_t *__restrict__ sk, const uint32_t *__restrict__ in_t,
    const uint32_t *__restrict__ in_p, const uint32_t *__restrict__ in_n, uint64_t n, int s,
    uint64_t per_wg, uint32_t *__restrict__ cursor, uint32_t *__restrict__ out_t,
    uint32_t *__restrict__ out_p, uint32_t *__restrict__ out_n, const int32_t *__restrict__ need_high) {
    __shared__ uint32_t s_t[PERM_TILE], s_p[PERM_TILE], s_n[PERM_TILE];
    __shared__ uint32_t s_cnt[PERM_RADIX];
    __shared__ uint32_t s_lstart[PERM_RADIX];
    __shared__ uint32_t s_cur[PERM_RADIX];
    __shared__ uint32_t s_bucket[PERM_RADIX];
    __shared__ uint32_t s_tmp[PERM_THREADS / WAVE];
    constexpr int DPT = PERM_RADIX / PERM_THREADS;   // digits per thread
    const int tid = threadIdx.x;
    const uint64_t lo = (uint64_t)blockIdx.x * per_wg;
    if (lo >= n) return;
    const uint64_t hi = lo + per_wg < n ? lo + per_wg : n;
    const bool full = FROM_SORT && need_high && *need_high != 0;

    // ---- count the chunk's digits and reserve one run per digit
    for (int i = tid; i < PERM_RADIX; i += PERM_THREADS) s_cnt[i] = 0;
    __syncthreads();
    // eight loads in flight per thread before their LDS updates
    for (uint64_t i0 = lo + tid; i0 < hi; i0 += 8 * PERM_THREADS) {
        uint32_t tt[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const uint64_t i = i0 + (uint64_t)q * PERM_THREADS;
            tt[q] = i < hi ? in_t[i] : 0u;
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            if (i0 + (uint64_t)q * PERM_THREADS < hi) {
                const uint32_t d = (tt[q] >> s) & (PERM_RADIX - 1);
                atomicAdd(&s_cnt[d], 1u);
                s_bucket[d] = tt[q] >> s;   // every writer of digit d writes the same bucket
            }
        }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < DPT; ++q) {
        const int d = tid * DPT + q;
        const uint32_t c = s_cnt[d];
        if (c) s_cur[d] = atomicAdd(&cursor[s_bucket[d]], c);
    }
    __syncthreads();

    // ---- stream the chunk tile by tile
    for (uint64_t base = lo; base < hi; base += PERM_TILE) {
        for (int i = tid; i < PERM_RADIX; i += PERM_THREADS) s_cnt[i] = 0;
        __syncthreads();
        uint32_t t[PERM_ITEMS], pv[PERM_ITEMS], nx[PERM_ITEMS], off[PERM_ITEMS];
        bool ok[PERM_ITEMS];
#pragma unroll
        for (int j = 0; j < PERM_ITEMS; ++j) {
            const uint64_t i = base + (uint64_t)j * PERM_THREADS + tid;
            ok[j] = i < hi;
            if (!ok[j]) continue;
            t[j] = in_t[i];
            if (FROM_SORT) {
                // consecutive lanes hold consecutive sorted positions: the
                // neighbours' keys and times come from the adjacent lanes
                // (the wave's first and last lanes load theirs)
                const uint64_t k = sk[i];
                const int lane = tid & (WAVE - 1);
                uint64_t kp = shfl_up64(k), kn = shfl_down64(k);
                uint32_t tp = (uint32_t)__shfl_up((int)t[j], 1, WAVE);
                uint32_t tn = (uint32_t)__shfl_down((int)t[j], 1, WAVE);
                if (lane == 0 && i > 0) { kp = sk[i - 1]; tp = in_t[i - 1]; }
                if ((lane == WAVE - 1 || i + 1 >= hi) && i + 1 < n) { kn = sk[i + 1]; tn = in_t[i + 1]; }
                if (i > 0 && kp == k) pv[j] = tp;
                else if (i > 0 && !full && same_low(kp, k)) link_prev(sk, in_t, n, i, pv[j]);
                else pv[j] = NONE;
                if (i + 1 < n && kn == k) nx[j] = tn;
                else if (i + 1 < n && !full && same_low(kn, k)) link_next(sk, in_t, n, i, nx[j]);
                else nx[j] = NONE;
            } else {
                pv[j] = in_p[i];
                nx[j] = in_n[i];
            }
            off[j] = atomicAdd(&s_cnt[(t[j] >> s) & (PERM_RADIX - 1)], 1u);
        }
        __syncthreads();
        uint32_t c[DPT], mine = 0, total;
#pragma unroll
        for (int q = 0; q < DPT; ++q) {
            c[q] = s_cnt[tid * DPT + q];
            mine += c[q];
        }
        uint32_t run = block_excl_scan(mine, s_tmp, &total);
#pragma unroll
        for (int q = 0; q < DPT; ++q) {
            s_lstart[tid * DPT + q] = run;
            run += c[q];
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < PERM_ITEMS; ++j) {
            if (!ok[j]) continue;
            const uint32_t pos = s_lstart[(t[j] >> s) & (PERM_RADIX - 1)] + off[j];
            s_t[pos] = t[j];
            s_p[pos] = pv[j];
            s_n[pos] = nx[j];
        }
        __syncthreads();
        for (uint32_t j = tid; j < total; j += PERM_THREADS) {
            const uint32_t tt = s_t[j];
            const uint32_t d = (tt >> s) & (PERM_RADIX - 1);
            const uint32_t dst = s_cur[d] + (j - s_lstart[d]);
            if (dst < n) {
                out_t[dst] = tt;
                out_p[dst] = s_p[j];
                out_n[dst] = s_n[j];
            }
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < DPT; ++q) s_cur[tid * DPT + q] += c[q];
        __syncthreads();
    }
}

// cursor[b] = b << s: each bucket's output run starts at its first t
__global__ void perm_cursor_kernel(uint32_t *__restrict__ cursor, uint64_t nb, int s) {
    const uint64_t b = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b < nb) cursor[b] = (uint32_t)(b << s);
}

// every 4096-range of t holds exactly its own triples: place them by t in
// LDS and write prev / next in time order
__global__ __launch_bounds__(256) void perm_local_kernel(const uint32_t *__restrict__ in_t,
                                                         const uint32_t *__restrict__ in_p,
                                                         const uint32_t *__restrict__ in_n, uint64_t n,
                                                         uint32_t *__restrict__ prev,
                                                         uint32_t *__restrict__ next) {
    constexpr uint32_t SPAN = 1u << PERM_LOCAL_BITS;
    __shared__ uint32_t s_p[SPAN], s_n[SPAN];
    const uint64_t r0 = (uint64_t)blockIdx.x * SPAN;
    const uint32_t cnt = n - r0 < SPAN ? (uint32_t)(n - r0) : SPAN;
    for (uint32_t j = threadIdx.x; j < cnt; j += blockDim.x) {
        const uint32_t tt = in_t[r0 + j];
        const uint32_t slot = (uint32_t)(tt - r0) & (SPAN - 1);
        s_p[slot] = in_p[r0 + j];
        s_n[slot] = in_n[r0 + j];
    }
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < cnt; j += blockDim.x) {
        prev[r0 + j] = s_p[j];
        next[r0 + j] = s_n[j];
    }
}

struct SortWs {
    int32_t *hdr;
    uint32_t *hist, *start, *counters;
    uint64_t *k1, *k2;
    uint32_t *v1, *v2;
    uint64_t *status;
    uint32_t *cursor;
    size_t bytes;
};

// Partition plan for the way back to time order.  The last pass uses
// 4096-ranges of t.  The first pass has at most 1024 buckets; every later pass
// splits a bucket into at most 512, so a workgroup chunk (at most 2^20
// elements, smaller than any earlier bucket of >= 2^21) spans at most two
// earlier buckets, i.e. at most 1024 consecutive buckets of its own pass, and
// (bucket mod 1024) names them without collision inside the chunk.
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
    // first pass: up to 10 bits; later passes: up to 9 bits
    int width = 10;
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

}  // namespace pc

extern "C" {

size_t pc_prev_next_use_ws(uint64_t n) { return pc::carve_sort(nullptr, n).bytes; }

pc_status pc_prev_next_use(const uint64_t *keys, uint64_t n, uint32_t *prev, uint32_t *next,
                           void *ws, size_t ws_bytes, void *stream) {
    if (n >= (uint64_t)PC_NONE) return PC_ERR_TOO_LARGE;
    if (n > 0 && (!keys || !prev || !next)) return PC_ERR_INVALID;
    if (!ws) return PC_ERR_WORKSPACE;
    if (ws_bytes < pc_prev_next_use_ws(n)) return PC_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    pc::SortWs w = pc::carve_sort(ws, n);
    pc_status st = pc::fill_u32(reinterpret_cast<uint32_t *>(w.hdr), 0u, 1, s);
    if (st != PC_OK || n == 0) return st;

    const uint64_t tiles = (n + pc::SORT_TILE - 1) / pc::SORT_TILE;
    if ((st = pc::fill_u32(w.hist, 0u, pc::SORT_PASSES * pc::RADIX, s)) != PC_OK) return st;
    if ((st = pc::fill_u32(w.counters, 0u, pc::SORT_PASSES, s)) != PC_OK) return st;
    if ((st = pc::fill_u32(reinterpret_cast<uint32_t *>(w.status), 0u, tiles * pc::RADIX * 2, s)) != PC_OK)
        return st;

    const int cus = pc::device_cus();
    uint64_t hg = (n + 4095) / 4096;
    if (hg > (uint64_t)cus * 4) hg = (uint64_t)cus * 4;
    PC_LAUNCH(pc::K_SORT_HIST, pc::sort_hist_kernel, dim3((unsigned)hg), dim3(256), 0, s, keys, n, w.hist);
    PC_LAUNCH(pc::K_SORT_SCAN, pc::sort_scan_kernel, dim3(1), dim3(pc::RADIX), 0, s, w.hist, w.start);

    // passes 0-3 sort by the low 32 key bits; passes 4-7 run only if the
    // check finds a long mixed run (flag in header word 1)
    int32_t *need_high = w.hdr + 1;
    unsigned long long *mix_work = reinterpret_cast<unsigned long long *>(w.hdr + 2);
    if ((st = pc::fill_u32(reinterpret_cast<uint32_t *>(w.hdr + 1), 0u, 3, s)) != PC_OK) return st;
    const uint64_t *kin = keys;
    const uint32_t *vin = nullptr;
    for (int p = 0; p < pc::SORT_PASSES; ++p) {
        if (p == pc::SORT_PASSES / 2) {
            uint64_t cg = (n + 255) / 256;
            if (cg > (uint64_t)cus * 8) cg = (uint64_t)cus * 8;
            PC_LAUNCH(pc::K_SORT_CHECK, pc::sort_mix_check_kernel, dim3((unsigned)cg), dim3(256), 0, s, kin, n,
                      (uint64_t)2 * n + 4096, mix_work, need_high);
        }
        uint64_t *kout = (p & 1) ? w.k2 : w.k1;
        uint32_t *vout = (p & 1) ? w.v2 : w.v1;
        PC_LAUNCH(pc::K_SORT_PASS, pc::sort_pass_kernel, dim3((unsigned)tiles), dim3(pc::SORT_THREADS), 0, s,
                  kin, vin, kout, vout, n, 8 * p, w.start + p * pc::RADIX, w.status, w.counters + p,
                  (uint32_t)(p + 1), w.hdr, p >= pc::SORT_PASSES / 2 ? (const int32_t *)need_high : nullptr);
        kin = kout;
        vin = vout;
    }
    // links + partition back to time order.  The sort left (key, t) in
    // (k2, v2); triples (t, prev, next) ping-pong between the first sort
    // buffers (k1 viewed as two u32 arrays, v1) and, once the sorted keys
    // have been consumed, the second ones (k2 as two u32 arrays, v2).
    const pc::PermPlan pp = pc::plan_perm(n);
    uint32_t *bt[2] = {reinterpret_cast<uint32_t *>(w.k1), reinterpret_cast<uint32_t *>(w.k2)};
    uint32_t *bp[2] = {bt[0] + n, bt[1] + n};
    uint32_t *bn[2] = {w.v1, w.v2};
    // chunks of at most 2^20 elements: small enough that a chunk of a later
    // pass spans at most two buckets of the previous one, large enough that
    // each bucket cursor sees few atomics
    uint64_t per_wg = (n + (uint64_t)cus * 2 - 1) / ((uint64_t)cus * 2);
    per_wg = (per_wg + pc::PERM_TILE - 1) / pc::PERM_TILE * pc::PERM_TILE;
    if (per_wg > (1ull << 20)) per_wg = 1ull << 20;
    if (per_wg < (uint64_t)pc::PERM_TILE) per_wg = pc::PERM_TILE;
    const unsigned ptiles = (unsigned)((n + per_wg - 1) / per_wg);
    int cur = 0;
    for (int i = 0; i < pp.passes; ++i) {
        const unsigned cg = (unsigned)((pp.buckets[i] + 255) / 256);
        PC_LAUNCH(pc::K_FILL32, pc::perm_cursor_kernel, dim3(cg), dim3(256), 0, s, w.cursor, pp.buckets[i],
                  pp.s[i]);
        if (i == 0) {
            PC_LAUNCH(pc::K_LINK, pc::perm_partition_kernel<true>, dim3(ptiles), dim3(pc::PERM_THREADS), 0, s,
                      kin, vin, (const uint32_t *)nullptr, (const uint32_t *)nullptr, n, pp.s[i], per_wg,
                      w.cursor, bt[0], bp[0], bn[0], (const int32_t *)need_high);
            cur = 0;
        } else {
            const int nxt = cur ^ 1;
            PC_LAUNCH(pc::K_PERM, pc::perm_partition_kernel<false>, dim3(ptiles), dim3(pc::PERM_THREADS), 0,
                      s, (const uint64_t *)nullptr, bt[cur], bp[cur], bn[cur], n, pp.s[i], per_wg,
                      w.cursor, bt[nxt], bp[nxt], bn[nxt], (const int32_t *)nullptr);
            cur = nxt;
        }
    }
    PC_LAUNCH(pc::K_PERM_LOCAL, pc::perm_local_kernel, dim3((unsigned)((n + 4095) / 4096)), dim3(256), 0, s,
              bt[cur], bp[cur], bn[cur], n, prev, next);
    return PC_OK;
}

}  // extern "C"
