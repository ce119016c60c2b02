// Belady's MIN at many cache capacities (pc_belady): the offline ceiling the
// paper compares every online policy with (Sec. 3.2 "Belady's optimum"),
// and the LRU-Belady gap under concurrency (Appendix B).
//
// Demand paging: every accessed block is brought in; when the cache is full
// the victim is the resident block whose next use is farthest away, a block
// that is never used again being farthest of all.  Only next[] is needed.
// Identify a resident block with its next-use position: the block accessed
// at t was inserted at prev(t) with value t, so the access at t hits exactly
// when value t is still present, and is then replaced by next(t).  Values
// are distinct positions (next is one-to-one), blocks without a next use are
// only counted ("dead"), and the victim is a dead block if there is one,
// else the largest value.  Victim ties exist only among dead blocks, so the
// hit count is unique.
//
// GPU mapping: one workgroup of one wave per capacity, all capacities at
// once; each wave runs its capacity's simulation through the trace, 64
// accesses (one per lane) at a time.  The values below a threshold theta
// are bits of a bitmap over positions; the values at or above it, the ones
// evictions take, sit in a sorted buffer in LDS (largest first).  The
// bitmap's words for the 4096 positions just past the batch live in an LDS
// ring, the rest in global memory (with a one-bit-per-word summary).
// Before a batch the buffer's values that fall inside its 64 positions
// leave it for a window register, so the values present in the window are
// that register and one ring word.  Blocks accessed earlier in the same
// batch come back inside it: their next uses are one-hot bits of the window.
//   * When the batch needs no eviction, or only as many as there are dead
//     blocks, nothing in the window can leave: the hits are the window word
//     or'ed with those bits (a wave OR), and the batch's inserts go to the
//     dead count, the bitmap or the buffer in bulk.
//   * Otherwise the evictions (after the dead blocks) take the largest
//     values present, which are among the buffer's top 64 and the batch's
//     own inserts above theta; the wave decides them all at once from a
//     joint ranking of those 128 candidates (a prefix maximum and, per rank,
//     a lowest prefix sum over the batch).  When those candidates run out it
//     walks the batch in access order instead, refilling the buffer from the
//     bitmap's largest values above the window (whole words, top down) and
//     taking the window's largest value when nothing above it is left.
// Values inserted above theta are merged into the buffer in sorted order
// after the batch; a buffer above 256 values spills its lowest into the
// bitmap.  Global bitmap words are touched only by their capacity's wave,
// through relaxed device-scope atomics (they live in L2).  A word entering
// the ring may still hold bits inserted before: every 16 batches, after a
// fence, the words that entered are exchanged for zero and their bits are
// merged into the ring at the next such sync, long before the window gets
// there, so a batch waits on no global memory (the next uses themselves are
// loaded four batches ahead).  A refill syncs at once.
#include "pc_internal.h"

namespace pc {

constexpr uint32_t BEL_TARGET = 128;          // buffer size a refill aims for and a spill leaves
constexpr uint32_t BEL_SPILL_AT = 256;        // buffer size above which the lowest values are spilled
constexpr uint32_t BEL_BUF = BEL_SPILL_AT + 2 * WAVE;   // LDS buffer entries (largest fill: spill size + one batch)
constexpr uint64_t BEL_INF = 1ull << 40;      // theta before the first refill: everything in the bitmap
constexpr int32_t DEV_ERR_BELADY = 5;
constexpr uint64_t BEL_RING = 64;             // bitmap words just past the window held in LDS
constexpr uint64_t BEL_SYNC = 16;             // batches between two exchanges with the global bitmap
static_assert(2 * BEL_SYNC <= BEL_RING, "a word entering the ring is merged before the window reaches it");
constexpr int BEL_AHEAD = 4;                  // batches of next[] and depth[] loaded ahead

__device__ __forceinline__ uint64_t bm_load(const uint64_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t bm_or(uint64_t *p, uint64_t v) {
    return __hip_atomic_fetch_or(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t bm_and(uint64_t *p, uint64_t v) {
    return __hip_atomic_fetch_and(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t bm_xchg(uint64_t *p, uint64_t v) {
    return __hip_atomic_exchange(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// value x into the bitmap: its bit, and its word's bit in the summary
__device__ __forceinline__ void bm_insert(uint64_t *l0, uint64_t *l1, uint32_t x) {
    const uint32_t w = x >> 6;
    bm_or(&l0[w], 1ull << (x & 63));
    bm_or(&l1[w >> 6], 1ull << (w & 63));
}

// every earlier memory operation of the wave completes before later ones
__device__ __forceinline__ void wave_fence() { __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup"); }

__device__ __forceinline__ uint32_t wave_max(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_max(x), WAVE - 1);
}
__device__ __forceinline__ uint64_t wave_or64(uint64_t x) {
    const uint32_t lo = wave_incl_or((uint32_t)x), hi = wave_incl_or((uint32_t)(x >> 32));
    return (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)lo, WAVE - 1) |
           ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)hi, WAVE - 1) << 32);
}
// inclusive prefix OR of one uint64 per lane
__device__ __forceinline__ uint64_t wave_incl_or64(uint64_t x) {
    return (uint64_t)wave_incl_or((uint32_t)x) | ((uint64_t)wave_incl_or((uint32_t)(x >> 32)) << 32);
}
// sum of one uint32 per lane, exact (as two 16-bit halves)
__device__ __forceinline__ uint64_t wave_sum64(uint32_t x) {
    const uint32_t lo = wave_incl_scan(x & 0xFFFFu), hi = wave_incl_scan(x >> 16);
    return (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)lo, WAVE - 1) +
           ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)hi, WAVE - 1) << 16);
}

// next[t] of lane's access (NONE past the end), checked only when used so
// that the load stays in flight until then
__device__ __forceinline__ uint32_t load_next(const uint32_t *__restrict__ next, uint64_t t, uint64_t n) {
    return t < n ? next[t] : NONE;
}
// the loaded next[t], NONE for an invalid entry (flagged)
__device__ __forceinline__ uint32_t checked_next(uint32_t x, uint64_t t, uint64_t n, int32_t *err) {
    if (x != NONE && ((uint64_t)x <= t || (uint64_t)x >= n)) {
        atomicOr(err, DEV_ERR_BAD_LAYOUT);
        return NONE;
    }
    return x;
}

// number of lanes whose value v (0 = none) exceeds x: the 64 values are
// staged in LDS and every lane reads all of them (same addresses for all
// lanes: broadcast reads, four values per read)
__device__ __forceinline__ uint32_t count_above(uint32_t v, uint32_t x, uint32_t *s_tmp) {
    __syncthreads();
    s_tmp[threadIdx.x] = v;
    __syncthreads();
    const uint4 *q = reinterpret_cast<const uint4 *>(s_tmp);
    uint32_t r = 0;
#pragma unroll
    for (int i = 0; i < WAVE / 4; ++i) {
        const uint4 a = q[i];
        r += (a.x > x) + (a.y > x) + (a.z > x) + (a.w > x);
    }
    return r;
}

// ---- the simulation of one capacity
struct BelState {
    uint32_t *buf, *alt;   // buf[head .. head + bufn) descending; alt is the spare array
    uint32_t head, bufn;
    uint64_t theta;
    uint64_t bm_hi;        // every bitmap value is below this
    uint64_t *ring;        // LDS: bitmap words [wb, wb + BEL_RING) of window word wb, slot w % BEL_RING
    uint64_t ex_lo;        // ring words from here on may still have bits in the global bitmap
    uint64_t fl_lo;        // ring words [fl_lo, fl_lo + fl_n) were exchanged and are not merged yet:
    uint32_t fl_n;         //   lane i holds word fl_lo + i's bits in fl_val
    uint64_t fl_val;
    uint64_t w0;           // global bitmap words
};

// value x (not in the window) into the bitmap: an LDS ring word when the
// ring holds its word (ring end rend, exclusive, in words), else the global
// bitmap word and its summary bit
__device__ __forceinline__ void bel_insert(const BelState &S, uint64_t *l0, uint64_t *l1, uint32_t x,
                                           uint64_t rend) {
    if ((uint64_t)(x >> 6) < rend)
        atomicOr(reinterpret_cast<unsigned long long *>(&S.ring[(x >> 6) % BEL_RING]), 1ull << (x & 63));
    else
        bm_insert(l0, l1, x);
}

// Brings the ring up to date with the global bitmap for ring end rend: the
// words exchanged at the last sync are merged (their exchanges have returned
// after the fence), and the words that entered the ring since then are taken
// out of the global bitmap (their global inserts are complete after the
// fence).  Those exchanges return during the next batches and are merged at
// the next sync, BEL_SYNC batches before the window can reach them; with
// `full` they are waited for and merged at once.
__device__ __forceinline__ void ring_sync(BelState &S, uint64_t *l0, uint64_t *l1, uint64_t rend, bool full) {
    const int lane = threadIdx.x;
    if (!full && S.fl_n == 0 && S.bm_hi <= (S.ex_lo << 6)) {
        // nothing in flight, and the words to exchange hold no value
        if (rend > S.ex_lo) S.ex_lo = rend;
        return;
    }
    __builtin_amdgcn_s_waitcnt(0);   // this wave's global inserts and exchanges have completed
    wave_fence();
    if ((uint32_t)lane < S.fl_n && S.fl_val)
        atomicOr(reinterpret_cast<unsigned long long *>(&S.ring[(S.fl_lo + lane) % BEL_RING]), S.fl_val);
    const uint64_t m = rend > S.ex_lo ? rend - S.ex_lo : 0;   // at most BEL_SYNC + 1 words
    const uint64_t w = S.ex_lo + lane;
    uint64_t v = 0;
    if ((uint64_t)lane < m && w < S.w0) {
        v = bm_xchg(&l0[w], 0ull);
        bm_and(&l1[w >> 6], ~(1ull << (w & 63)));
    }
    S.fl_lo = S.ex_lo;
    S.fl_n = (uint32_t)m;
    S.fl_val = v;
    if (rend > S.ex_lo) S.ex_lo = rend;
    if (full) {
        __builtin_amdgcn_s_waitcnt(0);
        wave_fence();
        if ((uint32_t)lane < S.fl_n && S.fl_val)
            atomicOr(reinterpret_cast<unsigned long long *>(&S.ring[(S.fl_lo + lane) % BEL_RING]), S.fl_val);
        S.fl_n = 0;
        S.fl_val = 0;
    }
    __syncthreads();
}

// buffer back to index 0 (through the spare array)
__device__ __forceinline__ void compact(BelState &S) {
    if (S.head == 0) return;
    for (uint32_t i = threadIdx.x; i < S.bufn; i += WAVE) S.alt[i] = S.buf[S.head + i];
    __syncthreads();
    uint32_t *tmp = S.buf;
    S.buf = S.alt;
    S.alt = tmp;
    S.head = 0;
}

// the largest bitmap values in [lo, theta) to the buffer's tail until it
// holds BEL_TARGET values: whole words, top down (the global bitmap's words
// past the ring first, the summary skipping empty words, then the ring's);
// theta drops to the lowest value taken.  lo is the window's end and rend
// the ring's end (words).
__device__ void refill(BelState &S, uint64_t *l0, uint64_t *l1, uint64_t lo_all, uint64_t n, uint64_t rend) {
    const int lane = threadIdx.x;
    ring_sync(S, l0, l1, rend, true);   // every ring value in LDS, every insert visible
    compact(S);
    uint64_t hi = S.theta < n + WAVE ? S.theta : n + WAVE;   // exclusive
    if (S.bm_hi < hi) hi = S.bm_hi;
    // global words: values from the ring's end on
    const uint64_t lo = lo_all > (rend << 6) ? lo_all : (rend << 6);
    const uint64_t wlo = lo >> 6;
    const uint64_t lo_mask = ~((1ull << (lo & 63)) - 1);
    while (S.bufn < BEL_TARGET && hi > lo) {
        uint64_t w = (hi - 1) >> 6;
        const uint64_t room = hi - (w << 6);   // 1 .. 64 positions of word w below hi
        uint64_t bits = bm_load(&l0[w]) & (room >= 64 ? ~0ull : (1ull << room) - 1);
        if (w == wlo) bits &= lo_mask;
        if (!bits) {
            // the highest non-empty word below w
            const uint64_t g = w >> 6;
            uint64_t w2 = ~0ull;
            const uint64_t sb = bm_load(&l1[g]) & ((1ull << (w & 63)) - 1);
            if (sb) {
                w2 = (g << 6) + 63 - (uint64_t)__builtin_clzll(sb);
            } else {
                for (int64_t gb = (int64_t)g - 1; gb >= (int64_t)(wlo >> 6); gb -= WAVE) {
                    const int64_t my = gb - lane;
                    const uint64_t v = my >= (int64_t)(wlo >> 6) ? bm_load(&l1[my]) : 0ull;
                    const uint64_t nz = ballot(v != 0);
                    if (nz) {
                        const int L = __builtin_ctzll(nz);
                        const uint64_t vv = readlane64(v, L);
                        w2 = ((uint64_t)(gb - L) << 6) + 63 - (uint64_t)__builtin_clzll(vv);
                        break;
                    }
                }
            }
            if (w2 == ~0ull || w2 < wlo) {   // nothing left in [lo, hi)
                hi = lo;
                break;
            }
            w = w2;
            bits = bm_load(&l0[w]);
            if (w == wlo) bits &= lo_mask;
            if (!bits) {   // a stale summary bit: go on below this word
                hi = w << 6 > lo ? w << 6 : lo;
                continue;
            }
        }
        // the word's values, largest first
        if ((bits >> lane) & 1) {
            const uint64_t above = lane == WAVE - 1 ? 0ull : bits & (~0ull << (lane + 1));
            S.buf[S.bufn + (uint32_t)__popcll(above)] = (uint32_t)((w << 6) + lane);
        }
        S.bufn += (uint32_t)__popcll(bits);
        const uint64_t low = (w << 6) + (uint64_t)__builtin_ctzll(bits);
        S.theta = low;
        if (lane == 0) {
            const uint64_t old = bm_and(&l0[w], ~bits);
            if ((old & ~bits) == 0) bm_and(&l1[w >> 6], ~(1ull << (w & 63)));
        }
        hi = w << 6 > lo ? w << 6 : lo;
    }
    // ring words, top down, when the global ones did not suffice
    if (hi > lo_all && hi <= lo) {
        const uint64_t rlo_mask = ~((1ull << (lo_all & 63)) - 1);
        while (S.bufn < BEL_TARGET && hi > lo_all) {
            const uint64_t w = (hi - 1) >> 6;
            const uint64_t room = hi - (w << 6);
            uint64_t bits = S.ring[w % BEL_RING] & (room >= 64 ? ~0ull : (1ull << room) - 1);
            if (w == (lo_all >> 6)) bits &= rlo_mask;
            if (bits) {
                if ((bits >> lane) & 1) {
                    const uint64_t above = lane == WAVE - 1 ? 0ull : bits & (~0ull << (lane + 1));
                    S.buf[S.bufn + (uint32_t)__popcll(above)] = (uint32_t)((w << 6) + lane);
                }
                S.bufn += (uint32_t)__popcll(bits);
                S.theta = (w << 6) + (uint64_t)__builtin_ctzll(bits);
                __syncthreads();
                if (lane == 0) S.ring[w % BEL_RING] &= ~bits;
                __syncthreads();
            }
            hi = w << 6 > lo_all ? w << 6 : lo_all;
        }
    }
    // every bitmap value at or above hi has been taken
    if (hi < S.bm_hi) S.bm_hi = hi > lo_all ? hi : lo_all;
    __syncthreads();
}

// the buffer's top 64 values, one per lane (0 past its end)
__device__ __forceinline__ uint32_t buffer_top(const BelState &S) {
    return (uint32_t)threadIdx.x < S.bufn ? S.buf[S.head + threadIdx.x] : 0u;
}

__device__ __forceinline__ uint32_t clamp32(uint64_t v) { return v > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)v; }

__device__ void belady_one(const uint32_t *__restrict__ next, const uint32_t *__restrict__ depth, uint64_t n,
                           uint64_t c64, uint64_t *__restrict__ l0, uint64_t *__restrict__ l1, uint64_t w0,
                           uint8_t *__restrict__ flags, uint64_t *hits_out, uint64_t *dsum_out, int32_t *err,
                           uint32_t *s_a, uint32_t *s_b, uint32_t *s_new, uint32_t *s_tmp, uint64_t *s_sb,
                           uint64_t *s_ring) {
    const int lane = threadIdx.x;
    // the global bitmap starts empty, so the ring's first words are complete
    BelState S{s_a, s_b, 0, 0, BEL_INF, 0, s_ring, BEL_RING, 0, 0, 0, w0};
    for (uint64_t i = lane; i < BEL_RING; i += WAVE) s_ring[i] = 0;
    __syncthreads();
    // resident blocks never exceed n, so the capacity is clamped to 32 bits
    const uint32_t c = clamp32(c64 < n ? c64 : n);
    uint32_t dead = 0, size = 0;
    uint64_t hits = 0, dsum = 0;
    // next uses and depths loaded BEL_AHEAD batches ahead (xq, dq: this batch)
    uint32_t xa[BEL_AHEAD], da[BEL_AHEAD];
#pragma unroll
    for (int b = 0; b < BEL_AHEAD; ++b) {
        const uint64_t tb = (uint64_t)b * WAVE + lane;
        xa[b] = load_next(next, tb, n);
        da[b] = (tb < n && depth) ? depth[tb] : 0u;
    }
    for (uint64_t t0 = 0; t0 < n; t0 += WAVE) {
        const uint32_t xq = checked_next(xa[0], t0 + lane, n, err), dq = da[0];
        const uint64_t t = t0 + lane;
        const bool valid = t < n;
        const uint32_t xv = xq, dv = dq;
        const int nb = n - t0 < (uint64_t)WAVE ? (int)(n - t0) : WAVE;
        const uint64_t vmask = nb == WAVE ? ~0ull : (1ull << nb) - 1;
        const uint64_t we = t0 + WAVE;
        const uint32_t we32 = clamp32(we), t32 = (uint32_t)t0;

        // keep the buffer out of this batch's positions: its values inside the
        // window join the window word.  They are its smallest ones (the buffer
        // is descending and holds no value below the window), distinct
        // positions of the window, so at most its last 64 entries, one per lane.
        uint64_t wlow = 0;
        if (S.theta < we) {
            const uint32_t bn = S.bufn;
            const bool has = (uint32_t)lane < bn;
            const uint32_t v = has ? S.buf[S.head + bn - 1 - lane] : NONE;
            const bool in = has && (uint64_t)v < we;
            wlow = wave_or64(in ? 1ull << (v - t32) : 0ull);
            S.bufn = bn - (uint32_t)__popcll(ballot(in));
            S.theta = we;
        }

        // values present in the window: that register and the window's ring
        // word (complete: merged at a sync at least BEL_SYNC batches ago),
        // taken and cleared; the ring now ends BEL_RING words past the window
        const uint64_t w = t0 >> 6;
        const uint64_t rend = w + BEL_RING;
        uint64_t wbits = wlow;
        if (S.bm_hi > t0) {   // else the bitmap holds nothing at or past the window
            wbits |= S.ring[w % BEL_RING];
            __syncthreads();
            if (lane == 0) S.ring[w % BEL_RING] = 0;
            __syncthreads();
        }
        const bool inwin = xv != NONE && xv < we32;
        const uint64_t link = wave_or64(inwin ? 1ull << (xv - t32) : 0ull);
        uint64_t hm = (wbits | link) & vmask;
        const uint32_t misses = (uint32_t)__popcll(vmask & ~hm);
        const uint32_t E = size + misses > c ? size + misses - c : 0u;
        if (E > dead && dead + S.bufn < (uint32_t)WAVE) refill(S, l0, l1, we, n, rend);

        bool to_buffer, to_bitmap;
        uint32_t popped = 0;
        if (E <= dead) {
            // nothing in the window can leave: bulk
            dead += (uint32_t)__popcll(ballot(valid && xv == NONE)) - E;
            size = size + misses - E;
            to_buffer = valid && xv != NONE && xv >= we32 && (uint64_t)xv >= S.theta;
            to_bitmap = valid && xv != NONE && xv >= we32 && (uint64_t)xv < S.theta;
        } else {
            // access by access.  The batch's inserts above the window are ranked
            // by value; so are they jointly with the buffer's top 64 values
            const bool pend = valid && xv != NONE && xv >= we32;
            const uint64_t pmask = ballot(pend);
            // pending values above this one (values are distinct)
            const uint32_t rank = count_above(pend ? xv : 0u, xv, s_tmp);
            __syncthreads();
            if (pend) s_new[rank] = xv;
            __syncthreads();
            const uint32_t np = (uint32_t)__popcll(pmask);
            const uint32_t sorted = (uint32_t)lane < np ? s_new[lane] : 0u;
            uint32_t top = buffer_top(S);
            const uint32_t nbt = S.bufn < (uint32_t)WAVE ? S.bufn : (uint32_t)WAVE;
            const uint32_t th32 = clamp32(S.theta);
            // joint rank: a pending value's rank plus the top buffer values above
            // it; a top buffer value's index plus the pending values above it
            uint32_t jr = 0, jb = 0;
            if (pend) {
                uint32_t lo = 0, hi = nbt;
                while (lo < hi) {
                    const uint32_t mid = (lo + hi) >> 1;
                    if (S.buf[S.head + mid] > xv) lo = mid + 1; else hi = mid;
                }
                jr = rank + lo;
            }
            const bool isb = (uint32_t)lane < nbt;
            if (isb) {
                uint32_t lo = 0, hi = np;
                while (lo < hi) {
                    const uint32_t mid = (lo + hi) >> 1;
                    if (s_new[mid] > top) lo = mid + 1; else hi = mid;
                }
                jb = (uint32_t)lane + lo;
            }
            const uint64_t b_lo = wave_or64(isb && jb < 64 ? 1ull << jb : 0ull);
            const uint64_t b_hi = wave_or64(isb && jb >= 64 ? 1ull << (jb - 64) : 0ull);
            // candidates at or above theta rank first; below them the bitmap
            // may hold larger values, which only the general walk below handles
            const uint32_t nhigh = nbt + (uint32_t)__popcll(ballot(pend && (uint64_t)xv >= S.theta));
            (void)th32;
            // evictions: the misses after the cache has filled up
            uint64_t ev = vmask & ~hm;
            for (uint32_t k = size; k < c && ev; ++k) ev &= ev - 1;
            const uint64_t dm = ballot(valid && xv == NONE);
            // (1) Evictions that find no dead block.  With D(j) evictions up to
            // and including access j and S(j) dead blocks available before it
            // (a dead insert counts from the next access on), the number left
            // unserved is the running maximum of D(j) - S(j): the real
            // evictions are the accesses where that maximum grows.
            const uint64_t le = lane == WAVE - 1 ? ~0ull : (2ull << lane) - 1;   // lanes up to this one
            const int64_t gap = (int64_t)__popcll(ev & le) - (int64_t)dead - (int64_t)__popcll(dm & (le >> 1));
            const uint32_t un = wave_incl_max(gap > 0 ? (uint32_t)gap : 0u);
            const uint32_t un_prev = (uint32_t)__shfl((int)un, (lane + WAVE - 1) & (WAVE - 1), WAVE);
            const uint64_t real = ballot(un > (lane ? un_prev : 0u));
            const uint32_t E = (uint32_t)__popcll(real);
            // (2) Which candidates the real evictions take.  Each takes the
            // largest one present (the lowest joint rank); the buffer's are
            // present from the start, a pending one after its own access.  For
            // a joint rank k let R(k) be the number of evictions that take a
            // candidate ranked below k.  With A(k) buffer candidates below k,
            // and r_i the count after the i-th eviction, r_i = min(r_{i-1} + 1,
            // A(k) + P_i(k)) where P_i(k) counts the pending candidates below k
            // inserted before it, hence R(k) = min(E, A(k) + E + m(k)) with
            // m(k) the lowest prefix sum (from 0) of the sequence "-1 per
            // eviction, then +1 per such insert", access by access.  The
            // candidate of rank k is taken iff R(k + 1) > R(k).
            s_sb[lane] = 0;
            s_sb[lane + WAVE] = 0;
            __syncthreads();
            if (pend) s_sb[jr] = 1ull << lane;   // jr < 128: rank < 64, plus at most 64 buffer values
            __syncthreads();
            const uint64_t i0 = wave_incl_or64(s_sb[lane]), i1 = wave_incl_or64(s_sb[lane + WAVE]);
            const uint64_t tot0 = readlane64(i0, WAVE - 1), tot1 = readlane64(i1, WAVE - 1);
            // (the shuffles run on every lane: a lane that is off reads as 0)
            const int prev_lane = (lane + WAVE - 1) & (WAVE - 1);
            const uint64_t sh0 = shfl64(i0, prev_lane), sh1 = shfl64(i1, prev_lane);
            const uint64_t below0 = lane ? sh0 : 0ull;            // access bits of pending ranks < lane
            const uint64_t below1 = tot0 | (lane ? sh1 : 0ull);   // ranks < lane + 64
            const uint64_t below2 = tot0 | tot1;                  // ranks < 128
            const uint64_t lt = (1ull << lane) - 1;
            const int a0 = __popcll(b_lo & lt), a1 = __popcll(b_lo) + __popcll(b_hi & lt);
            const int a2 = __popcll(b_lo) + __popcll(b_hi);
            // ranks 64 and up exist only when there are more than 64 candidates
            const bool wide = nbt + np > (uint32_t)WAVE;
            int r0 = 0, r2 = 0, m0 = 0, m2 = 0;
            int r1 = 0, m1 = 0;
            if (wide) {
#pragma unroll
                for (int j = 0; j < WAVE; ++j) {
                    const int pj = (int)((real >> j) & 1);
                    r0 -= pj;
                    r1 -= pj;
                    r2 -= pj;
                    m0 = r0 < m0 ? r0 : m0;
                    m1 = r1 < m1 ? r1 : m1;
                    m2 = r2 < m2 ? r2 : m2;
                    r0 += (int)((below0 >> j) & 1);
                    r1 += (int)((below1 >> j) & 1);
                    r2 += (int)((below2 >> j) & 1);
                }
            } else {
#pragma unroll
                for (int j = 0; j < WAVE; ++j) {
                    const int pj = (int)((real >> j) & 1);
                    r0 -= pj;
                    r2 -= pj;
                    m0 = r0 < m0 ? r0 : m0;
                    m2 = r2 < m2 ? r2 : m2;
                    r0 += (int)((below0 >> j) & 1);
                    r2 += (int)((below2 >> j) & 1);
                }
                m1 = m2;   // every rank from 64 on counts all candidates
            }
            const int Ei = (int)E;
            const int R0 = a0 + Ei + m0 < Ei ? a0 + Ei + m0 : Ei;   // R(lane)
            const int R1 = a1 + Ei + m1 < Ei ? a1 + Ei + m1 : Ei;   // R(lane + 64) (= R(128) when not wide)
            const int R2 = a2 + Ei + m2 < Ei ? a2 + Ei + m2 : Ei;   // R(128)
            const int Rn = nhigh < (uint32_t)WAVE ? __builtin_amdgcn_readlane(R0, (int)nhigh)
                           : nhigh < 2u * WAVE ? __builtin_amdgcn_readlane(R1, (int)nhigh - WAVE) : R2;
            const int nxt_lane = (lane + 1) & (WAVE - 1);
            const int R0n = __shfl(R0, nxt_lane, WAVE), R1n = __shfl(R1, nxt_lane, WAVE);
            const int R0up = lane < WAVE - 1 ? R0n : __builtin_amdgcn_readlane(R1, 0);   // R(lane + 1)
            const int R1up = lane < WAVE - 1 ? R1n : R2;                                  // R(lane + 65)
            const uint64_t gl = ballot(R0up > R0), gh = ballot(R1up > R1);
            const bool ok = Rn == Ei;
            const uint32_t d = dead + (uint32_t)__popcll(dm) - ((uint32_t)__popcll(ev) - E);
            uint64_t gone = 0;   // by pending rank
            if (ok) {
                dead = d;
                size = c;   // evictions happened, so the cache is full
                popped = (uint32_t)__popcll(gl & b_lo) + (uint32_t)__popcll(gh & b_hi);
                const bool g = jr < 64 ? (gl >> jr) & 1 : (gh >> (jr - 64)) & 1;
                gone = ballot(pend && g);   // lane mask
            } else {
            // the general walk: the window in a register, a refill when the
            // buffer and the batch's inserts above theta run out, the window's
            // largest value when nothing above the window is left
            uint64_t avail = 0, rgone = 0;   // by pending rank: inserted so far / evicted again
            uint64_t wreg = wbits;
            hm = 0;
            for (int j = 0; j < nb; ++j) {
                const uint64_t bit = 1ull << j;
                const uint32_t x = (uint32_t)__builtin_amdgcn_readlane((int)xv, j);
                if (wreg & bit) {
                    wreg &= ~bit;
                    hm |= bit;
                } else if (size < c) {
                    ++size;
                } else if (dead) {
                    --dead;
                } else {
                    const uint64_t cand = avail & ~rgone;   // lowest rank = largest value
                    const uint32_t pm = cand ? (uint32_t)__builtin_amdgcn_readlane((int)sorted, __builtin_ctzll(cand)) : 0u;
                    uint32_t pb = popped < S.bufn ? (uint32_t)__builtin_amdgcn_readlane((int)top, popped) : 0u;
                    if (pb == 0 && pm < clamp32(S.theta)) {
                        // buffer exhausted and the bitmap may hold larger values
                        S.head += popped;
                        S.bufn -= popped;
                        popped = 0;
                        refill(S, l0, l1, we, n, rend);
                        top = buffer_top(S);
                        pb = S.bufn ? (uint32_t)__builtin_amdgcn_readlane((int)top, 0) : 0u;
                    }
                    if (pm > pb) {
                        rgone |= cand & (~cand + 1);
                    } else if (pb) {
                        ++popped;
                    } else if (wreg & ~((bit << 1) - 1)) {
                        // nothing resident above the window: its largest value
                        wreg &= ~(1ull << (63 - __builtin_clzll(wreg)));
                    } else {   // nothing to evict: cannot happen with c resident blocks
                        if (lane == 0) atomicOr(err, DEV_ERR_BELADY);
                        return;
                    }
                }
                // lane j's block stays resident with its next use
                if (x == NONE) {
                    ++dead;
                } else if (x < we32) {
                    wreg |= 1ull << (x - t32);
                } else {
                    avail |= 1ull << (uint32_t)__builtin_amdgcn_readlane((int)rank, j);
                }
            }
            gone = ballot(pend && ((rgone >> rank) & 1));
            }
            const bool alive = pend && !((gone >> lane) & 1);
            to_buffer = alive && (uint64_t)xv >= S.theta;
            to_bitmap = alive && (uint64_t)xv < S.theta;
        }

        // the batch's results
        const bool h = (hm >> lane) & 1;
        hits += (uint64_t)__popcll(hm);
        dsum += wave_sum64(h ? dv : 0u);
        if (flags && valid) flags[t] = h ? 1 : 0;
        if (ballot(to_bitmap)) {
            if (to_bitmap) bel_insert(S, l0, l1, xv, rend);
            const uint64_t m = (uint64_t)wave_max(to_bitmap ? xv : 0u) + 1;
            if (m > S.bm_hi) S.bm_hi = m;
        }

        // buffer: drop the popped values, merge the batch's values above theta
        S.head += popped;
        S.bufn -= popped;
        const uint64_t alive = ballot(to_buffer);
        const uint32_t nn = (uint32_t)__popcll(alive);
        if (nn) {
            // rank among the new values (all distinct), largest first
            const uint32_t r = count_above(to_buffer ? xv : 0u, xv, s_tmp);
            // buffer values above it (descending array: a lower bound)
            uint32_t lo = 0, hi = S.bufn;
            while (lo < hi) {
                const uint32_t mid = (lo + hi) >> 1;
                if (S.buf[S.head + mid] > xv) lo = mid + 1; else hi = mid;
            }
            __syncthreads();   // s_new may still be read above
            if (to_buffer) {
                s_new[r] = xv;
                S.alt[r + lo] = xv;
            }
            __syncthreads();
            for (uint32_t i = lane; i < S.bufn; i += WAVE) {
                const uint32_t b = S.buf[S.head + i];
                uint32_t a = 0, z = nn;   // new values above b
                while (a < z) {
                    const uint32_t mid = (a + z) >> 1;
                    if (s_new[mid] > b) a = mid + 1; else z = mid;
                }
                S.alt[i + a] = b;
            }
            __syncthreads();
            uint32_t *tmp = S.buf;
            S.buf = S.alt;
            S.alt = tmp;
            S.head = 0;
            S.bufn += nn;
        }
        // spill the lowest values when the buffer grows large
        if (S.bufn > BEL_SPILL_AT) {
            const uint64_t top_spilled = (uint64_t)S.buf[S.head + BEL_TARGET] + 1;
            for (uint32_t i = BEL_TARGET + lane; i < S.bufn; i += WAVE)
                bel_insert(S, l0, l1, S.buf[S.head + i], rend);
            if (top_spilled > S.bm_hi) S.bm_hi = top_spilled;
            S.bufn = BEL_TARGET;
            S.theta = S.buf[S.head + BEL_TARGET - 1];
        }
        __syncthreads();
        // every BEL_SYNC batches: the ring against the global bitmap, for the
        // next batch's ring end
        if ((w + 1) % BEL_SYNC == 0) ring_sync(S, l0, l1, rend + 1, false);
        // the loads BEL_AHEAD batches ahead
#pragma unroll
        for (int b = 0; b + 1 < BEL_AHEAD; ++b) {
            xa[b] = xa[b + 1];
            da[b] = da[b + 1];
        }
        const uint64_t tn = t + (uint64_t)BEL_AHEAD * WAVE;
        xa[BEL_AHEAD - 1] = load_next(next, tn, n);
        da[BEL_AHEAD - 1] = (tn < n && depth) ? depth[tn] : 0u;
    }
    if (lane == 0) {
        *hits_out = hits;
        *dsum_out = dsum;
    }
}

__global__ __launch_bounds__(WAVE) void belady_kernel(const uint32_t *__restrict__ next,
                                                      const uint32_t *__restrict__ depth, uint64_t n,
                                                      const uint64_t *__restrict__ caps, uint64_t *__restrict__ l0s,
                                                      uint64_t *__restrict__ l1s, uint64_t w0, uint64_t w1,
                                                      uint64_t *__restrict__ hits, uint64_t *__restrict__ dsum,
                                                      uint8_t *__restrict__ flags, int32_t *__restrict__ err) {
    __shared__ uint32_t s_a[BEL_BUF], s_b[BEL_BUF], s_new[WAVE];
    __shared__ __align__(16) uint32_t s_tmp[WAVE];
    __shared__ uint64_t s_sb[2 * WAVE];
    __shared__ uint64_t s_ring[BEL_RING];
    const uint32_t k = blockIdx.x;
    const uint64_t c = caps[k];
    uint8_t *fl = flags ? flags + (uint64_t)k * n : nullptr;
    if (c == 0) {
        if (fl)
            for (uint64_t t = threadIdx.x; t < n; t += WAVE) fl[t] = 0;
        if (threadIdx.x == 0) {
            hits[k] = 0;
            dsum[k] = 0;
        }
        return;
    }
    belady_one(next, depth, n, c, l0s + (uint64_t)k * w0, l1s + (uint64_t)k * w1, w0, fl, hits + k, dsum + k, err,
               s_a, s_b, s_new, s_tmp, s_sb, s_ring);
}

// bitmap words per capacity: one bit per position plus a word of slack, and
// the summary (one bit per bitmap word)
static uint64_t bel_w0(uint64_t n) { return (n + 2 * WAVE) / 64 + 1; }
static uint64_t bel_w1(uint64_t n) { return bel_w0(n) / 64 + 2; }

}  // namespace pc

extern "C" {

size_t pc_belady_ws(uint64_t n, uint32_t n_caps) {
    return pc::WS_HEADER + pc::align_up((size_t)n_caps * (pc::bel_w0(n) + pc::bel_w1(n)) * sizeof(uint64_t));
}

pc_status pc_belady(const uint32_t *next, const uint32_t *depth, uint64_t n, const uint64_t *caps, uint32_t n_caps,
                    uint64_t *hits, uint64_t *depthsum, uint8_t *hit_flags, void *ws, size_t ws_bytes,
                    void *stream) {
    if (n >= (uint64_t)PC_NONE) return PC_ERR_TOO_LARGE;
    if (n_caps == 0 || n_caps > PC_MAX_CAPS) return PC_ERR_INVALID;
    if (!caps || !hits || !depthsum) return PC_ERR_INVALID;
    if (n > 0 && !next) return PC_ERR_INVALID;
    if (!ws) return PC_ERR_WORKSPACE;
    if (ws_bytes < pc_belady_ws(n, n_caps)) return PC_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    int32_t *hdr = reinterpret_cast<int32_t *>(ws);
    uint64_t *l0 = reinterpret_cast<uint64_t *>((char *)ws + pc::WS_HEADER);
    const uint64_t w0 = pc::bel_w0(n), w1 = pc::bel_w1(n);
    uint64_t *l1 = l0 + (uint64_t)n_caps * w0;
    pc_status st;
    if ((st = pc::fill_u32(reinterpret_cast<uint32_t *>(hdr), 0u, 1, s)) != PC_OK) return st;
    if ((st = pc::fill_u32(reinterpret_cast<uint32_t *>(l0), 0u, 2 * (size_t)n_caps * (w0 + w1), s)) != PC_OK)
        return st;
    PC_LAUNCH(pc::K_BELADY, pc::belady_kernel, dim3(n_caps), dim3(pc::WAVE), 0, s, next, depth, n, caps, l0, l1, w0,
              w1, hits, depthsum, hit_flags, hdr);
    return PC_OK;
}

}  // extern "C"
