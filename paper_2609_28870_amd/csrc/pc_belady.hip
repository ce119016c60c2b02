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
// once; each wave runs its capacity's simulation through the trace.
//
//   c <= 1024: the resident set lives in registers, ceil(c / 64) slots per
//   lane.  Per access: one compare per slot and a ballot find the value t;
//   on a miss a free slot is taken, or the wave's largest value (a DPP
//   max-reduction) is replaced.
//
//   c > 1024: the values below a threshold theta are bits of a bitmap over
//   positions (with a one-bit-per-word summary); the values at or above it,
//   the ones evictions take, sit in a sorted buffer in LDS (largest first).
//   Accesses go 64 at a time, one per lane.  Before a batch the buffer is
//   kept clear of the batch's 64 positions (its values below t0 + 128 go to
//   the bitmap), so the batch's hits are the bitmap word of those positions
//   (read and cleared in one exchange) plus the accesses whose block was
//   accessed earlier in the same batch (a wave OR of one-hot next-use
//   offsets).  The misses and the resident count give the batch's number of
//   evictions.  If there are evictions and fewer than 64 dead blocks and
//   buffer values, the buffer is refilled with the bitmap's largest values
//   above the batch (whole words, top down, through the summary); with more
//   than 1024 blocks resident this always yields enough, so no eviction of
//   the batch can reach a bitmap value or a position of the batch.  The
//   evictions then follow the batch's access order: each takes a dead block,
//   or the larger of the buffer's largest value and the largest value
//   inserted earlier in the batch (a masked DPP max over the lanes).  Values
//   inserted by the batch go to the buffer (above theta, merged in sorted
//   order) or to the bitmap; a buffer above 1024 values spills its lowest
//   into the bitmap.  Bitmap words are touched only by their capacity's wave,
//   through relaxed device-scope atomics (they live in L2).
#include "pc_internal.h"

namespace pc {

constexpr uint32_t BEL_SMALL = 1024;          // capacities up to this keep the resident set in registers
constexpr uint32_t BEL_TARGET = 512;          // buffer size a refill aims for and a spill leaves
constexpr uint32_t BEL_SPILL_AT = 1024;       // buffer size above which the lowest values are spilled
constexpr uint32_t BEL_BUF = BEL_SPILL_AT + 2 * WAVE;   // LDS buffer entries (largest fill: spill size + one batch)
constexpr uint64_t BEL_INF = 1ull << 40;      // theta before the first refill: everything in the bitmap
constexpr int32_t DEV_ERR_BELADY = 5;

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
// sum of one uint32 per lane, exact (as two 16-bit halves)
__device__ __forceinline__ uint64_t wave_sum64(uint32_t x) {
    const uint32_t lo = wave_incl_scan(x & 0xFFFFu), hi = wave_incl_scan(x >> 16);
    return (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)lo, WAVE - 1) +
           ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)hi, WAVE - 1) << 16);
}

// next[t] of lane's access, NONE for an invalid entry (flagged)
__device__ __forceinline__ uint32_t load_next(const uint32_t *__restrict__ next, uint64_t t, uint64_t n,
                                              int32_t *err) {
    if (t >= n) return NONE;
    const uint32_t x = next[t];
    if (x != NONE && ((uint64_t)x <= t || (uint64_t)x >= n)) {
        atomicOr(err, DEV_ERR_BAD_LAYOUT);
        return NONE;
    }
    return x;
}

// ---- c <= 1024: SLOTS register slots per lane (0 = empty; no value is 0)
template <int SLOTS>
__device__ void belady_small(const uint32_t *__restrict__ next, const uint32_t *__restrict__ depth, uint64_t n,
                             uint32_t c, uint8_t *__restrict__ flags, uint64_t *hits_out, uint64_t *dsum_out,
                             int32_t *err) {
    const int lane = threadIdx.x;
    uint32_t R[SLOTS];
#pragma unroll
    for (int i = 0; i < SLOTS; ++i) R[i] = 0;
    uint32_t size = 0;
    uint64_t hits = 0, dsum = 0;
    for (uint64_t t0 = 0; t0 < n; t0 += WAVE) {
        const uint64_t t = t0 + lane;
        const uint32_t xv = load_next(next, t, n, err);
        const uint32_t dv = (t < n && depth) ? depth[t] : 0u;
        const int nb = n - t0 < (uint64_t)WAVE ? (int)(n - t0) : WAVE;
        uint64_t hm = 0;
        for (int j = 0; j < nb; ++j) {
            const uint32_t tj = (uint32_t)(t0 + j);
            const uint32_t x = (uint32_t)__builtin_amdgcn_readlane((int)xv, j);
            int hs = -1;
#pragma unroll
            for (int i = 0; i < SLOTS; ++i)
                if (tj != 0 && R[i] == tj) hs = i;
            if (ballot(hs >= 0)) {
                hm |= 1ull << j;
#pragma unroll
                for (int i = 0; i < SLOTS; ++i)
                    if (hs == i) R[i] = x;
            } else if (size < c) {
                int e = -1;
#pragma unroll
                for (int i = SLOTS - 1; i >= 0; --i)
                    if (R[i] == 0) e = i;
                const uint64_t em = ballot(e >= 0);   // non-empty: fewer than c <= 64 * SLOTS resident
                if (lane == __builtin_ctzll(em)) {
#pragma unroll
                    for (int i = 0; i < SLOTS; ++i)
                        if (e == i) R[i] = x;
                }
                ++size;
            } else {
                uint32_t m = 0;
#pragma unroll
                for (int i = 0; i < SLOTS; ++i) m = max(m, R[i]);
                const uint32_t M = wave_max(m);
                if (lane == __builtin_ctzll(ballot(m == M))) {
                    bool done = false;
#pragma unroll
                    for (int i = 0; i < SLOTS; ++i)
                        if (!done && R[i] == M) {
                            R[i] = x;
                            done = true;
                        }
                }
            }
        }
        const bool h = (hm >> lane) & 1;
        hits += (uint64_t)__popcll(hm);
        dsum += wave_sum64(h ? dv : 0u);
        if (flags && t < n) flags[t] = h ? 1 : 0;
    }
    if (lane == 0) {
        *hits_out = hits;
        *dsum_out = dsum;
    }
}

// ---- c > 1024: bitmap below theta, sorted LDS buffer at and above it
struct BelState {
    uint32_t *buf, *alt;   // buf[head .. head + bufn) descending; alt is the spare array
    uint32_t head, bufn;
    uint64_t theta;
};

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
// holds BEL_TARGET values: whole words, top down, the summary skipping
// empty words; theta drops to the lowest value taken
__device__ void refill(BelState &S, uint64_t *l0, uint64_t *l1, uint64_t lo, uint64_t n) {
    const int lane = threadIdx.x;
    compact(S);
    uint64_t hi = S.theta < n + WAVE ? S.theta : n + WAVE;   // exclusive
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
            if (w2 == ~0ull || w2 < wlo) break;
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
    wave_fence();
    __syncthreads();
}

__device__ void belady_large(const uint32_t *__restrict__ next, const uint32_t *__restrict__ depth, uint64_t n,
                             uint64_t c, uint64_t *__restrict__ l0, uint64_t *__restrict__ l1,
                             uint8_t *__restrict__ flags, uint64_t *hits_out, uint64_t *dsum_out, int32_t *err,
                             uint32_t *s_a, uint32_t *s_b, uint32_t *s_new) {
    const int lane = threadIdx.x;
    BelState S{s_a, s_b, 0, 0, BEL_INF};
    uint64_t dead = 0, size = 0, hits = 0, dsum = 0;
    for (uint64_t t0 = 0; t0 < n; t0 += WAVE) {
        const uint64_t t = t0 + lane;
        const bool valid = t < n;
        const uint32_t xv = load_next(next, t, n, err);
        const uint32_t dv = (valid && depth) ? depth[t] : 0u;
        const int nb = n - t0 < (uint64_t)WAVE ? (int)(n - t0) : WAVE;
        const uint64_t vmask = nb == WAVE ? ~0ull : (1ull << nb) - 1;
        const uint64_t win_end = t0 + WAVE;

        // keep the buffer out of this batch's positions
        if (S.theta < t0 + 2 * WAVE) {
            // values below t0 + 128 are the buffer's tail (descending)
            uint32_t lo = 0, hi = S.bufn;
            while (lo < hi) {
                const uint32_t mid = (lo + hi) >> 1;
                if ((uint64_t)S.buf[S.head + mid] >= t0 + 2 * WAVE) lo = mid + 1; else hi = mid;
            }
            for (uint32_t i = lo + lane; i < S.bufn; i += WAVE) bm_insert(l0, l1, S.buf[S.head + i]);
            S.bufn = lo;
            S.theta = t0 + 2 * WAVE;
            wave_fence();
        }

        // hits: the batch's bitmap word (taken and cleared), and blocks accessed
        // earlier in the batch (their next use falls inside it)
        const uint64_t w = t0 >> 6;
        uint64_t wbits = 0;
        if (lane == 0) {
            wbits = bm_xchg(&l0[w], 0ull);
            if (wbits) bm_and(&l1[w >> 6], ~(1ull << (w & 63)));
        }
        wbits = readlane64(wbits, 0);
        const bool inwin = xv != NONE && (uint64_t)xv < win_end;
        const uint64_t link = wave_or64(inwin ? 1ull << ((uint64_t)xv - t0) : 0ull);
        const uint64_t hm = (wbits | link) & vmask;
        const uint64_t misses = (uint64_t)__popcll(vmask & ~hm);
        const uint64_t E = size + misses > c ? size + misses - c : 0;
        if (E > 0 && dead + S.bufn < (uint64_t)WAVE) {
            refill(S, l0, l1, win_end, n);
            if (dead + S.bufn < (uint64_t)WAVE) {   // cannot happen with more than 1024 blocks resident
                if (lane == 0) atomicOr(err, DEV_ERR_BELADY);
                return;
            }
        }
        const uint64_t deadm = ballot(valid && xv == NONE);
        const uint64_t pend = ballot(valid && xv != NONE && (uint64_t)xv >= win_end && (uint64_t)xv >= S.theta);
        const bool to_bitmap = valid && xv != NONE && (uint64_t)xv >= win_end && (uint64_t)xv < S.theta;

        // evictions in access order
        uint64_t alive = pend;
        uint32_t popped = 0;
        if (E == 0) {
            dead += (uint64_t)__popcll(deadm);
            size += misses;
        } else if (dead >= E) {   // every eviction takes a dead block
            dead += (uint64_t)__popcll(deadm) - E;
            size = c;
        } else {
            alive = 0;
            for (int j = 0; j < nb; ++j) {
                const uint64_t bit = 1ull << j;
                if (!(hm & bit)) {
                    if (size == c) {
                        if (dead) {
                            --dead;
                        } else {
                            const uint32_t pb = popped < S.bufn ? S.buf[S.head + popped] : 0u;
                            const bool cand = (alive >> lane) & 1 & ((bit - 1) >> lane);
                            const uint32_t pm = wave_max(cand ? xv : 0u);
                            if (pm > pb) {
                                alive &= ~ballot(cand && xv == pm);
                            } else if (popped < S.bufn) {
                                ++popped;
                            } else {   // no candidate left: cannot happen (see refill)
                                if (lane == 0) atomicOr(err, DEV_ERR_BELADY);
                                return;
                            }
                        }
                    } else {
                        ++size;
                    }
                }
                if (deadm & bit) ++dead;
                if (pend & bit) alive |= bit;
            }
        }

        // the batch's results
        const bool h = (hm >> lane) & 1;
        hits += (uint64_t)__popcll(hm);
        dsum += wave_sum64(h ? dv : 0u);
        if (flags && valid) flags[t] = h ? 1 : 0;
        if (to_bitmap) bm_insert(l0, l1, xv);

        // buffer: drop the popped values, merge the surviving inserts
        S.head += popped;
        S.bufn -= popped;
        const uint32_t nn = (uint32_t)__popcll(alive);
        if (nn) {
            const bool mine = (alive >> lane) & 1;
            // rank among the new values (all distinct), largest first
            uint32_t r = 0;
            for (uint64_t m = alive; m; m &= m - 1) {
                const uint32_t v = (uint32_t)__builtin_amdgcn_readlane((int)xv, __builtin_ctzll(m));
                r += v > xv ? 1u : 0u;
            }
            // buffer values above it (descending array: a lower bound)
            uint32_t lo = 0, hi = S.bufn;
            while (lo < hi) {
                const uint32_t mid = (lo + hi) >> 1;
                if (S.buf[S.head + mid] > xv) lo = mid + 1; else hi = mid;
            }
            if (mine) {
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
            for (uint32_t i = BEL_TARGET + lane; i < S.bufn; i += WAVE) bm_insert(l0, l1, S.buf[S.head + i]);
            S.bufn = BEL_TARGET;
            S.theta = S.buf[S.head + BEL_TARGET - 1];
        }
        wave_fence();
        __syncthreads();
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
    if (c <= BEL_SMALL) {
        const uint32_t c32 = (uint32_t)c;
        if (c32 <= 64) belady_small<1>(next, depth, n, c32, fl, hits + k, dsum + k, err);
        else if (c32 <= 128) belady_small<2>(next, depth, n, c32, fl, hits + k, dsum + k, err);
        else if (c32 <= 256) belady_small<4>(next, depth, n, c32, fl, hits + k, dsum + k, err);
        else if (c32 <= 512) belady_small<8>(next, depth, n, c32, fl, hits + k, dsum + k, err);
        else belady_small<16>(next, depth, n, c32, fl, hits + k, dsum + k, err);
        return;
    }
    belady_large(next, depth, n, c, l0s + (uint64_t)k * w0, l1s + (uint64_t)k * w1, fl, hits + k, dsum + k, err,
                 s_a, s_b, s_new);
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
