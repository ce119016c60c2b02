// Internal helpers of libpc (gfx950 / CDNA4, wave64).  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "pc.h"

namespace pc {

constexpr uint32_t NONE = PC_NONE;
constexpr int WAVE = 64;

// ---------------------------------------------------------------- workspace
// Every workspace starts with a 256-byte header; word 0 is the device-side
// status code (0 = fine), cleared at the start of every call.
constexpr size_t WS_HEADER = 256;
constexpr size_t WS_ALIGN = 256;

inline size_t align_up(size_t x, size_t a = WS_ALIGN) { return (x + a - 1) / a * a; }

struct Carver {
    char *base;
    size_t off;
    template <class T>
    T *take(size_t count) {
        T *p = reinterpret_cast<T *>(base ? base + off : nullptr);
        off = align_up(off + count * sizeof(T));
        return p;
    }
};

// error codes written to the workspace header
constexpr int32_t DEV_ERR_LOOKBACK_TIMEOUT = 1;
constexpr int32_t DEV_ERR_BAD_LAYOUT = 2;
constexpr int32_t DEV_ERR_BAD_CAPS = 3;
constexpr int32_t DEV_ERR_BAD_HIST = 4;

// ------------------------------------------------------------ kernel launches
enum KernelId {
    K_FILL32 = 0,
    K_HASH,
    K_SORT_HIST,
    K_SORT_SCAN,
    K_SORT_PASS,
    K_LINK,
    K_PERM,
    K_PERM_LOCAL,
    K_SD_COLD,
    K_SD_SCAN,
    K_SD_TILES,
    K_SD_COUNT,
    K_SD_SEG,
    K_SD_PASS,
    K_SD_LOCAL,
    K_MRC_HIST,
    K_MRC_COST,
    K_REQ_ORDER,
    K_REQ_DIST,
    K_SESS_REQ,
    K_SESS_DIST,
    K_SESS_PROFILE,
    K_PROF_PACK,
    K_PROF_WALK,
    K_CHAIN_ANCHOR,
    K_CHAIN_STAIR,
    K_CHAIN_SCAN,
    K_CHAIN_COMPACT,
    K_CHAIN_MERGE,
    K_RUNS_COUNT,
    K_RUNS_SCAN,
    K_RUNS_COMPACT,
    K_RUNS_MERGE,
    K_RUNS_FILL,
    K_BELADY,
    K_MRC_MAP,
    K_COUNT
};

void prof_begin(int kid, hipStream_t s);
void prof_end(int kid, hipStream_t s);

// Launch, bracket with profiling events, and turn a launch error into
// PC_ERR_DEVICE.  Must be used inside a function returning pc_status.
#define PC_LAUNCH(kid, kernel, grid, block, shmem, stream, ...)                   \
    do {                                                                          \
        ::pc::prof_begin((kid), (stream));                                        \
        hipLaunchKernelGGL(kernel, (grid), (block), (shmem), (stream), __VA_ARGS__); \
        ::pc::prof_end((kid), (stream));                                          \
        if (hipGetLastError() != hipSuccess) return PC_ERR_DEVICE;                \
    } while (0)

// compute units of the current device (256 on MI355X)
int device_cus();

// Grid of a loop over `items` tiles: at most `per_cu` workgroups per compute
// unit (each takes every gridDim-th tile), so a launch that its gate turns
// off costs a few thousand empty workgroups, not one per tile.
unsigned capped(uint64_t items, int per_cu);

// fill a uint32 array with a value on a stream (used instead of memset so the
// same code stays valid under graph capture)
pc_status fill_u32(uint32_t *p, uint32_t value, size_t count, hipStream_t s);

// Gates: a launch given a device word runs only when the word is non-zero
// (nullptr: always), so a path chosen on the device needs no read-back.
pc_status fill_u32_gated(uint32_t *p, uint32_t value, size_t count, hipStream_t s, const int32_t *gate);

// pc_stack_distance with every launch gated; workspace as
// pc_stack_distance_ws(n)
pc_status stack_distance_gated(const uint32_t *prev, const uint32_t *next, uint64_t n, uint32_t *dist, void *ws,
                               hipStream_t s, const int32_t *gate);

// pc_prev_next_use over min(n, *n_dev) keys (n_dev: a count the GPU wrote;
// nullptr: n), grids and workspace sized for n (pc_prev_next_use_ws(n)),
// every launch gated; `rare`: a call whose gate is seldom on takes small
// persistent grids (cheap when off, slower when on)
pc_status prev_next_core(const uint64_t *keys, uint64_t n, const uint32_t *n_dev, uint32_t *prev, uint32_t *next,
                         const uint32_t *key_hist, void *ws, hipStream_t s, const int32_t *gate, bool rare);

// ------------------------------------------------------------ device helpers
__device__ __forceinline__ bool gated_off(const int32_t *gate) { return gate && *gate == 0; }
__device__ __forceinline__ uint64_t shfl64(uint64_t v, int src) {
    const uint32_t lo = (uint32_t)__shfl((int)(uint32_t)v, src, WAVE);
    const uint32_t hi = (uint32_t)__shfl((int)(uint32_t)(v >> 32), src, WAVE);
    return (uint64_t)lo | ((uint64_t)hi << 32);
}
__device__ __forceinline__ uint64_t dev_count(uint64_t n, const uint32_t *n_dev) {
    if (!n_dev) return n;
    const uint64_t m = *n_dev;
    return m < n ? m : n;
}

__device__ __forceinline__ uint64_t lanemask_lt() {
    const int lane = threadIdx.x & (WAVE - 1);
    return lane ? (~0ull >> (64 - lane)) : 0ull;
}

// popcount of (mask & lanes below me)
__device__ __forceinline__ uint32_t mbcnt(uint64_t mask) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// wave-wide vote straight from the compare (one VALU compare into an SGPR pair)
__device__ __forceinline__ uint64_t ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }

// Look-back status words carry their own payload (flag + count in one word),
// so relaxed device-scope atomics suffice: no other memory is published
// through them.  (Acquire / release at device scope would add an L2
// write-back or invalidate per access on this multi-XCD part.)
__device__ __forceinline__ uint32_t ld_status(const uint32_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_status(uint32_t *p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_status64(const uint64_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_status64(uint64_t *p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Inclusive prefix sum across the 64 lanes of a wave with DPP: four row
// shifts build the sums inside each row of 16 lanes, two row broadcasts carry
// row totals into the rows above (the gfx9 DPP scan).  Lanes shifted in from
// outside a row, and rows outside a broadcast's row mask, contribute 0.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, false);   // row_shr:1
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, false);   // row_shr:2
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, false);   // row_shr:4
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, false);   // row_shr:8
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);   // row_bcast:15
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);   // row_bcast:31
    return x;
}

// Inclusive prefix OR across the 64 lanes of a wave (same DPP pattern as the
// sum above; lanes shifted in from outside a row contribute 0).
__device__ __forceinline__ uint32_t wave_incl_or(uint32_t x) {
    x |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, false);   // row_shr:1
    x |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, false);   // row_shr:2
    x |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, false);   // row_shr:4
    x |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, false);   // row_shr:8
    x |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);   // row_bcast:15
    x |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);   // row_bcast:31
    return x;
}

// Inclusive prefix max across the 64 lanes of a wave (same DPP pattern;
// lanes shifted in from outside a row contribute 0).
__device__ __forceinline__ uint32_t wave_incl_max(uint32_t x) {
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, false));   // row_shr:1
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, false));   // row_shr:2
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, false));   // row_shr:4
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, false));   // row_shr:8
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false));   // row_bcast:15
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false));   // row_bcast:31
    return x;
}

// lane i receives lane i - 1's value (from_lower) or lane i + 1's
// (from_upper) with one DPP move across the whole wave (wave_shr:1 /
// wave_shl:1); the lane without a source keeps its own value
__device__ __forceinline__ uint32_t from_lower(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, 0x138, 0xf, 0xf, false);
}
__device__ __forceinline__ uint32_t from_upper(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, 0x130, 0xf, 0xf, false);
}
__device__ __forceinline__ uint64_t from_lower64(uint64_t v) {
    return (uint64_t)from_lower((uint32_t)v) | ((uint64_t)from_lower((uint32_t)(v >> 32)) << 32);
}
__device__ __forceinline__ uint64_t from_upper64(uint64_t v) {
    return (uint64_t)from_upper((uint32_t)v) | ((uint64_t)from_upper((uint32_t)(v >> 32)) << 32);
}
__device__ __forceinline__ uint64_t readlane64(uint64_t v, int i) {
    return (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, i) |
           ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), i) << 32);
}
// exclusive prefix sum across the 64 lanes of a wave
__device__ __forceinline__ uint32_t wave_excl_scan(uint32_t v) { return wave_incl_scan(v) - v; }

// popcount of (mask & lanes below me) + acc
__device__ __forceinline__ uint32_t mbcnt_acc(uint64_t mask, uint32_t acc) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)mask, acc));
}

// Three-input bitwise function (gfx950 v_bitop3): bit i of `table` is the
// result for (x, y, z) = (i >> 2 & 1, i >> 1 & 1, i & 1).
template <int TABLE>
__device__ __forceinline__ uint64_t bitop3(uint64_t x, uint64_t y, uint32_t z) {
    const uint32_t lo = __builtin_amdgcn_bitop3_b32((uint32_t)x, (uint32_t)y, z, TABLE);
    const uint32_t hi = __builtin_amdgcn_bitop3_b32((uint32_t)(x >> 32), (uint32_t)(y >> 32), z, TABLE);
    return ((uint64_t)hi << 32) | lo;
}
constexpr int BITOP_X_NOTY_Z = 0x20;    // x & ~y & z
constexpr int BITOP_X_YEQZ = 0x90;      // x & ~(y ^ z)

// Rank this lane's BITS-bit digit d among the valid lanes vm of the wave,
// walking the bits from the top: e keeps the lanes whose higher bits equal
// d's; at a bit where d has 1, the lanes of e with 0 there are smaller.
// Returns eq = valid lanes with digit d, and *lt = number of valid lanes
// below this one with a smaller digit.  Per bit: one ballot and six VALU
// operations, no LDS.
template <int BITS>
__device__ __forceinline__ uint64_t rank_digit(uint32_t d, uint64_t vm, uint32_t *lt) {
    // all votes first: the mask chain then never waits on a compare that has
    // just written its SGPR pair
    uint32_t m[BITS];
    uint64_t B[BITS];
#pragma unroll
    for (int b = 0; b < BITS; ++b) {
        m[b] = (uint32_t)__builtin_amdgcn_sbfe((int)d, b, 1);   // all ones when bit b is set
        __asm__("" : "+v"(m[b]));   // vote on m itself (one compare), not on a re-derived bit test
        B[b] = ballot(m[b] != 0);
    }
    uint64_t e = vm;
    uint32_t c = 0;
#pragma unroll
    for (int b = BITS - 1; b >= 0; --b) {
        c = mbcnt_acc(bitop3<BITOP_X_NOTY_Z>(e, B[b], m[b]), c);
        e = bitop3<BITOP_X_YEQZ>(e, B[b], m[b]);
    }
    // pin the count here: otherwise the compiler sinks the mbcnt chain to the
    // count's first use and keeps every intermediate mask alive until then
    __asm__ volatile("" : "+v"(c));
    *lt = c;
    return e;
}

// eq mask only (stable ranking by digit)
template <int BITS>
__device__ __forceinline__ uint64_t match_digit(uint32_t d, uint64_t vm) {
    uint32_t m[BITS];
    uint64_t B[BITS];
#pragma unroll
    for (int b = 0; b < BITS; ++b) {
        m[b] = (uint32_t)__builtin_amdgcn_sbfe((int)d, b, 1);
        __asm__("" : "+v"(m[b]));
        B[b] = ballot(m[b] != 0);
    }
    uint64_t e = vm;
#pragma unroll
    for (int b = BITS - 1; b >= 0; --b) e = bitop3<BITOP_X_YEQZ>(e, B[b], m[b]);
    return e;
}

// For 6-bit digits that are distinct across the valid lanes: the number of
// valid lanes below this one with a smaller digit.  The prefix OR of the
// one-hot digits is the set of digits seen in lower lanes (distinctness keeps
// this lane's own bit out of it once removed), so no per-bit ranking is
// needed.
__device__ __forceinline__ uint32_t count_smaller_distinct6(uint32_t d, bool ok) {
    const uint64_t one = ok ? 1ull << d : 0ull;
    const uint32_t lo = wave_incl_or((uint32_t)one), hi = wave_incl_or((uint32_t)(one >> 32));
    const uint64_t seen = (((uint64_t)hi << 32) | lo) ^ one;
    return (uint32_t)__popcll(seen & (one - 1));
}

// Block-wide exclusive scan of one value per thread (blockDim.x <= 1024).
// `tmp` must hold blockDim.x/64 uint32.  Returns the block total in *total.
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t *tmp, uint32_t *total) {
    const int lane = threadIdx.x & (WAVE - 1);
    const int w = threadIdx.x / WAVE;
    const int nw = blockDim.x / WAVE;
    uint32_t e = wave_excl_scan(v);
    if (lane == WAVE - 1) tmp[w] = e + v;
    __syncthreads();
    uint32_t base = 0, tot = 0;
    for (int i = 0; i < nw; ++i) {
        uint32_t s = tmp[i];
        if (i < w) base += s;
        tot += s;
    }
    __syncthreads();
    *total = tot;
    return base + e;
}

}  // namespace pc
