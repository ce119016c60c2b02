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

// ------------------------------------------------------------ kernel launches
enum KernelId {
    K_FILL32 = 0,
    K_HASH_DIGEST,
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

// fill a uint32 array with a value on a stream (used instead of memset so the
// same code stays valid under graph capture)
pc_status fill_u32(uint32_t *p, uint32_t value, size_t count, hipStream_t s);

// ------------------------------------------------------------ device helpers
__device__ __forceinline__ uint64_t lanemask_lt() {
    const int lane = threadIdx.x & (WAVE - 1);
    return lane ? (~0ull >> (64 - lane)) : 0ull;
}

// popcount of (mask & lanes below me)
__device__ __forceinline__ uint32_t mbcnt(uint64_t mask) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

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

// exclusive prefix sum across the 64 lanes of a wave
__device__ __forceinline__ uint32_t wave_excl_scan(uint32_t v) { return wave_incl_scan(v) - v; }

// Lanes whose `bits`-bit digit equals q (eq) and is smaller than q (lt), for
// q = this lane's own index, from the per-bit ballots B[0..bits) of the
// digits (bit b of every valid lane's digit) and the valid-lane mask vm.
// Walks the bits from the top: a lane is smaller than q at the first bit
// where it has 0 and q has 1, all higher bits being equal.
template <int BITS>
__device__ __forceinline__ void digit_masks(const uint64_t *B, uint64_t vm, uint32_t q, uint64_t &eq,
                                            uint64_t &lt) {
    uint64_t e = vm, l = 0;
#pragma unroll
    for (int b = BITS - 1; b >= 0; --b) {
        const bool bit = (q >> b) & 1;
        if (bit) l |= e & ~B[b];
        e &= bit ? B[b] : ~B[b];
    }
    eq = e;
    lt = l;
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
