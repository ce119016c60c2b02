// Previous / next use of every access (pc_prev_next_use).
//
// prev[t] = last earlier position with the same key, next[t] = first later
// one.  The paper's offline analysis ranks blocks by time until next access
// (Sec. 3.2 Belady; Sec. 5.2 BeladyCompute); prev == none marks a compulsory
// miss (Sec. 4.6).
//
// GPU mapping: a stable LSD radix sort of (key, t) groups equal keys with t
// ascending; neighbours in sorted order are exactly the (prev, next) links.
//   * one pass computes all eight 8-bit digit histograms (LDS-privatised,
//     then global atomics), one workgroup scans them into digit bases;
//   * each of the eight sort passes is a single "onesweep" kernel: a
//     workgroup takes the next tile from an atomic counter (so every tile it
//     waits on is already running), ranks its 4096 elements by digit with
//     wave ballots (stable: lanes in order, waves in order), publishes its
//     per-digit counts and reads its predecessors' with a decoupled
//     look-back, then writes the tile out through LDS so each digit run is a
//     contiguous burst;
//   * the link kernel reads sorted neighbours and scatters prev/next.
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
    uint32_t epoch, int32_t *__restrict__ err) {
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

// equal neighbours in (key, t) order are consecutive uses of one key
__global__ __launch_bounds__(256) void link_kernel(const uint64_t *__restrict__ sk,
                                                   const uint32_t *__restrict__ sv, uint64_t n,
                                                   uint32_t *__restrict__ prev,
                                                   uint32_t *__restrict__ next) {
    const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const uint64_t k = sk[i];
    const uint32_t t = sv[i];
    const uint32_t p = (i > 0 && sk[i - 1] == k) ? sv[i - 1] : NONE;
    const uint32_t q = (i + 1 < n && sk[i + 1] == k) ? sv[i + 1] : NONE;
    if (t < n) {   // always true for a complete sort; guards the scatter anyway
        prev[t] = p;
        next[t] = q;
    }
}

struct SortWs {
    int32_t *hdr;
    uint32_t *hist, *start, *counters;
    uint64_t *k1, *k2;
    uint32_t *v1, *v2;
    uint64_t *status;
    size_t bytes;
};

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

    const uint64_t *kin = keys;
    const uint32_t *vin = nullptr;
    for (int p = 0; p < pc::SORT_PASSES; ++p) {
        uint64_t *kout = (p & 1) ? w.k2 : w.k1;
        uint32_t *vout = (p & 1) ? w.v2 : w.v1;
        PC_LAUNCH(pc::K_SORT_PASS, pc::sort_pass_kernel, dim3((unsigned)tiles), dim3(pc::SORT_THREADS), 0, s,
                  kin, vin, kout, vout, n, 8 * p, w.start + p * pc::RADIX, w.status, w.counters + p,
                  (uint32_t)(p + 1), w.hdr);
        kin = kout;
        vin = vout;
    }
    const uint64_t lg = (n + 255) / 256;
    PC_LAUNCH(pc::K_LINK, pc::link_kernel, dim3((unsigned)lg), dim3(256), 0, s, kin, vin, n, prev, next);
    return PC_OK;
}

}  // extern "C"
