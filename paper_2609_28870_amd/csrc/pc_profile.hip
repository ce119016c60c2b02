// Workload characterisation from the index arrays (Sec. 4): reuse intervals
// in time (Sec. 4.2), block lifetimes (Sec. 4.1), access frequency and its
// link to lifetime (Sec. 4.3).  Every block's accesses form one chain through
// next[]; the chains are walked from their first access (prev = none), so
// each block is seen once, in time order, with its count, first and last
// times and the gap of every reuse.
#include "pc_internal.h"

namespace pc {

constexpr int PROF_THREADS = 256;
constexpr int PROF_WAVES = PROF_THREADS / WAVE;
constexpr int PROF_QUEUE = 128;   // pending chain starts per wave (>= 64 idle lanes + one 64-wide scan)

// bin of x over edges[0..k): the number of edges <= x (edges non-decreasing)
__device__ __forceinline__ uint32_t edge_bin(const uint64_t *e, uint32_t k, uint64_t x) {
    uint32_t lo = 0, hi = k;
    while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if (e[mid] <= x) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

// A[t] = next[t] | request(t) << 32: one coalesced read per chain step gives
// both the next access and the request whose timestamp the access takes.
__global__ __launch_bounds__(256) void prof_pack_kernel(const uint32_t *__restrict__ next,
                                                        const uint64_t *__restrict__ blk_off, uint32_t n_seqs,
                                                        uint64_t n, uint64_t *__restrict__ packed,
                                                        int32_t *__restrict__ err) {
    const int lane = threadIdx.x & (WAVE - 1);
    const uint32_t waves = gridDim.x * (blockDim.x / WAVE);
    const uint32_t w0 = __builtin_amdgcn_readfirstlane(blockIdx.x * (blockDim.x / WAVE) + threadIdx.x / WAVE);
    if (w0 == 0 && lane == 0 && (blk_off[0] != 0 || blk_off[n_seqs] != n)) atomicOr(err, DEV_ERR_BAD_LAYOUT);
    for (uint32_t r = w0; r < n_seqs; r += waves) {
        const uint64_t a = blk_off[r], b = blk_off[r + 1];
        if (a > b || b > n) {
            if (lane == 0) atomicOr(err, DEV_ERR_BAD_LAYOUT);
            continue;
        }
        for (uint64_t t = a + lane; t < b; t += WAVE) packed[t] = (uint64_t)next[t] | ((uint64_t)r << 32);
    }
}

// The chain walk.  Waves take 64-position chunks of the trace round-robin
// (a long session's blocks, whose chains are all long, spread over many
// waves); the chain starts found in a chunk go to a per-wave queue in LDS, and
// every lane whose chain has ended takes the next start, so lanes stay busy
// however unequal the chains are.  A lane holds packed[t] of its position t
// (the chain's next position and t's request); each step loads t's request
// timestamp and packed[] of the next position together (one memory latency
// per step, not two), bins the gap since the previous access and, at the
// chain's end, the block's lifetime and frequency.  Histograms accumulate in
// LDS and are added to the outputs at the end.
__global__ __launch_bounds__(PROF_THREADS) void prof_walk_kernel(
    const uint32_t *__restrict__ prev, const uint64_t *__restrict__ packed, const uint64_t *__restrict__ ts_us,
    uint32_t n_seqs, uint64_t n, const uint64_t *__restrict__ edges, uint32_t n_edges, uint32_t freq_max,
    uint64_t *__restrict__ interval, uint64_t *__restrict__ lifetime, uint64_t *__restrict__ freq,
    uint64_t *__restrict__ life_by_class, int32_t *__restrict__ err) {
    // LDS sized by the call (edges, bins, frequency bins): smaller
    // histograms leave room for more waves, and the walk is latency-bound
    extern __shared__ uint64_t smem[];
    __shared__ uint32_t s_queue[PROF_WAVES][PROF_QUEUE];
    const int tid = threadIdx.x;
    const int lane = tid & (WAVE - 1);
    const int wv = tid / WAVE;
    const uint32_t kb = n_edges + 1;
    uint64_t *s_edges = smem;                                               // n_edges
    uint32_t *s_ival = reinterpret_cast<uint32_t *>(s_edges + n_edges);     // kb
    uint32_t *s_class = s_ival + kb;                                        // classes * kb
    uint32_t *s_freq = s_class + PC_FREQ_CLASSES * kb;                      // freq_max + 1
    for (uint32_t i = tid; i < n_edges; i += PROF_THREADS) {
        s_edges[i] = edges[i];
        if (blockIdx.x == 0 && i + 1 < n_edges && edges[i] > edges[i + 1]) atomicOr(err, DEV_ERR_BAD_CAPS);
    }
    for (uint32_t i = tid; i < kb; i += PROF_THREADS) s_ival[i] = 0;
    for (uint32_t i = tid; i < PC_FREQ_CLASSES * kb; i += PROF_THREADS) s_class[i] = 0;
    for (uint32_t i = tid; i <= freq_max; i += PROF_THREADS) s_freq[i] = 0;
    __syncthreads();

    const uint64_t chunks = (n + WAVE - 1) / WAVE;
    const uint64_t stride = (uint64_t)gridDim.x * PROF_WAVES;
    uint64_t c = (uint64_t)blockIdx.x * PROF_WAVES + wv;   // next chunk to scan
    uint32_t qh = 0, qt = 0;                                 // queue head / tail (wave-uniform)
    bool active = false;
    uint32_t t = 0, f = 0;
    uint64_t a = 0;   // packed[t]
    uint64_t ts_first = 0, ts_last = 0;
    uint32_t *queue = s_queue[wv];
    for (;;) {
        const uint64_t idle = ballot(!active);
        const uint32_t n_idle = (uint32_t)__popcll(idle);
        // refill the queue with the chain starts of the next chunks
        while (qt - qh < n_idle && c < chunks) {
            const uint64_t pos = c * WAVE + lane;
            const bool head = pos < n && prev[pos] == NONE;
            const uint64_t hm = ballot(head);
            if (head) queue[(qt + mbcnt(hm)) % PROF_QUEUE] = (uint32_t)pos;
            qt += (uint32_t)__popcll(hm);
            c += stride;
        }
        __builtin_amdgcn_wave_barrier();
        const uint32_t avail = qt - qh;
        if (!active) {
            const uint32_t r = mbcnt(idle);
            if (r < avail) {
                t = queue[(qh + r) % PROF_QUEUE];
                a = packed[t];
                active = true;
                f = 0;
            }
        }
        qh += n_idle < avail ? n_idle : avail;
        __builtin_amdgcn_wave_barrier();
        if (ballot(active) == 0) break;   // no chain left: the queue is empty and every chunk scanned
        if (active) {
            const uint32_t nx = (uint32_t)a;
            const uint32_t r = (uint32_t)(a >> 32);
            const bool ends = nx == NONE || nx <= t || (uint64_t)nx >= n;   // chains run forward
            // both loads in flight at once
            const uint64_t ts = r < n_seqs ? ts_us[r] : 0;
            const uint64_t an = ends ? 0ull : packed[nx];
            if (f == 0) {
                ts_first = ts;
            } else {
                atomicAdd(&s_ival[edge_bin(s_edges, n_edges, ts - ts_last)], 1u);
            }
            ts_last = ts;
            ++f;
            if (ends) {   // anything but a later position ends the chain
                if (nx != NONE) atomicOr(err, DEV_ERR_BAD_LAYOUT);
                const uint32_t cls = 31u - (uint32_t)__builtin_clz(f);
                atomicAdd(&s_class[cls * kb + edge_bin(s_edges, n_edges, ts_last - ts_first)], 1u);
                atomicAdd(&s_freq[f < freq_max ? f : freq_max], 1u);
                active = false;
            } else {
                t = nx;
                a = an;
            }
        }
    }
    __syncthreads();
    for (uint32_t i = tid; i < kb; i += PROF_THREADS) {
        if (s_ival[i]) atomicAdd((unsigned long long *)&interval[i], (unsigned long long)s_ival[i]);
        uint64_t life = 0;
        for (uint32_t cl = 0; cl < PC_FREQ_CLASSES; ++cl) {
            const uint32_t v = s_class[cl * kb + i];
            life += v;
            if (v) atomicAdd((unsigned long long *)&life_by_class[cl * kb + i], (unsigned long long)v);
        }
        if (life) atomicAdd((unsigned long long *)&lifetime[i], (unsigned long long)life);
    }
    for (uint32_t i = tid; i <= freq_max; i += PROF_THREADS)
        if (s_freq[i]) atomicAdd((unsigned long long *)&freq[i], (unsigned long long)s_freq[i]);
}

struct ProfWs {
    int32_t *hdr;
    uint64_t *packed;
    size_t bytes;
};

static ProfWs carve_prof(void *ws, uint64_t n) {
    Carver c{(char *)ws, 0};
    ProfWs w;
    w.hdr = c.take<int32_t>(WS_HEADER / sizeof(int32_t));
    w.packed = c.take<uint64_t>(n);
    w.bytes = c.off;
    return w;
}

}  // namespace pc

extern "C" {

size_t pc_reuse_profile_ws(uint64_t n) { return pc::carve_prof(nullptr, n).bytes; }

pc_status pc_reuse_profile(const uint32_t *prev, const uint32_t *next, const uint64_t *blk_off, const uint64_t *ts_us,
                           uint32_t n_seqs, uint64_t n, const uint64_t *edges, uint32_t n_edges, uint32_t freq_max,
                           uint64_t *interval, uint64_t *lifetime, uint64_t *freq, uint64_t *life_by_class, void *ws,
                           size_t ws_bytes, void *stream) {
    if (n >= (uint64_t)PC_NONE) return PC_ERR_TOO_LARGE;
    if (n_seqs >= 0x80000000u) return PC_ERR_TOO_LARGE;
    if (n_edges < 1 || n_edges > PC_MAX_PROFILE_EDGES || freq_max < 1 || freq_max > PC_MAX_FREQ)
        return PC_ERR_INVALID;
    if (!edges || !interval || !lifetime || !freq || !life_by_class) return PC_ERR_INVALID;
    if (n > 0 && (!prev || !next || !blk_off || !ts_us || n_seqs == 0)) return PC_ERR_INVALID;
    if (!ws) return PC_ERR_WORKSPACE;
    if (ws_bytes < pc_reuse_profile_ws(n)) return PC_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    pc::ProfWs w = pc::carve_prof(ws, n);
    pc_status st = pc::fill_u32(reinterpret_cast<uint32_t *>(w.hdr), 0u, 1, s);
    if (st != PC_OK) return st;
    const size_t kb = (size_t)n_edges + 1;
    if ((st = pc::fill_u32(reinterpret_cast<uint32_t *>(interval), 0u, 2 * kb, s)) != PC_OK) return st;
    if ((st = pc::fill_u32(reinterpret_cast<uint32_t *>(lifetime), 0u, 2 * kb, s)) != PC_OK) return st;
    if ((st = pc::fill_u32(reinterpret_cast<uint32_t *>(freq), 0u, 2 * ((size_t)freq_max + 1), s)) != PC_OK)
        return st;
    if ((st = pc::fill_u32(reinterpret_cast<uint32_t *>(life_by_class), 0u, 2 * kb * PC_FREQ_CLASSES, s)) != PC_OK)
        return st;
    if (n == 0) return PC_OK;
    const int cus = pc::device_cus();
    uint64_t pg = ((uint64_t)n_seqs + 3) / 4;
    if (pg > (uint64_t)cus * 64) pg = (uint64_t)cus * 64;   // 64 per CU: 5.9 -> 5.3 ms on the full trace
    PC_LAUNCH(pc::K_PROF_PACK, pc::prof_pack_kernel, dim3((unsigned)pg), dim3(256), 0, s, next, blk_off, n_seqs, n,
              w.packed, w.hdr);
    const uint64_t chunks = (n + pc::WAVE - 1) / pc::WAVE;
    uint64_t grid = (chunks + pc::PROF_WAVES - 1) / pc::PROF_WAVES;
    if (grid > (uint64_t)cus * 7) grid = (uint64_t)cus * 7;   // about one resident round
    const size_t shmem = (size_t)n_edges * 8 + (kb + (size_t)PC_FREQ_CLASSES * kb + freq_max + 1) * 4;
    PC_LAUNCH(pc::K_PROF_WALK, pc::prof_walk_kernel, dim3((unsigned)grid), dim3(pc::PROF_THREADS), shmem, s, prev,
              w.packed, ts_us, n_seqs, n, edges, n_edges, freq_max, interval, lifetime, freq, life_by_class, w.hdr);
    return PC_OK;
}

}  // extern "C"
