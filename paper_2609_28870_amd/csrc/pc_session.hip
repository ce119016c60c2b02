// Session-level eviction (Sec. 5.3 "Block-Level vs. Session-Level Eviction":
// whole sessions are evicted at once) as a size-weighted stack distance.
//
// Readings (the paper gives no simulator detail for this mode):
//   - a session's footprint after one of its requests is the largest block
//     count among its requests so far (contexts are append-only, Sec. 2.3);
//   - resident sessions are kept in recency order of their latest request
//     and evicted whole from the least recent end while the resident
//     footprints exceed the capacity;
//   - a block hits if the session that made its previous access is resident
//     when the request arrives.
// Footprints only grow and sessions only join the top of the list, so the
// footprint held above a session only grows until its next request: q is
// resident at request tau iff w(lq) + W(lq, tau) <= c, where lq is q's latest
// request before tau, w the footprint after a request, and
//     W(a, tau) = sum of w(i) over requests i in (a, tau) whose session's next
//                 request is tau or later
// (the latest footprint of every other session active since a).  The
// distance of a block is w(lq) - 1 + W(lq, tau), a hit at c iff it is < c.
#include "pc_internal.h"

namespace pc {

// largest r in [lo, hi] with blk_off[r] <= t
__device__ __forceinline__ uint32_t sess_req_find(const uint64_t *__restrict__ blk_off, uint32_t lo, uint32_t hi,
                                                  uint64_t t) {
    while (lo < hi) {
        const uint32_t mid = lo + (hi - lo + 1) / 2;
        if (blk_off[mid] <= t) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

constexpr int PAGE_BITS = 12;   // the request table is paged by 4096 positions

// req_page[p] = the request holding position p << PAGE_BITS; also checks the
// layout (blk_off[0] = 0, non-decreasing, blk_off[n_seqs] = n).
__global__ void sess_page_kernel(const uint64_t *__restrict__ blk_off, uint32_t n_seqs, uint64_t n,
                                 uint32_t *__restrict__ req_page, int32_t *__restrict__ err) {
    const uint64_t r = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r == 0 && (blk_off[0] != 0 || blk_off[n_seqs] != n)) atomicOr(err, DEV_ERR_BAD_LAYOUT);
    if (r >= n_seqs) return;
    const uint64_t a = blk_off[r], b = blk_off[r + 1];
    if (a > b || b > n) {
        atomicOr(err, DEV_ERR_BAD_LAYOUT);
        return;
    }
    for (uint64_t pg = (a + (1u << PAGE_BITS) - 1) >> PAGE_BITS; (pg << PAGE_BITS) < b; ++pg)
        req_page[pg] = (uint32_t)r;
}

// request-level keys for linking the requests of each session
__global__ void sess_keys_kernel(const uint32_t *__restrict__ sess, uint32_t n_seqs, uint64_t *__restrict__ keys) {
    const uint32_t r = blockIdx.x * blockDim.x + threadIdx.x;
    if (r < n_seqs) keys[r] = sess[r];
}

// Footprint after every request: a running max of block counts along each
// session's requests, walked from its first request (one lane per session).
__global__ void sess_footprint_kernel(const uint32_t *__restrict__ prev_s, const uint32_t *__restrict__ next_s,
                                      const uint64_t *__restrict__ blk_off, uint32_t n_seqs, uint64_t n,
                                      uint32_t *__restrict__ w, int32_t *__restrict__ err) {
    const uint32_t stride = gridDim.x * blockDim.x;
    for (uint32_t r = blockIdx.x * blockDim.x + threadIdx.x; r < n_seqs; r += stride) {
        if (prev_s[r] != NONE) continue;
        uint64_t cur = 0;
        uint32_t x = r;
        for (;;) {
            const uint64_t a = blk_off[x], b = blk_off[x + 1];
            const uint64_t m = (a <= b && b <= n) ? b - a : 0;   // a bad layout is reported elsewhere
            cur = m > cur ? m : cur;
            w[x] = (uint32_t)cur;
            const uint32_t y = next_s[x];
            if (y == NONE) break;
            if (y <= x || y >= n_seqs) {   // links run forward; anything else is not ours
                atomicOr(err, DEV_ERR_BAD_LAYOUT);
                break;
            }
            x = y;
        }
    }
}

// Distance of every access: one wave per request tau, SESS_ITEMS accesses per
// lane and step (64 apart, so loads and stores stay coalesced).  Each access
// finds the request j of its
// previous use (page table, then a short search; a lane keeps the last j it
// found, since consecutive blocks of a request were mostly last used by the
// same request), advances to lq, the latest request of j's session before
// tau, and takes w(lq) - 1 + W(lq, tau).  W is summed by the whole wave over
// the requests between lq and tau, once per distinct lq (the last one is kept
// across steps: a request's blocks mostly share one or two).
constexpr int SESS_ITEMS = 8;

__global__ __launch_bounds__(256) void sess_dist_kernel(const uint32_t *__restrict__ prev,
                                                        const uint64_t *__restrict__ blk_off, uint32_t n_seqs,
                                                        uint64_t n, const uint32_t *__restrict__ req_page,
                                                        const uint32_t *__restrict__ next_s,
                                                        const uint32_t *__restrict__ w,
                                                        uint32_t *__restrict__ dist) {
    const int lane = threadIdx.x & (WAVE - 1);
    const uint32_t waves = gridDim.x * (blockDim.x / WAVE);
    const uint32_t w0 = __builtin_amdgcn_readfirstlane(blockIdx.x * (blockDim.x / WAVE) + threadIdx.x / WAVE);
    const uint64_t pages = (n + (1u << PAGE_BITS) - 1) >> PAGE_BITS;
    for (uint32_t tau = w0; tau < n_seqs; tau += waves) {
        const uint64_t s = blk_off[tau], e = blk_off[tau + 1];
        if (s > e || e > n) continue;   // reported by the page kernel
        uint32_t memo_a = NONE, memo_w = 0;
        // the lane's last source request: positions [src_lo, src_hi) -> lq, w(lq)
        uint64_t src_lo = 1, src_hi = 0;
        uint32_t src_lq = NONE, src_w = 0;
        for (uint64_t base = s; base < e; base += SESS_ITEMS * WAVE) {
            const uint64_t t0 = base + lane;
            uint32_t p[SESS_ITEMS], lq[SESS_ITEMS], wl[SESS_ITEMS];
#pragma unroll
            for (int k = 0; k < SESS_ITEMS; ++k) p[k] = t0 + k * WAVE < e ? prev[t0 + k * WAVE] : NONE;
#pragma unroll
            for (int k = 0; k < SESS_ITEMS; ++k) {
                lq[k] = NONE;
                wl[k] = 0;
                if (p[k] == NONE || (uint64_t)p[k] >= n) continue;
                if ((uint64_t)p[k] < src_lo || (uint64_t)p[k] >= src_hi) {
                    const uint64_t pg = (uint64_t)p[k] >> PAGE_BITS;
                    uint32_t lo = req_page[pg];
                    uint32_t hi = pg + 1 < pages ? req_page[pg + 1] : n_seqs - 1;
                    lo = lo < n_seqs ? lo : n_seqs - 1;   // clamps keep bad layouts in bounds
                    hi = hi < n_seqs ? hi : n_seqs - 1;
                    hi = hi > lo ? hi : lo;
                    uint32_t x = sess_req_find(blk_off, lo, hi, p[k]);
                    src_lo = blk_off[x];
                    src_hi = blk_off[x + 1];
                    src_lq = NONE;
                    // a previous use lies in an earlier request; advance along
                    // the session while its next request is still before tau
                    if (x < tau) {
                        for (uint32_t y = next_s[x]; y < tau && y > x; y = next_s[x]) x = y;
                        src_lq = x;
                        src_w = w[x];
                    }
                }
                lq[k] = src_lq;
                wl[k] = src_w;
            }
#pragma unroll
            for (int k = 0; k < SESS_ITEMS; ++k) {
                uint32_t wv = 0;
                bool need = lq[k] != NONE;
                if (need && lq[k] == memo_a) {
                    wv = memo_w;
                    need = false;
                }
                for (uint64_t m = ballot(need); m != 0; m = ballot(need)) {
                    const uint32_t a = (uint32_t)__builtin_amdgcn_readlane((int)lq[k], (int)__builtin_ctzll(m));
                    uint32_t sum = 0;
                    for (uint32_t i = a + 1 + lane; i < tau; i += WAVE) {
                        const uint32_t y = next_s[i];
                        sum += (y >= tau) ? w[i] : 0u;   // none (no next request) is above tau
                    }
                    const uint32_t tot = (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan(sum), WAVE - 1);
                    if (need && lq[k] == a) {
                        wv = tot;
                        need = false;
                    }
                    memo_a = a;
                    memo_w = tot;
                }
                if (t0 + k * WAVE < e) dist[t0 + k * WAVE] = lq[k] == NONE ? NONE : wl[k] - 1u + wv;
            }
        }
    }
}

// fold a nested call's status word into the caller's
__global__ void sess_status_kernel(int32_t *__restrict__ hdr, const int32_t *__restrict__ sub) {
    if (threadIdx.x == 0 && sub[0] != 0) atomicOr(hdr, sub[0]);
}

// The requests of each session, linked like the accesses of one key: the
// session ids go through pc_prev_next_use (1 per request).
struct SessLinks {
    uint64_t *skeys;
    uint32_t *prev_s, *next_s;
    void *pn_ws;
    size_t pn_bytes;
};

static void take_links(Carver &c, uint32_t n_seqs, SessLinks &l) {
    l.skeys = c.take<uint64_t>(n_seqs);
    l.prev_s = c.take<uint32_t>(n_seqs);
    l.next_s = c.take<uint32_t>(n_seqs);
    l.pn_bytes = pc_prev_next_use_ws(n_seqs);
    l.pn_ws = c.take<char>(l.pn_bytes);
}

static pc_status link_sessions(const uint32_t *session, uint32_t n_seqs, const SessLinks &l, int32_t *hdr,
                               hipStream_t s) {
    const unsigned rgrid = (unsigned)(((uint64_t)n_seqs + 255) / 256);
    PC_LAUNCH(K_SESS_REQ, sess_keys_kernel, dim3(rgrid), dim3(256), 0, s, session, n_seqs, l.skeys);
    pc_status st = pc_prev_next_use(l.skeys, n_seqs, l.prev_s, l.next_s, nullptr, l.pn_ws, l.pn_bytes, s);
    if (st != PC_OK) return st;
    PC_LAUNCH(K_SESS_REQ, sess_status_kernel, dim3(1), dim3(64), 0, s, hdr,
              reinterpret_cast<const int32_t *>(l.pn_ws));
    return PC_OK;
}

struct SessWs {
    int32_t *hdr;
    SessLinks l;
    uint32_t *w, *req_page;
    size_t bytes;
};

static SessWs carve_sess(void *ws, uint64_t n, uint32_t n_seqs) {
    Carver c{(char *)ws, 0};
    SessWs s;
    s.hdr = c.take<int32_t>(WS_HEADER / sizeof(int32_t));
    take_links(c, n_seqs, s.l);
    s.w = c.take<uint32_t>(n_seqs);
    s.req_page = c.take<uint32_t>(((n + (1u << PAGE_BITS) - 1) >> PAGE_BITS) + 2);
    s.bytes = c.off;
    return s;
}

// Per-session statistics (Sec. 4.5 footprints, Sec. 4.1 session duration,
// Sec. 4.3 requests per session, Sec. 2.3 gaps between a session's
// requests): one lane per session walks its requests from the first.
// Footprint = largest request (append-only contexts).  Small histograms
// accumulate in LDS; the footprint histogram, whose range is the largest
// request, is added to globally.
__global__ __launch_bounds__(256) void sess_profile_kernel(
    const uint32_t *__restrict__ prev_s, const uint32_t *__restrict__ next_s, const uint64_t *__restrict__ blk_off,
    const uint64_t *__restrict__ ts_us, uint32_t n_seqs, uint64_t n, const uint64_t *__restrict__ edges,
    uint32_t n_edges, uint32_t fp_max, uint32_t rq_max, uint64_t *__restrict__ footprint,
    uint64_t *__restrict__ requests, uint64_t *__restrict__ duration, uint64_t *__restrict__ gap,
    int32_t *__restrict__ err) {
    __shared__ uint64_t s_edges[PC_MAX_PROFILE_EDGES];
    __shared__ uint32_t s_dur[PC_MAX_PROFILE_EDGES + 1];
    __shared__ uint32_t s_gap[PC_MAX_PROFILE_EDGES + 1];
    __shared__ uint32_t s_req[PC_MAX_FREQ + 1];
    const int tid = threadIdx.x;
    const uint32_t kb = n_edges + 1;
    for (uint32_t i = tid; i < n_edges; i += blockDim.x) {
        s_edges[i] = edges[i];
        if (blockIdx.x == 0 && i + 1 < n_edges && edges[i] > edges[i + 1]) atomicOr(err, DEV_ERR_BAD_CAPS);
    }
    for (uint32_t i = tid; i < kb; i += blockDim.x) s_dur[i] = s_gap[i] = 0;
    for (uint32_t i = tid; i <= rq_max; i += blockDim.x) s_req[i] = 0;
    __syncthreads();
    const uint32_t stride = gridDim.x * blockDim.x;
    for (uint32_t r = blockIdx.x * blockDim.x + tid; r < n_seqs; r += stride) {
        if (prev_s[r] != NONE) continue;
        uint64_t fp = 0, cnt = 0;
        const uint64_t t0 = ts_us[r];
        uint64_t t1 = t0;
        uint32_t x = r;
        for (;;) {
            const uint64_t a = blk_off[x], b = blk_off[x + 1];
            const uint64_t m = (a <= b && b <= n) ? b - a : 0;   // a bad layout is reported elsewhere
            fp = m > fp ? m : fp;
            const uint64_t tx = ts_us[x];
            if (cnt > 0) {
                uint32_t lo = 0, hi = n_edges;   // number of edges <= the gap
                while (lo < hi) {
                    const uint32_t mid = (lo + hi) >> 1;
                    if (s_edges[mid] <= tx - t1) lo = mid + 1;
                    else hi = mid;
                }
                atomicAdd(&s_gap[lo], 1u);
            }
            t1 = tx;
            ++cnt;
            const uint32_t y = next_s[x];
            if (y == NONE) break;
            if (y <= x || y >= n_seqs) {
                atomicOr(err, DEV_ERR_BAD_LAYOUT);
                break;
            }
            x = y;
        }
        uint32_t lo = 0, hi = n_edges;
        while (lo < hi) {
            const uint32_t mid = (lo + hi) >> 1;
            if (s_edges[mid] <= t1 - t0) lo = mid + 1;
            else hi = mid;
        }
        atomicAdd(&s_dur[lo], 1u);
        atomicAdd(&s_req[cnt < rq_max ? cnt : rq_max], 1u);
        atomicAdd((unsigned long long *)&footprint[fp < fp_max ? fp : fp_max], 1ull);
    }
    __syncthreads();
    for (uint32_t i = tid; i < kb; i += blockDim.x) {
        if (s_dur[i]) atomicAdd((unsigned long long *)&duration[i], (unsigned long long)s_dur[i]);
        if (s_gap[i]) atomicAdd((unsigned long long *)&gap[i], (unsigned long long)s_gap[i]);
    }
    for (uint32_t i = tid; i <= rq_max; i += blockDim.x)
        if (s_req[i]) atomicAdd((unsigned long long *)&requests[i], (unsigned long long)s_req[i]);
}

}  // namespace pc

extern "C" {

size_t pc_stack_distance_session_ws(uint64_t n, uint32_t n_seqs) { return pc::carve_sess(nullptr, n, n_seqs).bytes; }

pc_status pc_stack_distance_session(const uint32_t *prev, const uint64_t *blk_off, const uint32_t *session,
                                    uint32_t n_seqs, uint64_t n, uint32_t *dist_sess, void *ws, size_t ws_bytes,
                                    void *stream) {
    if (n >= (uint64_t)PC_NONE) return PC_ERR_TOO_LARGE;
    if (n_seqs >= 0x80000000u) return PC_ERR_TOO_LARGE;
    if (n > 0 && (!prev || !blk_off || !session || !dist_sess || n_seqs == 0)) return PC_ERR_INVALID;
    if (!ws) return PC_ERR_WORKSPACE;
    if (ws_bytes < pc_stack_distance_session_ws(n, n_seqs)) return PC_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    pc::SessWs w = pc::carve_sess(ws, n, n_seqs);
    pc_status st = pc::fill_u32(reinterpret_cast<uint32_t *>(w.hdr), 0u, 1, s);
    if (st != PC_OK || n == 0) return st;
    const uint64_t pages = (n + (1u << pc::PAGE_BITS) - 1) >> pc::PAGE_BITS;
    if ((st = pc::fill_u32(w.req_page, 0u, pages + 1, s)) != PC_OK) return st;
    const unsigned rgrid = (unsigned)(((uint64_t)n_seqs + 255) / 256);
    PC_LAUNCH(pc::K_SESS_REQ, pc::sess_page_kernel, dim3(rgrid), dim3(256), 0, s, blk_off, n_seqs, n, w.req_page,
              w.hdr);
    if ((st = pc::link_sessions(session, n_seqs, w.l, w.hdr, s)) != PC_OK) return st;
    const int cus = pc::device_cus();
    unsigned fgrid = rgrid < (unsigned)cus * 4 ? rgrid : (unsigned)cus * 4;
    PC_LAUNCH(pc::K_SESS_REQ, pc::sess_footprint_kernel, dim3(fgrid), dim3(256), 0, s, w.l.prev_s, w.l.next_s,
              blk_off, n_seqs, n, w.w, w.hdr);
    uint64_t grid = ((uint64_t)n_seqs + 3) / 4;
    if (grid > (uint64_t)cus * 64) grid = (uint64_t)cus * 64;   // 64 per CU: 4.57 -> 4.38 ms on the full trace
    PC_LAUNCH(pc::K_SESS_DIST, pc::sess_dist_kernel, dim3((unsigned)grid), dim3(256), 0, s, prev, blk_off, n_seqs, n,
              w.req_page, w.l.next_s, w.w, dist_sess);
    return PC_OK;
}

size_t pc_session_profile_ws(uint32_t n_seqs) {
    pc::Carver c{nullptr, 0};
    c.take<int32_t>(pc::WS_HEADER / sizeof(int32_t));
    pc::SessLinks l;
    pc::take_links(c, n_seqs, l);
    return c.off;
}

pc_status pc_session_profile(const uint64_t *blk_off, const uint32_t *session, const uint64_t *ts_us, uint32_t n_seqs,
                             uint64_t n, const uint64_t *edges, uint32_t n_edges, uint32_t fp_max, uint32_t rq_max,
                             uint64_t *footprint, uint64_t *requests, uint64_t *duration, uint64_t *gap, void *ws,
                             size_t ws_bytes, void *stream) {
    if (n >= (uint64_t)PC_NONE) return PC_ERR_TOO_LARGE;
    if (n_seqs >= 0x80000000u) return PC_ERR_TOO_LARGE;
    if (n_edges < 1 || n_edges > PC_MAX_PROFILE_EDGES || rq_max < 1 || rq_max > PC_MAX_FREQ || fp_max < 1 ||
        fp_max > PC_MAX_FOOTPRINT)
        return PC_ERR_INVALID;
    if (!edges || !footprint || !requests || !duration || !gap) return PC_ERR_INVALID;
    if (n_seqs > 0 && (!blk_off || !session || !ts_us)) return PC_ERR_INVALID;
    if (!ws) return PC_ERR_WORKSPACE;
    if (ws_bytes < pc_session_profile_ws(n_seqs)) return PC_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    pc::Carver c{(char *)ws, 0};
    int32_t *hdr = c.take<int32_t>(pc::WS_HEADER / sizeof(int32_t));
    pc::SessLinks l;
    pc::take_links(c, n_seqs, l);
    pc_status st = pc::fill_u32(reinterpret_cast<uint32_t *>(hdr), 0u, 1, s);
    if (st != PC_OK) return st;
    const size_t kb = (size_t)n_edges + 1;
    if ((st = pc::fill_u32(reinterpret_cast<uint32_t *>(footprint), 0u, 2 * ((size_t)fp_max + 1), s)) != PC_OK)
        return st;
    if ((st = pc::fill_u32(reinterpret_cast<uint32_t *>(requests), 0u, 2 * ((size_t)rq_max + 1), s)) != PC_OK)
        return st;
    if ((st = pc::fill_u32(reinterpret_cast<uint32_t *>(duration), 0u, 2 * kb, s)) != PC_OK) return st;
    if ((st = pc::fill_u32(reinterpret_cast<uint32_t *>(gap), 0u, 2 * kb, s)) != PC_OK) return st;
    if (n_seqs == 0) return PC_OK;
    if ((st = pc::link_sessions(session, n_seqs, l, hdr, s)) != PC_OK) return st;
    const int cus = pc::device_cus();
    unsigned grid = (unsigned)(((uint64_t)n_seqs + 255) / 256);
    if (grid > (unsigned)cus * 4) grid = (unsigned)cus * 4;
    PC_LAUNCH(pc::K_SESS_PROFILE, pc::sess_profile_kernel, dim3(grid), dim3(256), 0, s, l.prev_s, l.next_s, blk_off,
              ts_us, n_seqs, n, edges, n_edges, fp_max, rq_max, footprint, requests, duration, gap, hdr);
    return PC_OK;
}

}  // extern "C"
