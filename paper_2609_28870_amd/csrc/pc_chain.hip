// Previous / next use of every access from the chain structure of the keys
// (pc_prev_next_chained).  Same outputs as pc_prev_next_use.
//
// A block key is chained over the whole token prefix (Sec. 2.2: a cached
// block is reusable only when everything before it matches), so an access
// at depth d of request r and one at depth d of request c carry the same key
// exactly when the two requests agree on their first d + 1 blocks (up to
// hash collisions, which the checks below catch).  Hence the latest earlier
// request sharing r's block at depth d is a step function of d that changes
// only where r leaves one earlier request's prefix: a request's reuse links
// come in long runs to very few earlier requests.
//
// GPU mapping, S = 64 = one wave of depths:
//   1. anchors: the key at every depth a*S of every request goes to slot
//      base(r) + a, base(r) = floor(blk_off[r] / S) + r (slots of different
//      requests never overlap; the one or two slots between requests hold a
//      filler key), and the generic prev/next runs over the slots
//      (~n/64 + n_seqs keys);
//   2. staircase: one wave per slot (r, a) takes the request c of the
//      anchor's previous use; lanes d = a*S .. a*S+63 compare r's and c's
//      keys and every lane before the first mismatch links to c at depth d,
//      writing the prev link at r and the mirrored next link at c (anchor
//      links are one-to-one, so each slot has at most one such claimant,
//      which also records the lanes it linked in the slot's claimed mask);
//   3. every access left without a prev or a next link (first and last
//      occurrences, and the lanes after a change of request inside a wave)
//      is compacted in time order and the generic prev/next runs over them;
//      the merge writes its links back, checking that a link it adds never
//      ends at an access that already has a staircase link on that side.
// Exactness: staircase links join equal keys at an earlier position and are
// one-to-one (anchor links are); merged links join consecutive compacted
// accesses with equal keys; the merge check makes prev one-to-one overall;
// every access without a prev went through the compacted prev/next, so no
// two of them share a key.  A one-to-one prev map whose links join equal keys
// and that has one start per key orders each key's accesses into one chain,
// i.e. it is the exact prev (and next its inverse).  If the check fails, the
// block layout is invalid, or too many accesses stay unresolved, the generic
// prev/next runs over all keys instead.  Both ways the outputs are exact.
#include "pc_internal.h"

namespace pc {

constexpr uint32_t UNK = 0xFFFFFFFEu;    // "no staircase link" (never a position: n < 2^32 - 1)
constexpr int CH_S = 64;                 // depths per anchor = lanes per wave
constexpr int CH_THREADS = 256;
constexpr int SCAN_THREADS = 1024;
constexpr int SCAN_ITEMS = 4;
constexpr int SCAN_TILE = SCAN_THREADS * SCAN_ITEMS;
constexpr uint64_t FILLER_KEY = 0xA5A5A5A5A5A5A5A5ull;

// header words of the chained workspace
constexpr int HW_STATUS = 0;
constexpr int HW_PATH = 1;       // 0 = chain path verified, 1 = generic over all keys
constexpr int HW_UNRESOLVED = 2; // accesses that went through the compacted prev/next
constexpr int HW_REASON = 3;     // why the generic path ran: 1 layout, 2 too many unresolved, 3 check, 4 nested error
constexpr int HW_BAD = 4;        // device flag: invalid block layout
constexpr int HW_FAIL = 5;       // device flag: a merge check failed
constexpr int HW_HIGH_ANCHOR = 6;     // the prev/next over the anchors also sorted by the high key bits
constexpr int HW_HIGH_UNRESOLVED = 7; // the prev/next over the unresolved accesses did
constexpr int HW_CHAIN = 8;      // gate: 1 while the chain path goes on
constexpr int HW_WORDS = 16;     // header words cleared by each call

__device__ __forceinline__ int wave_id_uniform() {
    return __builtin_amdgcn_readfirstlane((int)(threadIdx.x / WAVE));
}

// Per slot, written with the anchor keys: the anchor's position, the number
// of depths the slot covers (0 for a filler slot) and the anchor depth
// (NONE for a filler).  Depth a*S + lane sits at pos + lane, or pos - lane in
// the deepest-first layout.
struct Slot {
    uint64_t pos;
    uint32_t lanes, depth;
};
__device__ __forceinline__ Slot load_slot(const uint4 *__restrict__ rec, uint64_t j) {
    const uint4 v = rec[j];
    return Slot{(uint64_t)v.x | ((uint64_t)v.y << 32), v.z, v.w};
}
__device__ __forceinline__ uint64_t lane_pos(const Slot &q, int lane, int deepest) {
    return deepest ? q.pos - (uint64_t)lane : q.pos + (uint64_t)lane;
}

// Every request: blk_off[r] <= blk_off[r+1], blk_off[0] = 0, blk_off[R] = n.
__global__ void chain_layout_kernel(const uint64_t *__restrict__ off, uint32_t n_seqs, uint64_t n,
                                    int32_t *__restrict__ hdr) {
    const uint64_t r = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= n_seqs) return;
    const uint64_t a = off[r], b = off[r + 1];
    bool ok = a <= b && b <= n;
    if (r == 0) ok = ok && a == 0;
    if (r + 1 == n_seqs) ok = ok && b == n;
    if (!ok) {
        atomicOr(hdr + HW_BAD, 1);
        atomicOr(hdr + HW_STATUS, DEV_ERR_BAD_LAYOUT);
    }
}

// One wave per request: the request's anchors go to slots
// base(r) .. base(r) + ceil(len / S) - 1, base(r) = floor(blk_off[r] / S) + r,
// in time order (ascending depth, or descending in the deepest-first
// layout); the slots up to the next request's first one get filler keys.
__global__ __launch_bounds__(CH_THREADS) void chain_anchor_kernel(
    const uint64_t *__restrict__ keys, const uint64_t *__restrict__ off, uint32_t n_seqs, uint64_t n_slots,
    int deepest, uint64_t *__restrict__ akeys, uint4 *__restrict__ rec, const int32_t *__restrict__ hdr) {
    if (hdr[HW_BAD]) return;
    const int lane = threadIdx.x & (WAVE - 1);
    const uint64_t waves = (uint64_t)gridDim.x * (CH_THREADS / WAVE);
    for (uint64_t r = (uint64_t)blockIdx.x * (CH_THREADS / WAVE) + wave_id_uniform(); r < n_seqs; r += waves) {
        const uint64_t o0 = off[r], o1 = off[r + 1];
        const uint64_t len = o1 - o0, base = o0 / CH_S + r, n_anchor = (len + CH_S - 1) / CH_S;
        const uint64_t next_base = (r + 1 < n_seqs) ? o1 / CH_S + r + 1 : n_slots;
        for (uint64_t i = lane; base + i < next_base; i += WAVE) {
            const uint64_t j = base + i;
            if (i < n_anchor) {
                const uint64_t d = (deepest ? n_anchor - 1 - i : i) * CH_S;
                const uint64_t p = deepest ? o1 - 1 - d : o0 + d;
                const uint64_t lanes = len - d < (uint64_t)CH_S ? len - d : (uint64_t)CH_S;
                akeys[j] = keys[p];
                rec[j] = make_uint4((uint32_t)p, (uint32_t)(p >> 32), (uint32_t)lanes, (uint32_t)d);
            } else {
                akeys[j] = FILLER_KEY;
                rec[j] = make_uint4(0u, 0u, 0u, NONE);
            }
        }
    }
}

// Slots per wave iteration (BATCH): their loads are issued together so the
// three dependent levels (slot record and anchor links, linked records,
// keys) overlap across slots.  The linked keys are spread over the whole
// trace, and their latency grows with its size: two slots per iteration
// were fastest up to about 3e8 accesses (2.2e8: 0.99 against 1.09 ms with
// sixteen), eight from about 9e8 (4.3 against 5.0 ms with two) and sixteen
// at 2.1e9 (9.8 against 12.5 ms with two, 10.0 with eight).
static int stair_batch(uint64_t n) { return n >= (1ull << 30) ? 16 : n >= (1ull << 29) ? 8 : 2; }

// The prev links of one slot: the lanes before the first depth at which the
// slot's request and the linked anchor's request differ (both must cover
// the depth) link to the linked request at that depth; UNK elsewhere.
__device__ __forceinline__ uint32_t stair_claim(const Slot &q, const Slot &c, uint64_t kr, uint64_t kc, int lane,
                                                int deepest) {
    const bool eq = c.depth == q.depth && lane < (int)q.lanes && lane < (int)c.lanes && kc == kr;
    const uint64_t m = ballot(eq);
    const int lead = (~m == 0) ? WAVE : __builtin_ctzll(~m);
    return lane < lead ? (uint32_t)lane_pos(c, lane, deepest) : UNK;
}

// One wave per slot: the prev links of the slot's depths and their mirrored
// next links, the lanes left without a prev link (open[j].xy), and the
// lanes the linked slot got a next link for (claimed[link]).  A link to a
// filler slot or to an anchor at another depth (equal keys there are a
// collision) claims nothing.
template <int CH_BATCH>
__global__ __launch_bounds__(CH_THREADS) void chain_stair_kernel(
    const uint64_t *__restrict__ keys, uint64_t n_slots, const uint4 *__restrict__ rec,
    const uint32_t *__restrict__ aprev, int deepest, uint32_t *__restrict__ prev, uint32_t *__restrict__ next,
    int want_next, uint4 *__restrict__ open, uint2 *__restrict__ claimed, const int32_t *__restrict__ hdr) {
    if (hdr[HW_BAD]) return;
    const int lane = threadIdx.x & (WAVE - 1);
    const uint64_t waves = (uint64_t)gridDim.x * (CH_THREADS / WAVE);
    const Slot none{0, 0, NONE};
    for (uint64_t j0 = ((uint64_t)blockIdx.x * (CH_THREADS / WAVE) + wave_id_uniform()) * CH_BATCH; j0 < n_slots;
         j0 += waves * CH_BATCH) {
        Slot q[CH_BATCH], cp[CH_BATCH];
        uint32_t lp[CH_BATCH];
#pragma unroll
        for (int k = 0; k < CH_BATCH; ++k) {
            const bool in = j0 + k < n_slots;
            q[k] = in ? load_slot(rec, j0 + k) : none;
            lp[k] = in ? aprev[j0 + k] : NONE;
        }
#pragma unroll
        for (int k = 0; k < CH_BATCH; ++k) cp[k] = lp[k] != NONE ? load_slot(rec, lp[k]) : none;
        uint64_t kr[CH_BATCH], kp[CH_BATCH];
#pragma unroll
        for (int k = 0; k < CH_BATCH; ++k) {
            const bool v = lane < (int)q[k].lanes;
            kr[k] = v ? keys[lane_pos(q[k], lane, deepest)] : 0;
            kp[k] = v && cp[k].depth == q[k].depth && lane < (int)cp[k].lanes ? keys[lane_pos(cp[k], lane, deepest)]
                                                                              : ~kr[k];
        }
#pragma unroll
        for (int k = 0; k < CH_BATCH; ++k) {
            if (j0 + k >= n_slots) break;
            const bool v = lane < (int)q[k].lanes;
            const uint32_t p = stair_claim(q[k], cp[k], kr[k], kp[k], lane, deepest);
            const uint64_t pr = lane_pos(q[k], lane, deepest);
            if (v) prev[pr] = p;
            if (want_next && p != UNK) next[p] = (uint32_t)pr;
            const uint64_t mp = ballot(v && p == UNK), mc = ballot(p != UNK);
            if (lane == 0) {
                open[j0 + k] = make_uint4((uint32_t)mp, (uint32_t)(mp >> 32), 0u, 0u);
                if (lp[k] != NONE) claimed[lp[k]] = make_uint2((uint32_t)mc, (uint32_t)(mc >> 32));
            }
        }
    }
}

// Per slot: the lanes without a next link (valid and not claimed), into
// open[j].zw, and the count of lanes open on either side.
__global__ __launch_bounds__(256) void chain_count_kernel(uint64_t n_slots, const uint4 *__restrict__ rec,
                                                          const uint2 *__restrict__ claimed, uint4 *__restrict__ open,
                                                          uint32_t *__restrict__ cnt, const int32_t *__restrict__ hdr) {
    if (hdr[HW_BAD]) return;
    const uint64_t j = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= n_slots) return;
    const uint32_t lanes = rec[j].z;
    const uint64_t valid = lanes >= (uint32_t)WAVE ? ~0ull : (1ull << lanes) - 1;
    const uint2 c = claimed[j];
    const uint64_t mx = valid & ~((uint64_t)c.x | ((uint64_t)c.y << 32));
    const uint4 o = open[j];
    const uint64_t mp = (uint64_t)o.x | ((uint64_t)o.y << 32);
    open[j] = make_uint4(o.x, o.y, (uint32_t)mx, (uint32_t)(mx >> 32));
    cnt[j] = (uint32_t)__popcll(mp | mx);
}

// Exclusive scan of cnt[0 .. m) into out[0 .. m], out[m] = total: tile sums,
// one workgroup over the tile sums, then each tile again with its base.
__global__ __launch_bounds__(SCAN_THREADS) void chain_scan_tiles_kernel(const uint32_t *__restrict__ cnt,
                                                                        uint64_t m, uint32_t *__restrict__ tsum,
                                                                        const int32_t *__restrict__ hdr) {
    if (hdr[HW_BAD]) return;
    __shared__ uint32_t tmp[SCAN_THREADS / WAVE];
    const uint64_t t0 = (uint64_t)blockIdx.x * SCAN_TILE;
    uint32_t s = 0;
#pragma unroll
    for (int k = 0; k < SCAN_ITEMS; ++k) {
        const uint64_t i = t0 + (uint64_t)k * SCAN_THREADS + threadIdx.x;
        if (i < m) s += cnt[i];
    }
    uint32_t total = 0;
    block_excl_scan(s, tmp, &total);
    if (threadIdx.x == 0) tsum[blockIdx.x] = total;
}

__global__ __launch_bounds__(SCAN_THREADS) void chain_scan_top_kernel(uint32_t *__restrict__ tsum, uint64_t tiles,
                                                                      int32_t *__restrict__ hdr) {
    if (hdr[HW_BAD]) return;
    __shared__ uint32_t tmp[SCAN_THREADS / WAVE];
    uint32_t carry = 0;
    for (uint64_t t0 = 0; t0 < tiles; t0 += SCAN_THREADS) {
        const uint64_t i = t0 + threadIdx.x;
        const uint32_t v = i < tiles ? tsum[i] : 0;
        uint32_t total = 0;
        const uint32_t e = block_excl_scan(v, tmp, &total);
        if (i < tiles) tsum[i] = carry + e;
        carry += total;
    }
    if (threadIdx.x == 0) hdr[HW_UNRESOLVED] = (int32_t)carry;
}

__global__ __launch_bounds__(SCAN_THREADS) void chain_scan_apply_kernel(const uint32_t *__restrict__ cnt, uint64_t m,
                                                                        const uint32_t *__restrict__ tsum,
                                                                        uint32_t *__restrict__ out,
                                                                        const int32_t *__restrict__ hdr) {
    if (hdr[HW_BAD]) return;
    __shared__ uint32_t tmp[SCAN_THREADS / WAVE];
    // each thread scans SCAN_ITEMS consecutive entries
    const uint64_t i0 = (uint64_t)blockIdx.x * SCAN_TILE + (uint64_t)threadIdx.x * SCAN_ITEMS;
    uint32_t v[SCAN_ITEMS], s = 0;
#pragma unroll
    for (int k = 0; k < SCAN_ITEMS; ++k) {
        v[k] = (i0 + k < m) ? cnt[i0 + k] : 0;
        s += v[k];
    }
    uint32_t total = 0;
    uint32_t run = tsum[blockIdx.x] + block_excl_scan(s, tmp, &total);
#pragma unroll
    for (int k = 0; k < SCAN_ITEMS; ++k) {
        if (i0 + k < m) out[i0 + k] = run;
        run += v[k];
    }
    if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) out[m] = (uint32_t)hdr[HW_UNRESOLVED];
}

// The unresolved accesses, in time order, into (key, position, which sides
// are open), from the stair kernel's lane masks.  Most slots have no open
// lane (a request that continues an earlier one links all its depths but
// the last few), so a wave first reads 64 slots' masks, offsets and records,
// one per lane, and then takes only the slots with open lanes, two at a
// time, one lane per depth.
__global__ __launch_bounds__(CH_THREADS) void chain_compact_kernel(
    const uint64_t *__restrict__ keys, uint64_t n_slots, const uint4 *__restrict__ rec,
    const uint4 *__restrict__ open, const uint32_t *__restrict__ coff, int deepest,
    uint64_t *__restrict__ ckeys, uint32_t *__restrict__ cpos, uint8_t *__restrict__ cflag,
    const int32_t *__restrict__ hdr) {
    if (!hdr[HW_CHAIN]) return;   // (so the offsets stay below the unresolved capacity)
    const int lane = threadIdx.x & (WAVE - 1);
    const uint64_t waves = (uint64_t)gridDim.x * (CH_THREADS / WAVE);
    const uint64_t bit = 1ull << lane;
    const uint64_t above = ~((2ull << lane) - 1);   // lanes above this one (none for lane 63)
    for (uint64_t j0 = ((uint64_t)blockIdx.x * (CH_THREADS / WAVE) + wave_id_uniform()) * WAVE; j0 < n_slots;
         j0 += waves * WAVE) {
        const uint64_t j = j0 + lane;
        uint64_t mp = 0, mx = 0, pos = 0;
        uint32_t base = 0;
        if (j < n_slots) {
            const uint4 o = open[j];
            mp = (uint64_t)o.x | ((uint64_t)o.y << 32);
            mx = (uint64_t)o.z | ((uint64_t)o.w << 32);
            if (mp | mx) {
                pos = load_slot(rec, j).pos;
                base = coff[j];
            }
        }
        uint64_t todo = ballot((mp | mx) != 0);
        while (todo) {
            int src[2];
            src[0] = __builtin_ctzll(todo);
            todo &= todo - 1;
            src[1] = todo ? __builtin_ctzll(todo) : -1;
            if (todo) todo &= todo - 1;
            uint64_t m[2], p[2], kk[2];
            uint32_t b[2], f[2];
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                const int L = src[k] < 0 ? src[0] : src[k];
                const uint64_t a = shfl64(mp, L), x = shfl64(mx, L);
                m[k] = src[k] < 0 ? 0ull : (a | x);
                f[k] = (a & bit ? 1u : 0u) | (x & bit ? 2u : 0u);
                const uint64_t ps = shfl64(pos, L);
                p[k] = deepest ? ps - (uint64_t)lane : ps + (uint64_t)lane;
                b[k] = (uint32_t)__shfl((int)base, L, WAVE);
                kk[k] = (m[k] & bit) ? keys[p[k]] : 0ull;
            }
#pragma unroll
            for (int k = 0; k < 2; ++k) {
                if (m[k] & bit) {
                    // time order: lanes ascending, or descending in the deepest-first layout
                    const uint32_t rank = deepest ? (uint32_t)__popcll(m[k] & above) : mbcnt(m[k]);
                    const uint64_t o = (uint64_t)b[k] + rank;
                    ckeys[o] = kk[k];
                    cpos[o] = (uint32_t)p[k];
                    cflag[o] = (uint8_t)f[k];
                }
            }
        }
    }
}

// Links of the compacted accesses back into prev / next; flags an added link
// that would end at an access whose own side is already linked.  The number
// of compacted accesses is the one the scan wrote.
__global__ __launch_bounds__(CH_THREADS) void chain_merge_kernel(const uint32_t *__restrict__ cpos,
                                                                 const uint8_t *__restrict__ cflag,
                                                                 const uint32_t *__restrict__ cprev,
                                                                 const uint32_t *__restrict__ cnext,
                                                                 uint32_t *__restrict__ prev,
                                                                 uint32_t *__restrict__ next, int want_next,
                                                                 int32_t *__restrict__ hdr) {
    if (!hdr[HW_CHAIN]) return;
    const uint64_t m = (uint32_t)hdr[HW_UNRESOLVED];
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    bool bad = false;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < m; i += stride) {
        const uint32_t f = cflag[i];
        const uint32_t p = cpos[i];
        if (f & 1) {
            const uint32_t t = cprev[i];
            if (t != NONE) {
                bad |= !(cflag[t] & 2);
                prev[p] = cpos[t];
            } else {
                prev[p] = NONE;
            }
        }
        if (f & 2) {
            const uint32_t u = cnext[i];
            if (u != NONE) bad |= !(cflag[u] & 1);
            if (want_next) next[p] = u != NONE ? cpos[u] : NONE;
        }
    }
    if (bad) atomicOr(hdr + HW_FAIL, 1);
}

// an inner prev/next call's header: its status into ours (word 0), its
// high-bit flag (word 1) into word `high_word` of ours; only when the inner
// call ran (gate word of ours non-zero)
__global__ void chain_status_kernel(const int32_t *__restrict__ nested, int32_t *__restrict__ hdr, int high_word,
                                    int gate_word) {
    if (threadIdx.x != 0 || !hdr[gate_word]) return;
    if (nested[0]) atomicOr(hdr + HW_STATUS, nested[0]);
    hdr[high_word] = nested[1];
}

// After the layout check: the chain path starts if the layout is valid.
__global__ void chain_open_kernel(int32_t *__restrict__ hdr) {
    if (threadIdx.x == 0) hdr[HW_CHAIN] = hdr[HW_BAD] ? 0 : 1;
}

// After the unresolved count: the chain path goes on if the layout is valid,
// the anchors' prev/next reported no error and the unresolved accesses fit
// the workspace; otherwise the reason is recorded.
__global__ void chain_decide_kernel(int32_t *__restrict__ hdr, const int32_t *__restrict__ anchor_hdr,
                                    uint32_t m_cap) {
    if (threadIdx.x != 0) return;
    int32_t reason = 0;
    if (hdr[HW_BAD]) reason = 1;
    else if (anchor_hdr[0]) reason = 4;
    else if ((uint32_t)hdr[HW_UNRESOLVED] > m_cap) reason = 2;
    hdr[HW_REASON] = reason;
    hdr[HW_CHAIN] = reason == 0 ? 1 : 0;
}

// After the merge: the generic prev/next over all keys runs (HW_PATH = 1)
// if the chain path stopped, the inner prev/next reported an error or the
// merge check failed.
__global__ void chain_verdict_kernel(int32_t *__restrict__ hdr, const int32_t *__restrict__ inner_hdr) {
    if (threadIdx.x != 0) return;
    int32_t reason = hdr[HW_REASON];
    if (reason == 0 && inner_hdr[0]) reason = 4;
    if (reason == 0 && hdr[HW_FAIL]) reason = 3;
    hdr[HW_REASON] = reason;
    hdr[HW_PATH] = reason != 0 ? 1 : 0;
}

struct ChainWs {
    int32_t *hdr;
    void *generic;        // pc_prev_next_use workspace over all keys (also the unresolved stage's space)
    size_t generic_bytes;
    uint64_t *akeys;
    uint4 *rec;
    uint4 *open;
    uint2 *claimed;
    uint32_t *aprev, *anext, *cnt, *coff, *tsum;
    void *aws;            // pc_prev_next_use workspace over the slots
    size_t aws_bytes;
    size_t bytes;
};

static uint64_t chain_slots(uint64_t n, uint32_t n_seqs) { return n / CH_S + n_seqs + 1; }

static ChainWs carve_chain(void *ws, uint64_t n, uint32_t n_seqs) {
    Carver c{(char *)ws, 0};
    ChainWs w;
    const uint64_t ns = chain_slots(n, n_seqs);
    w.hdr = c.take<int32_t>(WS_HEADER / sizeof(int32_t));
    w.generic_bytes = pc_prev_next_use_ws(n);
    w.generic = c.take<char>(w.generic_bytes);
    w.akeys = c.take<uint64_t>(ns);
    w.rec = c.take<uint4>(ns);
    w.open = c.take<uint4>(ns);
    w.claimed = c.take<uint2>(ns);
    w.aprev = c.take<uint32_t>(ns);
    w.anext = c.take<uint32_t>(ns);
    w.cnt = c.take<uint32_t>(ns);
    w.coff = c.take<uint32_t>(ns + 1);
    w.tsum = c.take<uint32_t>((ns + SCAN_TILE - 1) / SCAN_TILE + 1);
    w.aws_bytes = pc_prev_next_use_ws(ns);
    w.aws = c.take<char>(w.aws_bytes);
    w.bytes = c.off;
    return w;
}

// The unresolved stage's arrays inside the generic workspace (unused until a
// fallback); false if they do not fit.
struct OpenWs {
    uint64_t *ckeys;
    uint32_t *cpos, *cprev, *cnext;
    uint8_t *cflag;
    void *ws;
    size_t ws_bytes;
};
static size_t carve_open(void *base, uint64_t m, OpenWs *o) {
    Carver c{(char *)base, 0};
    o->ckeys = c.take<uint64_t>(m);
    o->cpos = c.take<uint32_t>(m);
    o->cprev = c.take<uint32_t>(m);
    o->cnext = c.take<uint32_t>(m);
    o->cflag = c.take<uint8_t>(m);
    o->ws_bytes = pc_prev_next_use_ws(m);
    o->ws = c.take<char>(o->ws_bytes);
    return c.off;
}

// the most unresolved accesses the generic workspace holds (at most n)
static uint64_t open_capacity(const ChainWs &w, uint64_t n) {
    OpenWs o;
    uint64_t lo = 0, hi = n;
    while (lo < hi) {
        const uint64_t mid = lo + (hi - lo + 1) / 2;
        if (carve_open(nullptr, mid, &o) <= w.generic_bytes) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

static unsigned wave_grid(uint64_t items, int cus) {
    uint64_t g = (items + CH_THREADS / WAVE - 1) / (CH_THREADS / WAVE);
    const uint64_t cap = (uint64_t)cus * 128;
    if (g > cap) g = cap;
    return (unsigned)(g ? g : 1);
}

}  // namespace pc

extern "C" {

size_t pc_prev_next_chained_ws(uint64_t n, uint32_t n_seqs) { return pc::carve_chain(nullptr, n, n_seqs).bytes; }

pc_status pc_prev_next_chained(const uint64_t *keys, uint64_t n, const uint64_t *blk_off, uint32_t n_seqs,
                               uint32_t flags, uint32_t *prev, uint32_t *next, const uint32_t *key_hist,
                               void *ws, size_t ws_bytes, void *stream) {
    using namespace pc;
    if (n >= (uint64_t)PC_NONE) return PC_ERR_TOO_LARGE;
    if (n > 0 && (!keys || !prev || !next || !blk_off)) return PC_ERR_INVALID;
    if (flags & ~(PC_HASH_DEEPEST_FIRST | PC_PREV_ONLY)) return PC_ERR_INVALID;
    if (!ws) return PC_ERR_WORKSPACE;
    if (ws_bytes < pc_prev_next_chained_ws(n, n_seqs)) return PC_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    const ChainWs w = carve_chain(ws, n, n_seqs);
    pc_status st = fill_u32(reinterpret_cast<uint32_t *>(w.hdr), 0u, HW_WORDS, s);
    if (st != PC_OK || n == 0) return st;
    const int deepest = (flags & PC_HASH_DEEPEST_FIRST) ? 1 : 0;
    const int want_next = (flags & PC_PREV_ONLY) ? 0 : 1;
    const int cus = device_cus();

    // the generic prev/next over all keys, gated on `gate` (nullptr: always)
    auto generic = [&](const int32_t *gate) -> pc_status {
        pc_status g = prev_next_core(keys, n, nullptr, prev, next, key_hist, w.generic, s, gate, gate != nullptr);
        if (g != PC_OK) return g;
        PC_LAUNCH(K_FILL32, chain_status_kernel, dim3(1), dim3(64), 0, s, (const int32_t *)w.generic, w.hdr,
                  HW_HIGH_ANCHOR, HW_PATH);
        return PC_OK;
    };
    if (n_seqs == 0) {   // n > 0 accesses in no request: an invalid layout
        if ((st = fill_u32(reinterpret_cast<uint32_t *>(w.hdr + HW_STATUS), (uint32_t)DEV_ERR_BAD_LAYOUT, 1, s)) !=
                PC_OK ||
            (st = fill_u32(reinterpret_cast<uint32_t *>(w.hdr + HW_PATH), 1u, 1, s)) != PC_OK ||
            (st = fill_u32(reinterpret_cast<uint32_t *>(w.hdr + HW_REASON), 1u, 1, s)) != PC_OK)
            return st;
        return generic(nullptr);
    }

    // Every decision below is taken on the device: later launches are gated
    // on header words, so the call never waits for the GPU.
    const uint64_t ns = chain_slots(n, n_seqs);
    const int32_t *chain = w.hdr + HW_CHAIN;
    PC_LAUNCH(K_CHAIN_ANCHOR, chain_layout_kernel, dim3((unsigned)((n_seqs + 255) / 256)), dim3(256), 0, s,
              blk_off, n_seqs, n, w.hdr);
    PC_LAUNCH(K_CHAIN_ANCHOR, chain_open_kernel, dim3(1), dim3(64), 0, s, w.hdr);
    PC_LAUNCH(K_CHAIN_ANCHOR, chain_anchor_kernel, dim3(wave_grid(n_seqs, cus)), dim3(CH_THREADS), 0, s, keys,
              blk_off, n_seqs, ns, deepest, w.akeys, w.rec, (const int32_t *)w.hdr);
    if ((st = prev_next_core(w.akeys, ns, nullptr, w.aprev, w.anext, nullptr, w.aws, s, chain, false)) != PC_OK)
        return st;
    PC_LAUNCH(K_FILL32, chain_status_kernel, dim3(1), dim3(64), 0, s, (const int32_t *)w.aws, w.hdr, HW_HIGH_ANCHOR,
              HW_CHAIN);
    if ((st = fill_u32_gated(reinterpret_cast<uint32_t *>(w.claimed), 0u, 2 * ns, s, chain)) != PC_OK) return st;
    const int batch = stair_batch(n);
    const dim3 stair_grid(wave_grid((ns + batch - 1) / batch, cus));
    if (batch == 16)
        PC_LAUNCH(K_CHAIN_STAIR, chain_stair_kernel<16>, stair_grid, dim3(CH_THREADS), 0, s, keys, ns,
                  (const uint4 *)w.rec, w.aprev, deepest, prev, next, want_next, w.open, w.claimed,
                  (const int32_t *)w.hdr);
    else if (batch == 8)
        PC_LAUNCH(K_CHAIN_STAIR, chain_stair_kernel<8>, stair_grid, dim3(CH_THREADS), 0, s, keys, ns,
                  (const uint4 *)w.rec, w.aprev, deepest, prev, next, want_next, w.open, w.claimed,
                  (const int32_t *)w.hdr);
    else
        PC_LAUNCH(K_CHAIN_STAIR, chain_stair_kernel<2>, stair_grid, dim3(CH_THREADS), 0, s, keys, ns,
                  (const uint4 *)w.rec, w.aprev, deepest, prev, next, want_next, w.open, w.claimed,
                  (const int32_t *)w.hdr);
    PC_LAUNCH(K_CHAIN_SCAN, chain_count_kernel, dim3((unsigned)((ns + 255) / 256)), dim3(256), 0, s, ns,
              (const uint4 *)w.rec, (const uint2 *)w.claimed, w.open, w.cnt, (const int32_t *)w.hdr);
    const uint64_t tiles = (ns + SCAN_TILE - 1) / SCAN_TILE;
    PC_LAUNCH(K_CHAIN_SCAN, chain_scan_tiles_kernel, dim3((unsigned)tiles), dim3(SCAN_THREADS), 0, s, w.cnt, ns,
              w.tsum, (const int32_t *)w.hdr);
    PC_LAUNCH(K_CHAIN_SCAN, chain_scan_top_kernel, dim3(1), dim3(SCAN_THREADS), 0, s, w.tsum, tiles, w.hdr);
    PC_LAUNCH(K_CHAIN_SCAN, chain_scan_apply_kernel, dim3((unsigned)tiles), dim3(SCAN_THREADS), 0, s, w.cnt, ns,
              w.tsum, w.coff, (const int32_t *)w.hdr);

    // the unresolved accesses: compacted, their own prev/next (over the
    // count the scan wrote, sized for the most that fit), merged back
    const uint64_t m_cap = open_capacity(w, n);
    OpenWs o;
    carve_open(w.generic, m_cap, &o);
    PC_LAUNCH(K_CHAIN_SCAN, chain_decide_kernel, dim3(1), dim3(64), 0, s, w.hdr, (const int32_t *)w.aws,
              (uint32_t)m_cap);
    PC_LAUNCH(K_CHAIN_COMPACT, chain_compact_kernel, dim3(wave_grid((ns + WAVE - 1) / WAVE, cus)),
              dim3(CH_THREADS), 0, s, keys, ns, (const uint4 *)w.rec, (const uint4 *)w.open, w.coff, deepest,
              o.ckeys, o.cpos, o.cflag, (const int32_t *)w.hdr);
    const uint32_t *m_dev = reinterpret_cast<const uint32_t *>(w.hdr + HW_UNRESOLVED);
    if ((st = prev_next_core(o.ckeys, m_cap, m_dev, o.cprev, o.cnext, nullptr, o.ws, s, chain, false)) != PC_OK)
        return st;
    PC_LAUNCH(K_FILL32, chain_status_kernel, dim3(1), dim3(64), 0, s, (const int32_t *)o.ws, w.hdr,
              HW_HIGH_UNRESOLVED, HW_CHAIN);
    uint64_t mg = (m_cap + CH_THREADS - 1) / CH_THREADS;
    if (mg > (uint64_t)cus * 16) mg = (uint64_t)cus * 16;
    PC_LAUNCH(K_CHAIN_MERGE, chain_merge_kernel, dim3((unsigned)(mg ? mg : 1)), dim3(CH_THREADS), 0, s, o.cpos,
              o.cflag, o.cprev, o.cnext, prev, next, want_next, w.hdr);

    // the check's verdict; the generic path over all keys runs only if it
    // (or an earlier step) says so
    PC_LAUNCH(K_CHAIN_MERGE, chain_verdict_kernel, dim3(1), dim3(64), 0, s, w.hdr, (const int32_t *)o.ws);
    return generic(w.hdr + HW_PATH);
}

}  // extern "C"
