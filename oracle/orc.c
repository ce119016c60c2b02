/*
 * Plain CPU oracle for the prefix-cache hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the tests, the entry point's smoke check and the
 * benchmark's CPU-baseline leg use it.  It shares no code, header, constant
 * table or helper with the GPU library: every definition below is written
 * out again from the paper's statement of the problem and from the
 * published algorithms it names.
 *
 * It is deliberately slow and literal:
 *   - block hashing walks every request's tokens in order;
 *   - prev/next-use indices come from a "last seen" dictionary scan;
 *   - LRU is simulated per capacity with an explicit recency list
 *     (Mattson et al. 1970 define the stack; we simply run the list);
 *   - exact stack distances come from walking the MRU list, and a second,
 *     independent exact method uses a Fenwick tree over "last occurrence"
 *     marks (Bennett & Kruskal 1975);
 *   - Belady's MIN is simulated per capacity with a max-heap on next use.
 *
 * Conventions (the paper leaves them open; these are the oracle's readings):
 *   - positions are uint32, 0xFFFFFFFF = none (cold / never reused);
 *   - the distance D(t) counts the distinct other blocks touched since the
 *     previous access of the same block; a hit at capacity c means D < c;
 *   - only full blocks of a request are accesses, in ascending depth order.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_NONE 0xFFFFFFFFu

/* ------------------------------------------------------------------ */
/* Block identity (Sec. 2.2: a cached KV state is reusable only if the */
/* whole preceding token sequence matches; Sec. 3.1: 16-token blocks). */
/* The paper does not give the hash.  Reading: splitmix64's finalizer  */
/* (Steele, Lea & Flood 2014) as a step function folded over 64-bit    */
/* token-pair words, then chained from the parent block.               */
/* ------------------------------------------------------------------ */

/* The step and the finalizer are kept file-local (and inlined) for the
 * hashing and fingerprint loops below; orc_mix64 / orc_step export them. */
static inline uint64_t mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* one step: S(x, w) = mix64((x xor w) + golden gamma) */
static inline uint64_t step(uint64_t x, uint64_t w)
{
    return mix64((x ^ w) + 0x9E3779B97F4A7C15ull);
}

uint64_t orc_mix64(uint64_t z) { return mix64(z); }

uint64_t orc_step(uint64_t x, uint64_t w) { return step(x, w); }

/* digest of one block of B tokens (B even): fold S over the B/2 words
 * w_k = tok[2k] | tok[2k+1] << 32, starting from 0 */
static inline uint64_t block_digest(const int32_t *tok, uint32_t B)
{
    uint64_t d = 0;
    for (uint32_t k = 0; k < B / 2; k++) {
        uint64_t lo = (uint64_t)(uint32_t)tok[2 * k];
        uint64_t hi = (uint64_t)(uint32_t)tok[2 * k + 1];
        d = step(d, lo | (hi << 32));
    }
    return d;
}

uint64_t orc_block_digest(const int32_t *tok, uint32_t B) { return block_digest(tok, B); }

/* Hash every full block of every request, request by request.
 * Request r covers tokens[tok_start[r] .. tok_start[r]+tok_len[r]).
 * Output layout: requests in order, blocks of a request in depth order.
 * key of block b = S(key of block b-1, digest_b), key of block -1 = root
 * (or parent[r] when parent is given).  depth[i] = b.
 * Returns the number of blocks written. */
uint64_t orc_hash_requests(const int32_t *tokens, const uint64_t *tok_start,
                           const uint32_t *tok_len, uint64_t n_req, uint32_t B,
                           const uint64_t *parent, uint64_t root,
                           uint64_t *keys, uint32_t *depth)
{
    uint64_t out = 0;
    for (uint64_t r = 0; r < n_req; r++) {
        uint64_t key = parent ? parent[r] : root;
        uint32_t nb = tok_len[r] / B;
        const int32_t *t = tokens + tok_start[r];
        for (uint32_t b = 0; b < nb; b++) {
            key = step(key, block_digest(t + (uint64_t)b * B, B));
            keys[out] = key;
            if (depth) depth[out] = b;
            out++;
        }
    }
    return out;
}

/* ------------------------------------------------------------------ */
/* Dense ids: an open-addressing dictionary from key to first-seen id. */
/* ------------------------------------------------------------------ */

static uint64_t slot_of(uint64_t key, uint64_t mask)
{
    /* any well-mixed spread works; the dictionary is exact either way */
    return (key * 0x9E3779B97F4A7C15ull >> 17) & mask;
}

/* id[t] = index of key[t] among distinct keys in order of first access.
 * The table starts small and doubles whenever it is half full, so its size
 * follows the number of distinct keys, not the number of accesses.  The
 * slot of a key a few accesses ahead is prefetched (a hint only).
 * Returns the number of distinct keys, or (uint64_t)-1 on allocation failure
 * or when there are 2^32 - 1 or more distinct keys. */
uint64_t orc_key_ids(const uint64_t *keys, uint64_t n, uint32_t *id)
{
    uint64_t cap = 1u << 16;
    uint64_t *tk = (uint64_t *)malloc(cap * sizeof(uint64_t));
    uint32_t *tv = (uint32_t *)malloc(cap * sizeof(uint32_t));
    if (!tk || !tv) { free(tk); free(tv); return (uint64_t)-1; }
    for (uint64_t i = 0; i < cap; i++) tv[i] = ORC_NONE;
    uint64_t mask = cap - 1, distinct = 0;
    const uint64_t ahead = 16;
    for (uint64_t t = 0; t < n; t++) {
        if (t + ahead < n) {
            uint64_t ps = slot_of(keys[t + ahead], mask);
            __builtin_prefetch(&tk[ps]);
            __builtin_prefetch(&tv[ps]);
        }
        uint64_t s = slot_of(keys[t], mask);
        while (tv[s] != ORC_NONE && tk[s] != keys[t]) s = (s + 1) & mask;
        if (tv[s] == ORC_NONE) {
            if (distinct >= ORC_NONE) { free(tk); free(tv); return (uint64_t)-1; }
            tk[s] = keys[t];
            tv[s] = (uint32_t)distinct++;
            if (2 * distinct >= cap) {
                /* double the table and re-insert every key */
                uint64_t ncap = cap * 2, nmask = ncap - 1;
                uint64_t *nk = (uint64_t *)malloc(ncap * sizeof(uint64_t));
                uint32_t *nv = (uint32_t *)malloc(ncap * sizeof(uint32_t));
                if (!nk || !nv) { free(nk); free(nv); free(tk); free(tv); return (uint64_t)-1; }
                for (uint64_t i = 0; i < ncap; i++) nv[i] = ORC_NONE;
                for (uint64_t i = 0; i < cap; i++) {
                    if (tv[i] == ORC_NONE) continue;
                    uint64_t q = slot_of(tk[i], nmask);
                    while (nv[q] != ORC_NONE) q = (q + 1) & nmask;
                    nk[q] = tk[i];
                    nv[q] = tv[i];
                }
                free(tk); free(tv);
                tk = nk; tv = nv; cap = ncap; mask = nmask;
                id[t] = (uint32_t)(distinct - 1);
                continue;
            }
        }
        id[t] = tv[s];
    }
    free(tk); free(tv);
    return distinct;
}

/* Fingerprints of arrays too large to keep: sum over positions t of
 * mix64(mix64(t0 + t + 1) + a[t]) mod 2^64.  Every term depends on both the
 * position and the value, so changing, dropping or moving one element
 * changes the sum (up to a 64-bit collision).  t0 lets a long array be
 * fingerprinted in pieces: the sums of the pieces add up. */
uint64_t orc_fp_u32(const uint32_t *a, uint64_t n, uint64_t t0)
{
    uint64_t s = 0;
    for (uint64_t t = 0; t < n; t++) s += mix64(mix64(t0 + t + 1) + (uint64_t)a[t]);
    return s;
}

uint64_t orc_fp_u64(const uint64_t *a, uint64_t n, uint64_t t0)
{
    uint64_t s = 0;
    for (uint64_t t = 0; t < n; t++) s += mix64(mix64(t0 + t + 1) + a[t]);
    return s;
}

/* prev[t] = last earlier position with the same key, next[t] = first later
 * one; ORC_NONE when there is none.  Scan in time order keeping, per id,
 * the position where it was last seen. */
int orc_prev_next(const uint32_t *id, uint64_t n, uint64_t n_ids,
                  uint32_t *prev, uint32_t *next)
{
    uint32_t *last = (uint32_t *)malloc((n_ids ? n_ids : 1) * sizeof(uint32_t));
    if (!last) return -1;
    for (uint64_t u = 0; u < n_ids; u++) last[u] = ORC_NONE;
    for (uint64_t t = 0; t < n; t++) {
        uint32_t p = last[id[t]];
        prev[t] = p;
        next[t] = ORC_NONE;
        if (p != ORC_NONE) next[p] = (uint32_t)t;
        last[id[t]] = (uint32_t)t;
    }
    free(last);
    return 0;
}

/* ------------------------------------------------------------------ */
/* LRU as an explicit recency list (Sec. 5 "LRU as a bedrock").        */
/* ------------------------------------------------------------------ */

/* Exact stack distance by walking the MRU list: D(t) = number of distinct
 * blocks used more recently than key[t]'s previous use; ORC_NONE if cold.
 * O(N * D): only for small traces. */
int orc_stack_distance_walk(const uint32_t *id, uint64_t n, uint64_t n_ids, uint32_t *dist)
{
    uint32_t *nx = (uint32_t *)malloc((n_ids + 1) * sizeof(uint32_t));
    uint32_t *pv = (uint32_t *)malloc((n_ids + 1) * sizeof(uint32_t));
    uint8_t *seen = (uint8_t *)calloc(n_ids + 1, 1);
    if (!nx || !pv || !seen) { free(nx); free(pv); free(seen); return -1; }
    uint32_t head = ORC_NONE;
    for (uint64_t t = 0; t < n; t++) {
        uint32_t u = id[t];
        if (!seen[u]) {
            dist[t] = ORC_NONE;
            seen[u] = 1;
        } else {
            uint32_t d = 0, x = head;
            while (x != u) { x = nx[x]; d++; }
            dist[t] = d;
            /* unlink u */
            if (pv[u] != ORC_NONE) nx[pv[u]] = nx[u]; else head = nx[u];
            if (nx[u] != ORC_NONE) pv[nx[u]] = pv[u];
        }
        /* push u at the front */
        pv[u] = ORC_NONE;
        nx[u] = head;
        if (head != ORC_NONE) pv[head] = u;
        head = u;
    }
    free(nx); free(pv); free(seen);
    return 0;
}

/* Second exact method (Bennett & Kruskal 1975): keep a mark at the last
 * occurrence of every key; D(t) = marks strictly between prev(t) and t. */
static void bit_add(int32_t *bit, uint64_t n, uint64_t i, int32_t v)
{
    for (i++; i <= n; i += i & (~i + 1)) bit[i] += v;
}
static int64_t bit_sum(const int32_t *bit, uint64_t i) /* sum of [0, i) */
{
    int64_t s = 0;
    for (; i > 0; i -= i & (~i + 1)) s += bit[i];
    return s;
}
int orc_stack_distance_bit(const uint32_t *prev, uint64_t n, uint32_t *dist)
{
    int32_t *bit = (int32_t *)calloc(n + 1, sizeof(int32_t));
    if (!bit) return -1;
    for (uint64_t t = 0; t < n; t++) {
        uint32_t p = prev[t];
        if (p == ORC_NONE) {
            dist[t] = ORC_NONE;
        } else {
            dist[t] = (uint32_t)(bit_sum(bit, t) - bit_sum(bit, (uint64_t)p + 1));
            bit_add(bit, n, p, -1);
        }
        bit_add(bit, n, t, +1);
    }
    free(bit);
    return 0;
}

/* One LRU cache of `cap` blocks run over the whole trace.  A block that is
 * resident when accessed is a hit; otherwise it is inserted at the front and,
 * if the cache then holds more than cap blocks, the least recently used one
 * is evicted.  cap = 0 never hits.
 * Outputs: hit count, sum of depth over hits, optional per-access hit flags,
 * optional fingerprint of the hit set: sum of mix64(t + 1) over the hits t
 * (mod 2^64), which names which accesses hit, not only how many. */
int orc_lru_sim(const uint32_t *id, const uint32_t *depth, uint64_t n, uint64_t n_ids,
                uint64_t cap, uint64_t *hits_out, uint64_t *depth_hits_out, uint8_t *hit_flag,
                uint64_t *fp_out)
{
    uint32_t *nx = (uint32_t *)malloc((n_ids + 1) * sizeof(uint32_t));
    uint32_t *pv = (uint32_t *)malloc((n_ids + 1) * sizeof(uint32_t));
    uint8_t *in = (uint8_t *)calloc(n_ids + 1, 1);
    if (!nx || !pv || !in) { free(nx); free(pv); free(in); return -1; }
    uint32_t head = ORC_NONE, tail = ORC_NONE;
    uint64_t size = 0, hits = 0, dh = 0, fp = 0;
    for (uint64_t t = 0; t < n; t++) {
        uint32_t u = id[t];
        int hit = 0;
        if (cap == 0) {
            if (hit_flag) hit_flag[t] = 0;
            continue;
        }
        if (in[u]) {
            hit = 1;
            hits++;
            if (depth) dh += depth[t];
            if (fp_out) fp += mix64(t + 1);
            if (u != head) { /* move to front */
                nx[pv[u]] = nx[u];
                if (nx[u] != ORC_NONE) pv[nx[u]] = pv[u]; else tail = pv[u];
                pv[u] = ORC_NONE; nx[u] = head; pv[head] = u; head = u;
            }
        } else {
            in[u] = 1;
            pv[u] = ORC_NONE; nx[u] = head;
            if (head != ORC_NONE) pv[head] = u; else tail = u;
            head = u;
            if (++size > cap) { /* evict the least recently used */
                uint32_t v = tail;
                tail = pv[v];
                nx[tail] = ORC_NONE;
                in[v] = 0;
                size--;
            }
        }
        if (hit_flag) hit_flag[t] = (uint8_t)hit;
    }
    *hits_out = hits;
    if (depth_hits_out) *depth_hits_out = dh;
    if (fp_out) *fp_out = fp;
    free(nx); free(pv); free(in);
    return 0;
}

/* ------------------------------------------------------------------ */
/* Request-level residency (Sec. 3.1 "Simulator"): every block of a     */
/* request must be resident at once during its prefill, so the cache    */
/* evicts ahead of time (least recently used first, never a block of    */
/* the request in flight) to make room for the request's misses.        */
/* Readings: hits are decided on arrival, before any eviction for the   */
/* request; afterwards all its blocks are the most recent, the deepest  */
/* one least recent of them (the order a serving engine frees a         */
/* request's blocks in); keys inside one request must be distinct       */
/* (true for chained prefix hashes).  A capacity below the largest      */
/* request is infeasible.  Requests are given by blk_off[0..n_seqs]:    */
/* request r holds accesses [blk_off[r], blk_off[r+1]) in depth order.  */
/* ------------------------------------------------------------------ */

/* Exact request-level distance by walking the MRU list: for every block of
 * request r, the number of distinct blocks above it in the recency list as
 * it stands when r arrives (ORC_NONE if never used before).  Returns -2 if a
 * key repeats inside a request. */
int orc_stack_distance_req_walk(const uint32_t *id, const uint64_t *blk_off, uint64_t n_seqs,
                                uint64_t n_ids, uint32_t *dist)
{
    uint32_t *nx = (uint32_t *)malloc((n_ids + 1) * sizeof(uint32_t));
    uint32_t *pv = (uint32_t *)malloc((n_ids + 1) * sizeof(uint32_t));
    uint8_t *seen = (uint8_t *)calloc(n_ids + 1, 1);
    uint64_t *stamp = (uint64_t *)calloc(n_ids + 1, sizeof(uint64_t));
    if (!nx || !pv || !seen || !stamp) { free(nx); free(pv); free(seen); free(stamp); return -1; }
    uint32_t head = ORC_NONE;
    for (uint64_t r = 0; r < n_seqs; r++) {
        uint64_t a = blk_off[r], b = blk_off[r + 1];
        for (uint64_t t = a; t < b; t++) {
            uint32_t u = id[t];
            if (stamp[u] == r + 1) { free(nx); free(pv); free(seen); free(stamp); return -2; }
            stamp[u] = r + 1;
            if (!seen[u]) {
                dist[t] = ORC_NONE;
            } else {
                uint32_t d = 0, x = head;
                while (x != u) { x = nx[x]; d++; }
                dist[t] = d;
            }
        }
        /* make the request's blocks the most recent: deepest first, so the
         * shallowest ends on top */
        for (uint64_t t = b; t > a; t--) {
            uint32_t u = id[t - 1];
            if (seen[u]) {
                if (pv[u] != ORC_NONE) nx[pv[u]] = nx[u]; else head = nx[u];
                if (nx[u] != ORC_NONE) pv[nx[u]] = pv[u];
            }
            seen[u] = 1;
            pv[u] = ORC_NONE;
            nx[u] = head;
            if (head != ORC_NONE) pv[head] = u;
            head = u;
        }
    }
    free(nx); free(pv); free(seen); free(stamp);
    return 0;
}

/* Second exact method: a mark at each key's last use in "recency time",
 * where request r occupies [blk_off[r], blk_off[r+1]) with its deepest block
 * first.  The distance of a block of r is the number of marks strictly
 * between its last use and the start of r, read before r places its own
 * marks (Bennett & Kruskal 1975, queried at the request start). */
int orc_stack_distance_req_bit(const uint32_t *id, const uint64_t *blk_off, uint64_t n_seqs, uint64_t n_ids,
                               uint32_t *dist)
{
    uint64_t n = blk_off[n_seqs];
    int32_t *bit = (int32_t *)calloc(n + 1, sizeof(int32_t));
    uint32_t *last = (uint32_t *)malloc((n_ids + 1) * sizeof(uint32_t));
    if (!bit || !last) { free(bit); free(last); return -1; }
    for (uint64_t i = 0; i <= n_ids; i++) last[i] = ORC_NONE;
    for (uint64_t r = 0; r < n_seqs; r++) {
        uint64_t a = blk_off[r], b = blk_off[r + 1];
        for (uint64_t t = a; t < b; t++) {
            uint32_t p = last[id[t]];
            dist[t] = p == ORC_NONE ? ORC_NONE : (uint32_t)(bit_sum(bit, a) - bit_sum(bit, (uint64_t)p + 1));
        }
        for (uint64_t t = a; t < b; t++) {
            uint32_t u = id[t];
            uint64_t when = a + (b - 1 - t);   /* deepest block first */
            if (last[u] != ORC_NONE) bit_add(bit, n, last[u], -1);
            bit_add(bit, n, when, +1);
            last[u] = (uint32_t)when;
        }
    }
    free(bit); free(last);
    return 0;
}

/* One request-level LRU cache of `cap` blocks: hits decided on arrival;
 * then least recently used blocks that are not part of the request are
 * evicted until the request's misses fit; the misses are inserted and the
 * request's blocks become the most recent (deepest least recent).  Returns
 * -3 if a request has more blocks than cap (infeasible capacity). */
int orc_lru_sim_req(const uint32_t *id, const uint32_t *depth, const uint64_t *blk_off, uint64_t n_seqs,
                    uint64_t n_ids, uint64_t cap, uint64_t *hits_out, uint64_t *depth_hits_out,
                    uint8_t *hit_flag)
{
    uint32_t *nx = (uint32_t *)malloc((n_ids + 1) * sizeof(uint32_t));
    uint32_t *pv = (uint32_t *)malloc((n_ids + 1) * sizeof(uint32_t));
    uint8_t *in = (uint8_t *)calloc(n_ids + 1, 1);
    uint64_t *pin = (uint64_t *)calloc(n_ids + 1, sizeof(uint64_t));
    if (!nx || !pv || !in || !pin) { free(nx); free(pv); free(in); free(pin); return -1; }
    uint32_t head = ORC_NONE, tail = ORC_NONE;
    uint64_t size = 0, hits = 0, dh = 0;
    int rc = 0;
    for (uint64_t r = 0; r < n_seqs && rc == 0; r++) {
        uint64_t a = blk_off[r], b = blk_off[r + 1], misses = 0;
        if (b - a > cap) { rc = -3; break; }
        for (uint64_t t = a; t < b; t++) {
            uint32_t u = id[t];
            pin[u] = r + 1;
            int h = in[u];
            if (h) { hits++; if (depth) dh += depth[t]; } else misses++;
            if (hit_flag) hit_flag[t] = (uint8_t)h;
        }
        /* proactive eviction: walk from the least recent end, skipping
         * blocks of the request in flight */
        uint32_t x = tail;
        while (size + misses > cap) {
            while (pin[x] == r + 1) x = pv[x];
            uint32_t y = pv[x];
            if (pv[x] != ORC_NONE) nx[pv[x]] = nx[x]; else head = nx[x];
            if (nx[x] != ORC_NONE) pv[nx[x]] = pv[x]; else tail = pv[x];
            in[x] = 0;
            size--;
            x = y;
        }
        /* the request's blocks to the front, deepest first */
        for (uint64_t t = b; t > a; t--) {
            uint32_t u = id[t - 1];
            if (in[u]) {
                if (pv[u] != ORC_NONE) nx[pv[u]] = nx[u]; else head = nx[u];
                if (nx[u] != ORC_NONE) pv[nx[u]] = pv[u]; else tail = pv[u];
            } else {
                in[u] = 1;
                size++;
            }
            pv[u] = ORC_NONE;
            nx[u] = head;
            if (head != ORC_NONE) pv[head] = u; else tail = u;
            head = u;
        }
    }
    *hits_out = hits;
    if (depth_hits_out) *depth_hits_out = dh;
    free(nx); free(pv); free(in); free(pin);
    return rc;
}

/* ------------------------------------------------------------------ */
/* Belady's MIN (Sec. 3.2: offline ceiling), demand paging: every      */
/* accessed block is inserted; on overflow evict the resident block    */
/* whose next use is farthest away (never reused = farthest).          */
/* ------------------------------------------------------------------ */

typedef struct { uint64_t when; uint32_t u; } heap_ent;

static void heap_push(heap_ent *h, uint64_t *n, heap_ent e)
{
    uint64_t i = (*n)++;
    while (i > 0) {
        uint64_t p = (i - 1) / 2;
        if (h[p].when >= e.when) break;
        h[i] = h[p];
        i = p;
    }
    h[i] = e;
}

static heap_ent heap_pop(heap_ent *h, uint64_t *n)
{
    heap_ent top = h[0], last = h[--(*n)];
    uint64_t i = 0;
    for (;;) {
        uint64_t c = 2 * i + 1;
        if (c >= *n) break;
        if (c + 1 < *n && h[c + 1].when > h[c].when) c++;
        if (h[c].when <= last.when) break;
        h[i] = h[c];
        i = c;
    }
    if (*n > 0) h[i] = last;
    return top;
}

int orc_belady_sim(const uint32_t *id, const uint32_t *next, uint64_t n, uint64_t n_ids,
                   uint64_t cap, uint64_t *hits_out, uint8_t *hit_flag)
{
    /* heap entries are (next use, id); stale entries are skipped on pop */
    heap_ent *h = (heap_ent *)malloc((n + 1) * sizeof(heap_ent));
    uint64_t *cur = (uint64_t *)malloc((n_ids + 1) * sizeof(uint64_t));
    uint8_t *in = (uint8_t *)calloc(n_ids + 1, 1);
    if (!h || !cur || !in) { free(h); free(cur); free(in); return -1; }
    uint64_t hn = 0, size = 0, hits = 0;
    for (uint64_t t = 0; t < n; t++) {
        uint32_t u = id[t];
        uint64_t when = next[t] == ORC_NONE ? UINT64_MAX : (uint64_t)next[t];
        int hit = 0;
        if (cap == 0) { if (hit_flag) hit_flag[t] = 0; continue; }
        if (in[u]) {
            hit = 1;
            hits++;
        } else {
            if (size == cap) {
                /* evict the resident block used farthest in the future;
                 * u is not resident, so every live heap entry is another block */
                heap_ent v;
                do { v = heap_pop(h, &hn); } while (!in[v.u] || cur[v.u] != v.when);
                in[v.u] = 0;
                size--;
            }
            in[u] = 1;
            size++;
        }
        cur[u] = when;
        heap_ent e = { when, u };
        heap_push(h, &hn, e);
        if (hit_flag) hit_flag[t] = (uint8_t)hit;
    }
    *hits_out = hits;
    free(h); free(cur); free(in);
    return 0;
}

/* ------------------------------------------------------------------ */
/* Session-level eviction (Sec. 5.3 "Block-Level vs. Session-Level      */
/* Eviction"): whole sessions are the unit of eviction.  Readings:      */
/*  - a session's footprint after one of its requests is the largest   */
/*    block count among its requests so far (append-only context);     */
/*  - the cache keeps resident sessions in recency order of their      */
/*    latest request; after each request its session moves to the     */
/*    front with its new footprint, then whole sessions are evicted    */
/*    from the least recent end while the resident footprints exceed   */
/*    the capacity (the arriving session last of all);                 */
/*  - a block hits if the session that made the previous access of the */
/*    same block is resident when the request arrives.                 */
/* Requests are blk_off[0..n_seqs] as above; sess[r] < n_sess is the   */
/* session of request r.                                               */
/* ------------------------------------------------------------------ */

/* One session-level LRU cache of `cap` blocks, simulated literally. */
int orc_session_sim(const uint32_t *id, const uint32_t *depth, const uint64_t *blk_off, const uint32_t *sess,
                    uint64_t n_seqs, uint64_t n_ids, uint64_t n_sess, uint64_t cap, uint64_t *hits_out,
                    uint64_t *depth_hits_out, uint8_t *hit_flag)
{
    uint32_t *last = (uint32_t *)malloc((n_ids + 1) * sizeof(uint32_t));   /* session of the last access */
    uint32_t *nx = (uint32_t *)malloc((n_sess + 1) * sizeof(uint32_t));
    uint32_t *pv = (uint32_t *)malloc((n_sess + 1) * sizeof(uint32_t));
    uint64_t *fp = (uint64_t *)calloc(n_sess + 1, sizeof(uint64_t));
    uint8_t *in = (uint8_t *)calloc(n_sess + 1, 1);
    if (!last || !nx || !pv || !fp || !in) { free(last); free(nx); free(pv); free(fp); free(in); return -1; }
    for (uint64_t i = 0; i <= n_ids; i++) last[i] = ORC_NONE;
    uint32_t head = ORC_NONE, tail = ORC_NONE;
    uint64_t total = 0, hits = 0, dh = 0;
    for (uint64_t r = 0; r < n_seqs; r++) {
        uint64_t a = blk_off[r], b = blk_off[r + 1];
        uint32_t s = sess[r];
        for (uint64_t t = a; t < b; t++) {
            uint32_t q = last[id[t]];
            int h = q != ORC_NONE && in[q];
            if (h) { hits++; if (depth) dh += depth[t]; }
            if (hit_flag) hit_flag[t] = (uint8_t)h;
        }
        for (uint64_t t = a; t < b; t++) last[id[t]] = s;
        /* the session to the front with its new footprint */
        if (in[s]) {
            if (pv[s] != ORC_NONE) nx[pv[s]] = nx[s]; else head = nx[s];
            if (nx[s] != ORC_NONE) pv[nx[s]] = pv[s]; else tail = pv[s];
            total -= fp[s];
        }
        if (b - a > fp[s]) fp[s] = b - a;
        in[s] = 1;
        total += fp[s];
        pv[s] = ORC_NONE;
        nx[s] = head;
        if (head != ORC_NONE) pv[head] = s; else tail = s;
        head = s;
        /* whole sessions out from the least recent end */
        while (total > cap) {
            uint32_t x = tail;
            tail = pv[x];
            if (tail != ORC_NONE) nx[tail] = ORC_NONE; else head = ORC_NONE;
            in[x] = 0;
            total -= fp[x];
        }
    }
    *hits_out = hits;
    if (depth_hits_out) *depth_hits_out = dh;
    free(last); free(nx); free(pv); free(fp); free(in);
    return 0;
}

/* Session-level distance of every access by walking the session recency
 * list as it stands when the request arrives: with q the session of the
 * block's previous access, the footprints of q and of every session above
 * it, summed, less one (so the block hits at capacity c iff distance < c);
 * ORC_NONE if the block was never used before. */
int orc_stack_distance_session_walk(const uint32_t *id, const uint64_t *blk_off, const uint32_t *sess,
                                    uint64_t n_seqs, uint64_t n_ids, uint64_t n_sess, uint32_t *dist)
{
    uint32_t *last = (uint32_t *)malloc((n_ids + 1) * sizeof(uint32_t));
    uint32_t *nx = (uint32_t *)malloc((n_sess + 1) * sizeof(uint32_t));
    uint32_t *pv = (uint32_t *)malloc((n_sess + 1) * sizeof(uint32_t));
    uint64_t *fp = (uint64_t *)calloc(n_sess + 1, sizeof(uint64_t));
    uint8_t *seen = (uint8_t *)calloc(n_sess + 1, 1);
    if (!last || !nx || !pv || !fp || !seen) { free(last); free(nx); free(pv); free(fp); free(seen); return -1; }
    for (uint64_t i = 0; i <= n_ids; i++) last[i] = ORC_NONE;
    uint32_t head = ORC_NONE;
    for (uint64_t r = 0; r < n_seqs; r++) {
        uint64_t a = blk_off[r], b = blk_off[r + 1];
        uint32_t s = sess[r];
        for (uint64_t t = a; t < b; t++) {
            uint32_t q = last[id[t]];
            if (q == ORC_NONE) { dist[t] = ORC_NONE; continue; }
            uint64_t sum = 0;
            uint32_t x = head;
            for (;;) {
                sum += fp[x];
                if (x == q) break;
                x = nx[x];
            }
            dist[t] = (uint32_t)(sum - 1);   /* sum <= number of accesses < 2^32 */
        }
        for (uint64_t t = a; t < b; t++) last[id[t]] = s;
        if (seen[s]) {
            if (pv[s] != ORC_NONE) nx[pv[s]] = nx[s]; else head = nx[s];
            if (nx[s] != ORC_NONE) pv[nx[s]] = pv[s];
        }
        seen[s] = 1;
        if (b - a > fp[s]) fp[s] = b - a;
        pv[s] = ORC_NONE;
        nx[s] = head;
        if (head != ORC_NONE) pv[head] = s;
        head = s;
    }
    free(last); free(nx); free(pv); free(fp); free(seen);
    return 0;
}

/* ------------------------------------------------------------------ */
/* Capacity bins of a distance array, with the hit-set fingerprint of   */
/* each bin: bin k < K holds the accesses with caps[k-1] <= D < caps[k]  */
/* (caps[-1] = 0), bin K the cold ones and D >= caps[K-1].  An access    */
/* hits at caps[k] exactly when its bin is <= k, so prefix sums of the   */
/* bins give hits and the hit-set fingerprint (sum of mix64(t0 + t + 1)) */
/* at every capacity.  count and fp have K + 1 entries and are added to. */
/* ------------------------------------------------------------------ */
int orc_dist_bins(const uint32_t *dist, uint64_t n, uint64_t t0, const uint64_t *caps, uint32_t K,
                  uint64_t *count, uint64_t *fp)
{
    for (uint64_t t = 0; t < n; t++) {
        uint32_t d = dist[t];
        uint32_t b = K;
        if (d != ORC_NONE) {
            /* number of edges <= d */
            uint32_t lo = 0, hi = K;
            while (lo < hi) {
                uint32_t mid = (lo + hi) / 2;
                if (caps[mid] <= (uint64_t)d) lo = mid + 1; else hi = mid;
            }
            b = lo;
        }
        count[b] += 1;
        fp[b] += mix64(t0 + t + 1);
    }
    return 0;
}
