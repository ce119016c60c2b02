/*
 * libpc -- the prefix-cache eviction hot path on one AMD Instinct MI355X
 * (gfx950): chained block hashing, prev/next-use indexing, exact LRU stack
 * distance and the hit-ratio / compute-savings histograms over every cache
 * capacity at once.
 *
 * Paper: Y. Liu, M. Yu, J. Yang, "When Fancy Eviction Fails: Rethinking Cache
 * Replacement For LLM Prefix Reuse".  Each entry point cites the passage
 * that defines what it computes.
 *
 * Common rules
 *   - Every array argument is DEVICE memory (hipMalloc / a torch tensor on the
 *     GPU) unless stated otherwise.  The caller owns all memory; the library
 *     never allocates or frees, and only the read-back calls
 *     (pc_workspace_status, pc_prof_read) synchronise: where a call picks
 *     between two paths from its data, it does so on the device and gates
 *     the launches of both, so any sequence of calls can be captured into a
 *     graph.
 *     Scratch space comes only from
 *     the caller's workspace `ws` of at least the size the matching `*_ws`
 *     query returns (256-byte aligned).
 *   - Work is enqueued on `stream` and the call returns; outputs are valid once
 *     the stream has completed.  Calls are thread-safe given distinct
 *     workspaces; two calls that share a workspace must be ordered on a stream.
 *   - Positions are uint32; PC_NONE (0xFFFFFFFF) means "none" (no previous /
 *     next use, or an infinite distance).  Hence n must be below 2^32 - 1.
 *   - Arguments are checked before anything is launched; on error nothing is
 *     enqueued and outputs are untouched.  A failed launch returns
 *     PC_ERR_DEVICE.  Nothing throws across this interface.
 */
#ifndef PC_H
#define PC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    PC_OK = 0,
    PC_ERR_INVALID = -1,     /* NULL required pointer, bad block size, bad caps */
    PC_ERR_TOO_LARGE = -2,   /* n >= 2^32 - 1 (positions must fit uint32)       */
    PC_ERR_WORKSPACE = -3,   /* ws NULL or smaller than the query               */
    PC_ERR_DEVICE = -4,      /* a HIP call or kernel launch failed              */
    PC_ERR_UNSUPPORTED = -5  /* no usable gfx950 device                          */
} pc_status;

#define PC_NONE 0xFFFFFFFFu
#define PC_MAX_CAPS 4096u
#define PC_HASH_DEEPEST_FIRST 1u   /* pc_hash_blocks flag */
#define PC_PREV_ONLY 2u            /* pc_prev_next_chained flag: next is scratch */
#define PC_MAX_PROFILE_EDGES 128u  /* time-histogram edges of the profiles */
#define PC_MAX_FREQ 2048u          /* largest exact frequency / request-count bin */
#define PC_FREQ_CLASSES 32u        /* frequency classes floor(log2 f) */
#define PC_MAX_FOOTPRINT (1u << 24) /* largest exact footprint bin */

/* Human-readable name of a status code (static storage). */
const char *pc_status_string(pc_status s);

/* Library version as major*10000 + minor*100 + patch. */
int pc_version(void);

/* ------------------------------------------------------------------------
 * Chained block hashing.
 *
 * Paper: a cached KV state is reusable only if the whole preceding token
 * sequence matches (Sec. 2.2 "LLM Serving Prefix Cache"); KV state is managed
 * in fixed-size blocks of 16 tokens (Sec. 2.2; Sec. 3.1 "Traces": 16-token
 * blocks with block identity scoped across sessions).  The paper does not
 * give the hash; this library fixes it as follows (all arithmetic mod 2^64):
 *     mix64(z)  = splitmix64 finalizer (Steele, Lea & Flood 2014)
 *     S(x, w)   = mix64((x ^ w) + 0x9E3779B97F4A7C15)
 *     word k    = (uint32)tok[2k] | (uint64)(uint32)tok[2k+1] << 32
 *     digest(b) = S folded over the B/2 words of block b, starting from 0
 *     key(b)    = S(key(b-1), digest(b)),  key(-1) = parent[r] or root
 * Only full blocks count: request r yields floor(tok_len[r] / B) accesses, in
 * ascending depth order.
 *
 *   tokens     int32[n_tokens] token buffer
 *   tok_start  uint64[n_seqs]  first token of request r inside `tokens`
 *   tok_len    uint32[n_seqs]  token count of request r (views may overlap:
 *                               all turns of one session can share one stream)
 *   block_size B, even, 2..1024
 *   parent     uint64[n_seqs] chain start per request, or NULL to use `root`
 *   blk_off    uint64[n_seqs+1] exclusive prefix sum of floor(tok_len/B):
 *                               block b of request r goes to keys[blk_off[r]+b];
 *                               blk_off[n_seqs] must equal n_blocks
 *   keys       uint64[n_blocks] output
 *   depth      uint32[n_blocks] output block index b inside its request, or NULL
 *   key_hist   uint32[4 * 256] output, or NULL: key_hist[256 p + d] counts the
 *              keys written whose byte p (bits 8p .. 8p+7) is d, p = 0..3.
 *              Zeroed by the call.  Handing it to pc_prev_next_use spares that
 *              call a full read of the keys.
 *   flags      0, or PC_HASH_DEEPEST_FIRST: each request's blocks (keys and
 *              depths) are written in descending depth order inside the
 *              request's range, i.e. block b goes to blk_off[r+1] - 1 - b
 *              (the recency order of request-level residency; the same as
 *              pc_request_order applied afterwards).
 * A request whose tokens run past n_tokens, or whose blocks run past
 * n_blocks, is skipped and the workspace status (pc_workspace_status) is set
 * to 2; nothing is read or written out of bounds.
 * ------------------------------------------------------------------------ */
size_t pc_hash_blocks_ws(uint32_t n_seqs);
pc_status pc_hash_blocks(const int32_t *tokens, uint64_t n_tokens, const uint64_t *tok_start,
                         const uint32_t *tok_len, uint32_t n_seqs, uint32_t block_size,
                         const uint64_t *parent, uint64_t root, const uint64_t *blk_off,
                         uint64_t n_blocks, uint64_t *keys, uint32_t *depth, uint32_t *key_hist,
                         uint32_t flags, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Previous / next use of every access.
 *
 * prev[t] = max{ i < t : keys[i] == keys[t] } or PC_NONE;
 * next[t] = min{ i > t : keys[i] == keys[t] } or PC_NONE.
 * The next-use time is what Belady-style offline analysis ranks blocks by
 * (Sec. 3.2 "Belady's optimum"; Sec. 5.2 "BeladyCompute", time until next
 * access); prev == PC_NONE marks a compulsory miss (Sec. 4.6).
 *
 *   keys      uint64[n]; prev, next uint32[n] outputs.
 *   key_hist  uint32[4 * 256] or NULL: the byte histograms of the low four key
 *             bytes as pc_hash_blocks counts them, for exactly these keys; NULL
 *             counts them here (one more read of the keys).  A histogram whose
 *             rows do not each sum to n sets the workspace status to 4; one
 *             that sums right but does not match the keys gives unspecified
 *             outputs (never an access out of bounds).
 * Keys are grouped by their low 32 bits first; only when many different keys
 * share those bits does the call also sort by the high 32 bits.  Once the
 * stream has completed, 32-bit word 1 of the workspace tells which happened
 * (1 = the high bits were sorted too); the outputs are the same either way.
 * ------------------------------------------------------------------------ */
size_t pc_prev_next_use_ws(uint64_t n);
pc_status pc_prev_next_use(const uint64_t *keys, uint64_t n, uint32_t *prev, uint32_t *next,
                           const uint32_t *key_hist, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Previous / next use of every access of a chained-key trace.
 *
 * Same prev and next as pc_prev_next_use, for keys laid out as
 * pc_hash_blocks writes them: request r's blocks at blk_off[r] ..
 * blk_off[r+1] - 1, ascending depth (flags 0) or descending depth
 * (PC_HASH_DEEPEST_FIRST).  Chained keys fix the whole prefix (Sec. 2.2), so
 * a request's reuse links come in long runs to very few earlier requests:
 * the call links anchors every 64 depths with the generic prev/next, extends
 * each anchor link over the 64 depths it covers by comparing keys, runs the
 * generic prev/next over the accesses left without a link (first and last
 * uses, mostly), and checks the merged result.  The outputs are exact for any
 * keys: when the check fails, the block layout is invalid, or the unresolved
 * accesses do not fit the workspace, the generic prev/next runs over all keys.
 *
 *   keys      uint64[n]; prev, next uint32[n] outputs.
 *   blk_off   uint64[n_seqs+1], blk_off[0] = 0, non-decreasing, blk_off[n_seqs]
 *             = n.  Any other layout sets the workspace status to 2 and takes
 *             the generic path (outputs still exact).
 *   flags     0 or PC_HASH_DEEPEST_FIRST, or'ed with PC_PREV_ONLY when only
 *             prev is wanted (session-level eviction, Sec. 5.3, reads no next
 *             use): next is still required, as scratch for the generic path,
 *             and its contents after the call are unspecified; the chain path
 *             then skips its next links (about 4 bytes per access).
 *   key_hist  as for pc_prev_next_use; used only by the generic path over all
 *             keys.
 * Every choice between the two paths is made on the device: the unresolved
 * stage is sized for the most unresolved accesses the workspace holds and
 * works on the count the GPU wrote, and the generic path's launches are
 * gated on the verdict, so the call does not synchronise.  Workspace words
 * after the call:
 * word 1 = 1 if the generic path ran over all keys, word 2 = the number of
 * accesses that went through the generic prev/next of the unresolved ones,
 * word 3 = why the generic path ran (1 layout, 2 too many unresolved,
 * 3 check failed, 4 an inner call reported an error), word 6 = 1 if the
 * prev/next over the anchors (or, when word 1 = 1, over all keys) also
 * sorted by the high key bits, word 7 = the same for the unresolved ones.
 * ------------------------------------------------------------------------ */
size_t pc_prev_next_chained_ws(uint64_t n, uint32_t n_seqs);
pc_status pc_prev_next_chained(const uint64_t *keys, uint64_t n, const uint64_t *blk_off, uint32_t n_seqs,
                               uint32_t flags, uint32_t *prev, uint32_t *next, const uint32_t *key_hist,
                               void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Exact LRU stack distance of every access.
 *
 * dist[t] = #{ i in (prev(t), t) : next(i) > t }  (next(i) = PC_NONE counts
 * as infinity), i.e. the number of distinct other blocks touched since the
 * previous access of the same block; PC_NONE when prev(t) = PC_NONE.  LRU is
 * a stack algorithm, so an access hits in an LRU cache of c blocks exactly
 * when dist < c, at every c at once (Sec. 5 "LRU as a bedrock"; Appendix B
 * "stack distance between reuses", "reuses reachable within capacity").
 *
 *   prev, next uint32[n] as produced by pc_prev_next_use; dist uint32[n] out.
 * ------------------------------------------------------------------------ */
size_t pc_stack_distance_ws(uint64_t n);
pc_status pc_stack_distance(const uint32_t *prev, const uint32_t *next, uint64_t n,
                            uint32_t *dist, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Exact LRU stack distance without allocation, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same dist as pc_stack_distance, with
 * the workspace taken from a fixed 128 MiB device array inside the library
 * (one per GPU, held until the process ends) instead of the caller: the
 * call allocates nothing and synchronises nothing.  The caller passes the
 * inputs and the output as for pc_stack_distance.
 *   n above pc_stack_distance_noalloc_max_n() (about 8.0e6 accesses: the n
 *   whose workspace still fits the array) returns PC_ERR_TOO_LARGE before
 *   anything is enqueued.
 * Every call on one GPU shares that GPU's array: calls that overlap on one
 * device (two streams, two threads) race and must be ordered by the caller.
 * The array keeps the last call's contents; each call clears what it reads.
 * The device-side status word lives in that array and is not reported:
 * prev / next that are not mutual links give unspecified distances (never a
 * write out of bounds).  Keep pc_prof_enable off for calls that must not
 * allocate (the timing events are created on demand).
 * ------------------------------------------------------------------------ */
uint64_t pc_stack_distance_noalloc_max_n(void);
pc_status pc_stack_distance_noalloc(const uint32_t *prev, const uint32_t *next, uint64_t n, uint32_t *dist,
                                    void *stream);

/* ------------------------------------------------------------------------
 * Exact LRU stack distance of every access, from the runs of the prev stream.
 *
 * Same dist as pc_stack_distance (Sec. 5; Appendix B).  When t - 1 and t are
 * both warm and prev(t) = prev(t - 1) + 1, the reuse window of t is that of
 * t - 1 shifted by one position, with one block leaving and one entering, so
 * dist(t) = dist(t - 1); a maximal chain of such accesses is a run.  Chained
 * block keys give about one run per request, so the call counts over runs
 * instead of accesses: per run, the earlier runs whose previous uses come
 * first (the previous uses of a run are one contiguous range, disjoint from
 * every other run's), then the run's distance along all its accesses.
 *
 *   prev, next uint32[n] as produced by pc_prev_next_use; dist uint32[n] out.
 * With more than n/16 + 1024 runs (streams without that structure) the
 * dominance count of pc_stack_distance runs instead (same result).  The
 * choice is made on the device: the call does not synchronise, and every
 * launch of the path not taken returns at once, so a graph capture of the
 * call replays correctly for any input.  Workspace words after the call:
 * word 1 = 1 if pc_stack_distance's count ran, word 2 = the number of runs,
 * word 3 = the number of cold accesses.
 * ------------------------------------------------------------------------ */
size_t pc_stack_distance_runs_ws(uint64_t n);
pc_status pc_stack_distance_runs(const uint32_t *prev, const uint32_t *next, uint64_t n,
                                 uint32_t *dist, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Request-level residency (Sec. 3.1 "Simulator": every block of a request
 * must be resident at once during its prefill, so room is made ahead of time
 * by evicting least recently used blocks that are not part of the request).
 * Readings: a block hits if it is resident when its request arrives;
 * afterwards the request's blocks are the most recent, its deepest block the
 * least recent of them.  For a capacity c of at least the largest request's
 * block count this cache is a stack algorithm too: a block hits exactly when
 * dist_req < c, where dist_req counts the distinct blocks above it in the
 * recency list when its request arrives.  Capacities below the largest
 * request cannot hold that request (Sec. 3.1 "Cache-size regimes") and are
 * the caller's to exclude.  Keys inside one request must be distinct (chained
 * prefix hashes are); otherwise the results are unspecified (memory-safe).
 *
 * Pipeline: pc_hash_blocks with PC_HASH_DEEPEST_FIRST writes each request's
 * accesses in that recency order (deepest block first), or pc_request_order
 * reorders keys written in depth order; pc_prev_next_use and
 * pc_stack_distance run unchanged on the reordered keys;
 * pc_stack_distance_req turns their outputs into dist_req (same order).  All
 * arrays of one pipeline share that order.
 * ------------------------------------------------------------------------ */

/* Each request's accesses in reverse: keys_out[blk_off[r+1]-1-j] =
 * keys[blk_off[r]+j] (and the same for depth when given).  blk_off is the
 * uint64[n_seqs+1] request table of pc_hash_blocks (blk_off[n_seqs] = n).
 * Outputs must not alias inputs.  A request with blk_off[r] > blk_off[r+1]
 * or past n is skipped and the workspace status is set to 2. */
size_t pc_request_order_ws(void);
pc_status pc_request_order(const uint64_t *keys, const uint32_t *depth, const uint64_t *blk_off,
                           uint32_t n_seqs, uint64_t n, uint64_t *keys_out, uint32_t *depth_out,
                           void *ws, size_t ws_bytes, void *stream);

/* dist_req from prev and dist of the reordered accesses (uint32[n] each,
 * recency order, as pc_prev_next_use and pc_stack_distance give them) and
 * the request table.  With v = prev + 1 (0 for a cold access) and t in
 * request r, s = blk_off[r]:
 *   dist_req[t] = dist[t] - #{ j in [s, t) : v(j) < v(t) },
 * PC_NONE when prev[t] = PC_NONE.  The blocks above t's block when its
 * request arrives are the distinct blocks used between prev[t] and s; the
 * per-access distance also counts the request's accesses in [s, t) whose
 * blocks were not among them, which are those with v(j) < v(t).  Chained
 * prefix keys make the count t - s (one pass over prev and dist); other key
 * streams are counted directly where they break that order (slower, same
 * result).  blk_off[0] != 0, blk_off[n_seqs] != n or a decreasing step sets
 * the workspace status to 2 (results unspecified, memory-safe). */
size_t pc_stack_distance_req_ws(void);
pc_status pc_stack_distance_req(const uint32_t *prev, const uint32_t *dist, const uint64_t *blk_off,
                                uint32_t n_seqs, uint64_t n, uint32_t *dist_req, void *ws,
                                size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Session-level eviction (Sec. 5.3 "Block-Level vs. Session-Level Eviction":
 * whole sessions are evicted at once, trading hit ratio at small capacities
 * for far less metadata).  Readings: a session's footprint after one of its
 * requests is the largest block count among its requests so far; resident
 * sessions are kept in recency order of their latest request and evicted
 * whole from the least recent end while their footprints exceed the
 * capacity (the arriving session last); a block hits if the session that
 * made its previous access is resident when the request arrives.  Footprints
 * only grow, so this is a stack algorithm: a block hits at capacity c
 * exactly when dist_sess < c, where dist_sess is the footprint of that
 * session plus the latest footprints of all sessions active since its
 * latest request, less one.  Keys inside one request must be distinct;
 * otherwise results are unspecified (memory-safe).
 *
 *   prev     uint32[n] from pc_prev_next_use over the keys in request order
 *   blk_off  uint64[n_seqs+1] request table (blk_off[n_seqs] = n)
 *   session  uint32[n_seqs] session of each request (any ids)
 *   dist_sess uint32[n] out, PC_NONE where prev is PC_NONE
 * A bad request table sets the workspace status to 2; a look-back timeout
 * in the request-level linking sets 1.
 * ------------------------------------------------------------------------ */
size_t pc_stack_distance_session_ws(uint64_t n, uint32_t n_seqs);
pc_status pc_stack_distance_session(const uint32_t *prev, const uint64_t *blk_off, const uint32_t *session,
                                    uint32_t n_seqs, uint64_t n, uint32_t *dist_sess, void *ws,
                                    size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Workload characterisation (Sec. 4) from the index arrays.  Times are
 * request timestamps in microseconds (uint64[n_seqs], non-decreasing; a
 * block access takes its request's time).  Time histograms use the bin
 * convention of pc_mrc_weighted: bin k < K holds values v with
 * edges[k-1] <= v < edges[k] (edges[-1] = 0), bin K holds v >= edges[K-1];
 * 1 <= K = n_edges <= PC_MAX_PROFILE_EDGES, edges non-decreasing (checked on
 * the device: status 3).  Every output is zeroed on `stream`, then
 * accumulated; a bad request table sets status 2.
 * ------------------------------------------------------------------------ */

/* Per reuse and per block, from prev/next (pc_prev_next_use) in request
 * order:
 *   interval[K+1]      reuses t (prev exists) by ts(t) - ts(prev t)
 *                      (Sec. 4.2 reuse intervals)
 *   lifetime[K+1]      blocks by ts(last access) - ts(first access), 0 for a
 *                      block used once (Sec. 4.1 lifetimes)
 *   freq[freq_max+1]   blocks by access count f, bin min(f, freq_max), bin 0
 *                      empty; with it the chance of a further access after k
 *                      accesses is #(f >= k+1) / #(f >= k) (Sec. 4.3)
 *   life_by_class[PC_FREQ_CLASSES * (K+1)]  lifetime histogram per frequency
 *                      class floor(log2 f), class-major (Sec. 4.3, lifetime
 *                      against frequency)
 * 1 <= freq_max <= PC_MAX_FREQ. */
size_t pc_reuse_profile_ws(uint64_t n);
pc_status pc_reuse_profile(const uint32_t *prev, const uint32_t *next, const uint64_t *blk_off,
                           const uint64_t *ts_us, uint32_t n_seqs, uint64_t n, const uint64_t *edges,
                           uint32_t n_edges, uint32_t freq_max, uint64_t *interval, uint64_t *lifetime,
                           uint64_t *freq, uint64_t *life_by_class, void *ws, size_t ws_bytes, void *stream);

/* Per session, from the request table and the session of every request:
 *   footprint[fp_max+1]  sessions by footprint, the largest request's block
 *                        count (contexts are append-only), bin min(fp, fp_max)
 *                        (Sec. 4.5; its CCDF and Lorenz curve follow)
 *   requests[rq_max+1]   sessions by number of requests, bin min(count, rq_max)
 *                        (Sec. 4.3 requests per session)
 *   duration[K+1]        sessions by ts(last request) - ts(first request)
 *                        (Sec. 4.1 session duration)
 *   gap[K+1]             requests with an earlier request of the same session
 *                        by the time since it (Sec. 4.2 inter-request time)
 * 1 <= rq_max <= PC_MAX_FREQ, 1 <= fp_max <= PC_MAX_FOOTPRINT. */
size_t pc_session_profile_ws(uint32_t n_seqs);
pc_status pc_session_profile(const uint64_t *blk_off, const uint32_t *session, const uint64_t *ts_us,
                             uint32_t n_seqs, uint64_t n, const uint64_t *edges, uint32_t n_edges,
                             uint32_t fp_max, uint32_t rq_max, uint64_t *footprint, uint64_t *requests,
                             uint64_t *duration, uint64_t *gap, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Hit-ratio and compute-savings histograms over capacity edges.
 *
 * Paper: block hit ratio counts every access, compulsory misses included
 * (Sec. 3.2); the compute-savings ratio weights every hit by the recompute
 * cost it avoids and divides by the cost of all accesses (Sec. 5.2
 * "Compute-awareness"); the cost grows with the block's token depth
 * (Sec. 4.4 "Position-Dependent Miss Costs"); a linear-in-depth model is
 * the extreme case (Appendix C).  Here cost(t) = alpha + beta * depth[t].
 *
 * Bin k in [0, n_caps) counts accesses with caps[k-1] <= dist < caps[k]
 * (caps[-1] = 0); bin n_caps counts dist >= caps[n_caps-1] and dist == PC_NONE.
 * So hits at capacity caps[k] = sum of count[0..k].  Per bin:
 *     count[k]     uint64  number of accesses
 *     depthsum[k]  uint64  sum of depth over them (0 when depth is NULL)
 *     cost_hi:lo   uint128 alpha*count[k] + beta*depthsum[k] (exact)
 * When `next` is not NULL, nextuse_hist[k] bins the next-use gap next[t] - t
 * on the same edges (PC_NONE goes to bin n_caps).
 *
 *   dist   uint32[n]; depth uint32[n] or NULL; next uint32[n] or NULL
 *   caps   uint64[n_caps] non-decreasing, 1 <= n_caps <= PC_MAX_CAPS (device
 *          memory; the order is checked on the device: a decreasing pair sets
 *          the workspace status to 3 and leaves the bins undefined)
 *   count, depthsum, cost_lo, cost_hi: uint64[n_caps+1] outputs (required)
 *   nextuse_hist: uint64[n_caps+1] output, required when next != NULL; when
 *          given it is always zeroed (and stays zero when next is NULL)
 * Outputs are zeroed on `stream` first, then accumulated.  One pass over the
 * inputs counts up to 1024 edges; more edges take one more pass per 1024.
 * ------------------------------------------------------------------------ */
size_t pc_mrc_weighted_ws(uint64_t n, uint32_t n_caps);
pc_status pc_mrc_weighted(const uint32_t *dist, const uint32_t *depth, const uint32_t *next,
                          uint64_t n, const uint64_t *caps, uint32_t n_caps, uint64_t alpha,
                          uint64_t beta, uint64_t *count, uint64_t *depthsum, uint64_t *cost_lo,
                          uint64_t *cost_hi, uint64_t *nextuse_hist, void *ws, size_t ws_bytes,
                          void *stream);

/* ------------------------------------------------------------------------
 * The same bins with each access's depth taken from the request layout
 * instead of an array: depth[t] = t - blk_off[r] for the request r holding
 * position t (flags 0), or blk_off[r+1] - 1 - t (PC_HASH_DEEPEST_FIRST),
 * which is the block's depth in its request's prefix when the keys are laid
 * out as pc_hash_blocks writes them with the same flags (Sec. 4.4, the miss
 * cost grows with the block's position in the prompt).  The hash
 * then need not write depth, and the bins read 12 bytes of layout map per
 * 64 accesses (built in the workspace) instead of 256 bytes of depth.
 *
 *   flags     0 or PC_HASH_DEEPEST_FIRST.
 *   blk_off   uint64[n_seqs+1] device memory, blk_off[0] = 0, non-decreasing,
 *             blk_off[n_seqs] = n (empty requests allowed); any other layout
 *             sets the workspace status to 2 and leaves the bins undefined.
 *   other arguments, outputs and status as for pc_mrc_weighted; the
 *   workspace (pc_mrc_weighted_layout_ws) holds 12 bytes per 64 accesses.
 * ------------------------------------------------------------------------ */
size_t pc_mrc_weighted_layout_ws(uint64_t n, uint32_t n_caps);
pc_status pc_mrc_weighted_layout(const uint32_t *dist, const uint64_t *blk_off, uint32_t n_seqs, uint32_t flags,
                                 const uint32_t *next, uint64_t n, const uint64_t *caps, uint32_t n_caps,
                                 uint64_t alpha, uint64_t beta, uint64_t *count, uint64_t *depthsum,
                                 uint64_t *cost_lo, uint64_t *cost_hi, uint64_t *nextuse_hist, void *ws,
                                 size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Belady's MIN at many capacities at once: the offline ceiling every online
 * policy is compared with (Sec. 3.2 "Belady's optimum"; Appendix B, the
 * LRU-Belady gap under concurrency).  Demand paging: every accessed block
 * is brought in, and when the cache already holds c blocks the resident
 * block whose next use is farthest away leaves first (a block never used
 * again is the farthest).  Hit counts are unique (victim ties occur only
 * among blocks that are never used again).  Capacities are in blocks and
 * need not be ordered; c = 0 never hits.
 *
 *   next      uint32[n] from pc_prev_next_use (PC_NONE: never used again);
 *             an entry that is not PC_NONE and not in (t, n) sets the
 *             workspace status to 2 and counts as PC_NONE
 *   depth     uint32[n] or NULL (depth sums are then 0)
 *   caps      uint64[n_caps] device memory, 1 <= n_caps <= PC_MAX_CAPS
 *   hits      uint64[n_caps] out: hits at caps[k]
 *   depthsum  uint64[n_caps] out: sum of depth over those hits (with the
 *             linear cost of pc_mrc_weighted: saved = alpha*hits + beta*depthsum)
 *   hit_flags uint8[n_caps * n] out or NULL: hit_flags[k*n + t] = 1 when
 *             access t hits at caps[k]
 * One wave simulates one capacity through the whole trace, all capacities
 * at once: the call takes time linear in n, not one memory pass (on MI355X
 * about 0.8 s per 2.8e7 accesses for a capacity that rarely evicts, up to
 * 2.3 s for one that evicts on most accesses).
 * Workspace: about n_caps * n / 8 bytes of bitmaps.  Status 5 reports an
 * internal consistency check (not expected for a valid next[]).
 * ------------------------------------------------------------------------ */
size_t pc_belady_ws(uint64_t n, uint32_t n_caps);
pc_status pc_belady(const uint32_t *next, const uint32_t *depth, uint64_t n, const uint64_t *caps,
                    uint32_t n_caps, uint64_t *hits, uint64_t *depthsum, uint8_t *hit_flags, void *ws,
                    size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * Device-side status.  Every call clears word 0 of its workspace; kernels
 * record a non-zero code there instead of faulting or hanging:
 *   1  a wait on another workgroup (decoupled look-back) gave up after a
 *      bounded spin (outputs undefined);
 *   2  a bad layout: pc_hash_blocks, a request's tokens or blocks fall
 *      outside the arrays (that request was skipped); the calls that take a
 *      request table, a table that is not a non-decreasing prefix ending at
 *      n; pc_stack_distance, prev / next that are not mutual links (outputs
 *      undefined, nothing written out of bounds);
 *   3  pc_mrc_weighted and the profiles: edges not non-decreasing (bins
 *      undefined);
 *   4  pc_prev_next_use: a given key histogram does not sum to n;
 *   5  pc_belady: an internal consistency check failed (results undefined).
 * This call copies the code of workspace `ws` to *code_out after
 * synchronising `stream` (with pc_prof_read, the only synchronising calls
 * in the library).
 * ------------------------------------------------------------------------ */
pc_status pc_workspace_status(const void *ws, size_t ws_bytes, void *stream, int32_t *code_out);

/* ------------------------------------------------------------------------
 * Optional per-kernel timing with HIP events on the launch stream.
 * pc_prof_enable(1) makes every later launch record an event pair; after the
 * caller has synchronised, pc_prof_read fills per-kernel launch counts and
 * summed milliseconds (kernels in a fixed internal order) and clears them.
 * Host-side state, not thread-safe.
 * ------------------------------------------------------------------------ */
void pc_prof_enable(int on);
int pc_prof_kernel_count(void);
const char *pc_prof_kernel_name(int i);
pc_status pc_prof_read(uint64_t *launches, double *total_ms, int n);

#ifdef __cplusplus
}
#endif

#endif /* PC_H */
