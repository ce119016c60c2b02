"""Plain CPU oracle for the prefix-cache hot path.

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  The product library
never calls it, and it shares no code with it.

Each function states the definition it computes and the passage of the paper
(*When Fancy Eviction Fails*, Liu, Yu & Yang) that fixes it:

* ``hash_requests``: block identity -- a block's KV state is reusable only if
  the whole token sequence before and including it matches (Sec. 2.2); blocks
  are 16 tokens (Sec. 2.2, Sec. 3.1).  The hash itself is not given in the
  paper; the reading used is splitmix64's finalizer as a step function folded
  over token-pair words and chained from the parent block.
* ``prev_next``: previous / next access of the same block; the next-use time
  is what Belady-style analysis ranks by (Sec. 3.2, Sec. 5.2 "BeladyCompute").
* ``lru``: one LRU cache simulated per capacity (Sec. 5 "LRU as a bedrock");
  the block hit ratio counts every access, compulsory misses included
  (Sec. 3.2, Sec. 4.6).
* ``stack_distance_walk`` / ``stack_distance_bit``: the exact LRU stack
  distance (distinct blocks touched since the previous access); Appendix B
  reads "reuses reachable within capacity C" off these distances.
* ``mrc_bins`` / ``curves``: hit ratio and compute-savings ratio -- every hit
  weighted by the recompute cost it avoids, over the cost of all accesses
  (Sec. 5.2 "Compute-awareness"); uniform cost gives the hit ratio back.
* ``belady``: demand-paging MIN per capacity (the offline ceiling, Sec. 3.2).
* ``nextuse_hist``: histogram of next-use gaps ``next(t) - t``.
* ``stack_distance_req_walk`` / ``stack_distance_req_bit`` / ``lru_req`` /
  ``mrc_bins_req``: the same under request-level residency, the paper's
  simulator semantics (Sec. 3.1 "Simulator": all blocks of a request resident
  at once, room made ahead of time); readings: hits decided on arrival, the
  request's deepest block least recent afterwards, capacities below the
  largest request infeasible (Sec. 3.1 "Cache-size regimes").
* ``stack_distance_session_walk`` / ``lru_session`` / ``mrc_bins_session``:
  session-level eviction (Sec. 5.3 "Block-Level vs. Session-Level
  Eviction": whole sessions evicted at once); readings: a session's
  footprint is its largest request so far, sessions are kept in LRU order
  and evicted whole from the least recent end, and a block hits if the
  session that last used it is resident when the request arrives.
"""
from __future__ import annotations

import ctypes
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from . import build as _build

NONE = 0xFFFFFFFF
_lib = None

_u64p = ctypes.POINTER(ctypes.c_uint64)
_u32p = ctypes.POINTER(ctypes.c_uint32)
_i32p = ctypes.POINTER(ctypes.c_int32)
_u8p = ctypes.POINTER(ctypes.c_uint8)


def lib():
    global _lib
    if _lib is None:
        path = _build.build(force=False)
        L = ctypes.CDLL(path)
        L.orc_mix64.restype = ctypes.c_uint64
        L.orc_mix64.argtypes = [ctypes.c_uint64]
        L.orc_step.restype = ctypes.c_uint64
        L.orc_step.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        L.orc_block_digest.restype = ctypes.c_uint64
        L.orc_block_digest.argtypes = [_i32p, ctypes.c_uint32]
        L.orc_hash_requests.restype = ctypes.c_uint64
        L.orc_hash_requests.argtypes = [_i32p, _u64p, _u32p, ctypes.c_uint64, ctypes.c_uint32,
                                        _u64p, ctypes.c_uint64, _u64p, _u32p]
        L.orc_key_ids.restype = ctypes.c_uint64
        L.orc_key_ids.argtypes = [_u64p, ctypes.c_uint64, _u32p]
        L.orc_prev_next.restype = ctypes.c_int
        L.orc_prev_next.argtypes = [_u32p, ctypes.c_uint64, ctypes.c_uint64, _u32p, _u32p]
        L.orc_stack_distance_walk.restype = ctypes.c_int
        L.orc_stack_distance_walk.argtypes = [_u32p, ctypes.c_uint64, ctypes.c_uint64, _u32p]
        L.orc_stack_distance_bit.restype = ctypes.c_int
        L.orc_stack_distance_bit.argtypes = [_u32p, ctypes.c_uint64, _u32p]
        L.orc_lru_sim.restype = ctypes.c_int
        L.orc_lru_sim.argtypes = [_u32p, _u32p, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                                  _u64p, _u64p, _u8p, _u64p]
        L.orc_fp_u32.restype = ctypes.c_uint64
        L.orc_fp_u32.argtypes = [_u32p, ctypes.c_uint64, ctypes.c_uint64]
        L.orc_dist_bins.restype = ctypes.c_int
        L.orc_dist_bins.argtypes = [_u32p, ctypes.c_uint64, ctypes.c_uint64, _u64p, ctypes.c_uint32, _u64p, _u64p]
        L.orc_fp_u64.restype = ctypes.c_uint64
        L.orc_fp_u64.argtypes = [_u64p, ctypes.c_uint64, ctypes.c_uint64]
        L.orc_stack_distance_req_walk.restype = ctypes.c_int
        L.orc_stack_distance_req_walk.argtypes = [_u32p, _u64p, ctypes.c_uint64, ctypes.c_uint64, _u32p]
        L.orc_stack_distance_req_bit.restype = ctypes.c_int
        L.orc_stack_distance_req_bit.argtypes = [_u32p, _u64p, ctypes.c_uint64, ctypes.c_uint64, _u32p]
        L.orc_session_sim.restype = ctypes.c_int
        L.orc_session_sim.argtypes = [_u32p, _u32p, _u64p, _u32p, ctypes.c_uint64, ctypes.c_uint64,
                                      ctypes.c_uint64, ctypes.c_uint64, _u64p, _u64p, _u8p]
        L.orc_stack_distance_session_walk.restype = ctypes.c_int
        L.orc_stack_distance_session_walk.argtypes = [_u32p, _u64p, _u32p, ctypes.c_uint64, ctypes.c_uint64,
                                                      ctypes.c_uint64, _u32p]
        L.orc_lru_sim_req.restype = ctypes.c_int
        L.orc_lru_sim_req.argtypes = [_u32p, _u32p, _u64p, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                                      _u64p, _u64p, _u8p]
        L.orc_belady_sim.restype = ctypes.c_int
        L.orc_belady_sim.argtypes = [_u32p, _u32p, ctypes.c_uint64, ctypes.c_uint64,
                                     ctypes.c_uint64, _u64p, _u8p]
        _lib = L
    return _lib


def _p(a: np.ndarray, t):
    return a.ctypes.data_as(t)


def _c(a, dtype):
    return np.ascontiguousarray(np.asarray(a), dtype=dtype)


def mix64(z: int) -> int:
    return int(lib().orc_mix64(z & (2 ** 64 - 1)))


def step(x: int, w: int) -> int:
    return int(lib().orc_step(x & (2 ** 64 - 1), w & (2 ** 64 - 1)))


def block_digest(tokens):
    """Digest of one block: S folded over its token-pair words from 0."""
    t = _c(tokens, np.int32)
    if t.size < 2 or t.size % 2:
        raise ValueError("a block has an even number of tokens")
    return int(lib().orc_block_digest(_p(t, _i32p), t.size))


def hash_requests(tokens, tok_start, tok_len, block_size=16, parent=None, root=0, threads=1):
    """Keys and depths of every full block of every request, request-major.

    key(b) = S(key(b-1), digest(block b)), key(-1) = root or parent[r];
    digest = S folded over the block's token-pair words from 0;
    S(x, w) = mix64((x xor w) + 0x9E3779B97F4A7C15).
    With threads > 1, contiguous ranges of requests are hashed by separate
    threads into their own slices of the output (requests are independent)."""
    if block_size < 2 or block_size % 2:
        raise ValueError("block size must be even and >= 2")
    tokens = _c(tokens, np.int32)
    tok_start = _c(tok_start, np.uint64)
    tok_len = _c(tok_len, np.uint32)
    nb = tok_len.astype(np.uint64) // np.uint64(block_size)
    off = np.zeros(tok_len.size + 1, np.uint64)
    np.cumsum(nb, out=off[1:])
    n = int(off[-1])
    keys = np.empty(n, np.uint64)
    depth = np.empty(n, np.uint32)
    par = _c(parent, np.uint64) if parent is not None else None

    def part(r0, r1):
        o = int(off[r0])
        got = lib().orc_hash_requests(
            _p(tokens, _i32p), _p(tok_start[r0:r1], _u64p), _p(tok_len[r0:r1], _u32p), r1 - r0, block_size,
            _p(par[r0:r1], _u64p) if par is not None else None, root, _p(keys[o:], _u64p),
            _p(depth[o:], _u32p))
        assert got == int(off[r1]) - o

    R = tok_len.size
    if threads <= 1 or R < 2 * threads:
        if R:
            part(0, R)
    else:
        # split by accesses, so every thread gets about the same work
        cuts = np.searchsorted(off, np.linspace(0, n, threads + 1)[1:-1].astype(np.uint64))
        bounds = [0] + sorted(set(int(c) for c in cuts)) + [R]
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(lambda ab: part(*ab), [(a, b) for a, b in zip(bounds[:-1], bounds[1:]) if b > a]))
    return keys, depth


def fingerprint(a, t0=0):
    """sum over t of mix64(mix64(t0 + t + 1) + a[t]) mod 2^64 for a uint32 or
    uint64 array (a whole-array check for arrays too large to store)."""
    a = np.asarray(a)
    if a.dtype in (np.uint32, np.int32):
        a = _c(a.view(np.uint32) if a.dtype == np.int32 else a, np.uint32)
        return int(lib().orc_fp_u32(_p(a, _u32p), a.size, t0))
    a = _c(a.view(np.uint64) if a.dtype == np.int64 else a, np.uint64)
    return int(lib().orc_fp_u64(_p(a, _u64p), a.size, t0))


def hash_trace(trace, block_size=None, threads=1):
    return hash_requests(trace.tokens, trace.tok_start, trace.tok_len,
                         block_size or trace.block_size, threads=threads)


def key_ids(keys):
    keys = _c(keys, np.uint64)
    ids = np.empty(keys.size, np.uint32)
    n_ids = lib().orc_key_ids(_p(keys, _u64p), keys.size, _p(ids, _u32p))
    if n_ids == 2 ** 64 - 1:
        raise MemoryError("oracle dictionary")
    return ids, int(n_ids)


def prev_next(keys, ids=None):
    if ids is None:
        ids = key_ids(keys)
    id_, n_ids = ids
    prev = np.empty(id_.size, np.uint32)
    nxt = np.empty(id_.size, np.uint32)
    assert lib().orc_prev_next(_p(id_, _u32p), id_.size, n_ids, _p(prev, _u32p), _p(nxt, _u32p)) == 0
    return prev, nxt


def stack_distance_walk(keys, ids=None):
    """Exact D by walking the MRU list (O(N*D), small traces only)."""
    if ids is None:
        ids = key_ids(keys)
    id_, n_ids = ids
    d = np.empty(id_.size, np.uint32)
    assert lib().orc_stack_distance_walk(_p(id_, _u32p), id_.size, n_ids, _p(d, _u32p)) == 0
    return d


def stack_distance_bit(prev):
    """Exact D from prev[] with a Fenwick tree over last-occurrence marks."""
    prev = _c(prev, np.uint32)
    d = np.empty(prev.size, np.uint32)
    assert lib().orc_stack_distance_bit(_p(prev, _u32p), prev.size, _p(d, _u32p)) == 0
    return d


def lru(keys, caps, depth=None, ids=None, flags=False, threads=1, fingerprints=False):
    """Per capacity: (hits, sum of depth over hits[, fingerprint][, per-access
    hit flags]); the fingerprint is the sum of mix64(t + 1) over the hits t.
    With threads > 1 the capacities are simulated concurrently, one
    simulation per thread (each is the same single-threaded list walk)."""
    if ids is None:
        ids = key_ids(keys)
    id_, n_ids = ids
    dep = _c(depth, np.uint32) if depth is not None else None

    def one(c):
        h = ctypes.c_uint64(0)
        dh = ctypes.c_uint64(0)
        fp = ctypes.c_uint64(0)
        fl = np.empty(id_.size, np.uint8) if flags else None
        assert lib().orc_lru_sim(_p(id_, _u32p), _p(dep, _u32p) if dep is not None else None,
                                 id_.size, n_ids, int(c), ctypes.byref(h), ctypes.byref(dh),
                                 _p(fl, _u8p) if fl is not None else None,
                                 ctypes.byref(fp) if fingerprints else None) == 0
        r = (h.value, dh.value) + ((fp.value,) if fingerprints else ())
        return r + (fl,) if flags else r

    return _per_capacity(one, caps, threads)


def belady(keys, caps, ids=None, nxt=None, flags=False, threads=1):
    """Hits of demand-paging MIN at each capacity (Sec. 3.2: the offline
    ceiling): every access brings its block in, and a full cache evicts the
    resident block whose next use is farthest (never used again counts as
    farthest).  With ``flags`` also the per-access hit flags."""
    if ids is None:
        ids = key_ids(keys)
    id_, n_ids = ids
    if nxt is None:
        _, nxt = prev_next(keys, ids)
    nxt = _c(nxt, np.uint32)

    def one(c):
        h = ctypes.c_uint64(0)
        fl = np.empty(id_.size, np.uint8) if flags else None
        assert lib().orc_belady_sim(_p(id_, _u32p), _p(nxt, _u32p), id_.size, n_ids, int(c),
                                    ctypes.byref(h), _p(fl, _u8p) if fl is not None else None) == 0
        return (h.value, fl) if flags else h.value

    return _per_capacity(one, caps, threads)


def mrc_bins(keys, caps, depth=None, alpha=1, beta=0, ids=None, threads=1):
    """Bins over the capacity edges, from one LRU simulation per capacity.

    Bin k (k < K) holds the accesses that hit at caps[k] but not at the
    previous edge; bin K holds the accesses that miss at every capacity
    (cold or too far).  Returns python-int lists count[K+1], depthsum[K+1],
    cost[K+1] with cost = alpha*count + beta*depthsum (exact integers)."""
    keys = _c(keys, np.uint64)
    n = keys.size
    if depth is None:
        depth = np.zeros(n, np.uint32)
    res = lru(keys, caps, depth, ids, threads=threads)
    count, dsum = [], []
    ph, pd = 0, 0
    for h, dh in res:
        count.append(h - ph)
        dsum.append(dh - pd)
        ph, pd = h, dh
    count.append(n - ph)
    dsum.append(int(np.asarray(depth, np.uint64).sum(dtype=np.uint64)) - pd)
    cost = [alpha * c + beta * d for c, d in zip(count, dsum)]
    return count, dsum, cost


def curves(count, cost):
    """Cumulative hit ratio and compute-savings ratio at each capacity edge.

    HR(c_k) = hits(c_k) / N, CSR(c_k) = saved(c_k) / total cost, both from
    exact integers rounded once to float64 before one division."""
    n = sum(count)
    total = sum(cost)
    hr, csr = [], []
    h, s = 0, 0
    for k in range(len(count) - 1):
        h += count[k]
        s += cost[k]
        hr.append(float(h) / float(n) if n else 0.0)
        csr.append(float(s) / float(total) if total else 0.0)
    return hr, csr


def nextuse_hist(nxt, caps, t0=0):
    """Histogram of next(t) - t over the capacity edges (never reused -> last
    bin); bin k = number of edges <= gap.  ``nxt`` may be the slice of a
    longer array that starts at position t0."""
    nxt = np.asarray(nxt, np.uint32)
    t = np.arange(t0, t0 + nxt.size, dtype=np.uint64)
    caps = np.asarray(caps, np.uint64)
    hist = [0] * (caps.size + 1)
    none = nxt == NONE
    gap = nxt.astype(np.uint64) - t
    k = np.searchsorted(caps, gap[~none], side="right")
    bc = np.bincount(k, minlength=caps.size + 1)
    for i in range(caps.size + 1):
        hist[i] = int(bc[i])
    hist[caps.size] += int(none.sum())
    return hist


def dist_bins(dist, caps, t0=0, count=None, fp=None):
    """Capacity bins of a distance array (the pc_mrc_weighted convention)
    and, per bin, the sum of mix64(t + 1) over its accesses t.  Prefix sums
    give the hits and the hit-set fingerprint at every capacity.  Adds into
    ``count`` / ``fp`` (uint64[K+1]) when given, so a long array can be
    binned in pieces; returns them."""
    d = _c(dist, np.uint32)
    cp = _c(caps, np.uint64)
    k = cp.size
    count = np.zeros(k + 1, np.uint64) if count is None else count
    fp = np.zeros(k + 1, np.uint64) if fp is None else fp
    assert lib().orc_dist_bins(_p(d, _u32p), d.size, t0, _p(cp, _u64p), k, _p(count, _u64p), _p(fp, _u64p)) == 0
    return count, fp


# ------------------------------------------------------------ request level

def _req(blk_off):
    blk_off = _c(blk_off, np.uint64)
    return blk_off, blk_off.size - 1


def stack_distance_req_walk(keys, blk_off, ids=None):
    """Request-level distance of every access (depth order within each
    request) by walking the recency list: distinct blocks above the block
    when its request arrives; NONE if never used before."""
    if ids is None:
        ids = key_ids(keys)
    id_, n_ids = ids
    bo, ns = _req(blk_off)
    d = np.empty(id_.size, np.uint32)
    rc = lib().orc_stack_distance_req_walk(_p(id_, _u32p), _p(bo, _u64p), ns, n_ids, _p(d, _u32p))
    if rc == -2:
        raise ValueError("a key repeats inside one request")
    assert rc == 0
    return d


def stack_distance_req_bit(keys, blk_off, ids=None):
    """Same, with a Fenwick tree over last-use marks in recency time."""
    if ids is None:
        ids = key_ids(keys)
    id_, n_ids = ids
    bo, ns = _req(blk_off)
    d = np.empty(id_.size, np.uint32)
    assert lib().orc_stack_distance_req_bit(_p(id_, _u32p), _p(bo, _u64p), ns, n_ids, _p(d, _u32p)) == 0
    return d


def lru_req(keys, blk_off, caps, depth=None, ids=None, flags=False, threads=1):
    """Per capacity: (hits, depth sum over hits[, flags]) of a request-level
    LRU cache, or None where the capacity is below the largest request."""
    if ids is None:
        ids = key_ids(keys)
    id_, n_ids = ids
    bo, ns = _req(blk_off)
    dep = _c(depth, np.uint32) if depth is not None else None

    def one(c):
        h = ctypes.c_uint64(0)
        dh = ctypes.c_uint64(0)
        fl = np.empty(id_.size, np.uint8) if flags else None
        rc = lib().orc_lru_sim_req(_p(id_, _u32p), _p(dep, _u32p) if dep is not None else None, _p(bo, _u64p),
                                   ns, n_ids, int(c), ctypes.byref(h), ctypes.byref(dh),
                                   _p(fl, _u8p) if fl is not None else None)
        if rc == -3:
            return None
        assert rc == 0
        return (h.value, dh.value, fl) if flags else (h.value, dh.value)

    return _per_capacity(one, caps, threads)


def _per_capacity(one, caps, threads):
    """[one(c) for c in caps], on a thread pool when threads > 1 (each call
    is one single-threaded simulation; ctypes releases the GIL)."""
    caps = list(caps)
    if threads <= 1 or len(caps) <= 1:
        return [one(c) for c in caps]
    with ThreadPoolExecutor(min(threads, len(caps))) as ex:
        return list(ex.map(one, caps))


def max_request_blocks(blk_off):
    bo = np.asarray(blk_off, np.uint64)
    return int((bo[1:] - bo[:-1]).max()) if bo.size > 1 else 0


def mrc_bins_req(keys, blk_off, caps, depth=None, alpha=1, beta=0, ids=None, threads=1):
    """Bins over the capacity edges from one request-level simulation per
    capacity.  Only feasible edges (>= the largest request) are simulated;
    the bins of infeasible edges hold the accesses whose request-level
    distance lies below them, which is what the GPU reports for them, so
    they are filled from the walk instead and flagged by the caller."""
    keys = _c(keys, np.uint64)
    n = keys.size
    if depth is None:
        depth = np.zeros(n, np.uint32)
    caps = [int(c) for c in caps]
    mx = max_request_blocks(blk_off)
    feas = [c >= mx and c > 0 for c in caps]
    sim = lru_req(keys, blk_off, [c for c, f in zip(caps, feas) if f], depth, ids, threads=threads)
    it = iter(sim)
    res = []
    d = None
    for c, f in zip(caps, feas):
        if f:
            res.append(next(it))
        else:
            if d is None:
                d = stack_distance_req_walk(keys, blk_off, ids).astype(np.int64)
                d[d == NONE] = -1
            hit = (d >= 0) & (d < c)
            res.append((int(hit.sum()), int(np.asarray(depth, np.uint64)[hit].sum())))
    count, dsum = [], []
    ph, pd = 0, 0
    for h, dh in res:
        count.append(h - ph)
        dsum.append(dh - pd)
        ph, pd = h, dh
    count.append(n - ph)
    dsum.append(int(np.asarray(depth, np.uint64).sum(dtype=np.uint64)) - pd)
    cost = [alpha * c + beta * d for c, d in zip(count, dsum)]
    return count, dsum, cost, feas


def _sess(sess, n_seqs):
    sess = _c(sess, np.uint32)
    assert sess.size == n_seqs
    return sess, (int(sess.max()) + 1 if sess.size else 0)


def stack_distance_session_walk(keys, blk_off, sess, ids=None):
    """Session-level distance of every access by walking the session recency
    list: footprints of the session that last used the block and of every
    session above it, less one; NONE if the block was never used before."""
    if ids is None:
        ids = key_ids(keys)
    id_, n_ids = ids
    bo, ns = _req(blk_off)
    sv, n_sess = _sess(sess, ns)
    d = np.empty(id_.size, np.uint32)
    assert lib().orc_stack_distance_session_walk(_p(id_, _u32p), _p(bo, _u64p), _p(sv, _u32p), ns, n_ids,
                                                 n_sess, _p(d, _u32p)) == 0
    return d


def lru_session(keys, blk_off, sess, caps, depth=None, ids=None, flags=False, threads=1):
    """Per capacity: (hits, depth sum over hits[, flags]) of a session-level
    LRU cache simulated literally."""
    if ids is None:
        ids = key_ids(keys)
    id_, n_ids = ids
    bo, ns = _req(blk_off)
    sv, n_sess = _sess(sess, ns)
    dep = _c(depth, np.uint32) if depth is not None else None

    def one(c):
        h = ctypes.c_uint64(0)
        dh = ctypes.c_uint64(0)
        fl = np.empty(id_.size, np.uint8) if flags else None
        assert lib().orc_session_sim(_p(id_, _u32p), _p(dep, _u32p) if dep is not None else None, _p(bo, _u64p),
                                     _p(sv, _u32p), ns, n_ids, n_sess, int(c), ctypes.byref(h), ctypes.byref(dh),
                                     _p(fl, _u8p) if fl is not None else None) == 0
        return (h.value, dh.value, fl) if flags else (h.value, dh.value)

    return _per_capacity(one, caps, threads)


def mrc_bins_session(keys, blk_off, sess, caps, depth=None, alpha=1, beta=0, ids=None, threads=1):
    """Bins over the capacity edges from one session-level simulation per
    capacity (same layout as ``mrc_bins``)."""
    keys = _c(keys, np.uint64)
    n = keys.size
    if depth is None:
        depth = np.zeros(n, np.uint32)
    res = lru_session(keys, blk_off, sess, caps, depth, ids, threads=threads)
    count, dsum = [], []
    ph, pd = 0, 0
    for h, dh in res:
        count.append(h - ph)
        dsum.append(dh - pd)
        ph, pd = h, dh
    count.append(n - ph)
    dsum.append(int(np.asarray(depth, np.uint64).sum(dtype=np.uint64)) - pd)
    cost = [alpha * c + beta * d for c, d in zip(count, dsum)]
    return count, dsum, cost


# ------------------------------------------------------------- f4 profiles
# Workload characterisation (Sec. 4): reuse intervals in time (Sec. 4.2),
# block lifetimes (Sec. 4.1), access frequency and the chance of a further
# reuse after k accesses (Sec. 4.3), per-session footprints, turns, duration
# and inter-request gaps (Sec. 4.5, Sec. 4.1, Sec. 2.3).  Times are request
# timestamps in microseconds; a block's accesses take their request's time.
# Histograms use the capacity-bin convention: bin k < K holds values in
# [edges[k-1], edges[k]) (edges[-1] = 0), bin K holds values >= edges[K-1].

def _bins(x, edges):
    return np.searchsorted(np.asarray(edges, np.uint64), np.asarray(x, np.uint64), side="right")


def _hist(x, edges):
    return [int(v) for v in np.bincount(_bins(x, edges), minlength=len(edges) + 1)]


def access_times(blk_off, ts_us):
    """Timestamp of every access: its request's."""
    bo = np.asarray(blk_off, np.int64)
    return np.repeat(np.asarray(ts_us, np.uint64), np.diff(bo))


def reuse_profile(keys, blk_off, ts_us, edges, freq_max):
    """Per-block and per-reuse statistics of an access stream.

    interval: histogram over reuses t (prev(t) exists) of ts(t) - ts(prev t);
    lifetime: histogram over blocks of ts(last access) - ts(first access);
    freq: blocks by number of accesses f, bin min(f, freq_max) (bin 0 empty);
    life_by_class: lifetime histogram per frequency class floor(log2 f)
    (32 classes, flattened class-major)."""
    keys = _c(keys, np.uint64)
    ids, n_ids = key_ids(keys)
    prev, _ = prev_next(keys, (ids, n_ids))
    ts = access_times(blk_off, ts_us)
    has = prev != NONE
    interval = ts[has] - ts[prev[has]]
    order = np.arange(keys.size)
    first = np.full(n_ids, keys.size, np.int64)
    np.minimum.at(first, ids, order)
    last = np.full(n_ids, -1, np.int64)
    np.maximum.at(last, ids, order)
    count = np.bincount(ids, minlength=n_ids)
    life = ts[last] - ts[first]
    cls = np.floor(np.log2(count)).astype(np.int64)
    k = len(edges) + 1
    lb = np.zeros(32 * k, np.int64)
    np.add.at(lb, cls * k + _bins(life, edges), 1)
    return {"interval": _hist(interval, edges), "lifetime": _hist(life, edges),
            "freq": [int(v) for v in np.bincount(np.minimum(count, freq_max), minlength=freq_max + 1)],
            "life_by_class": [int(v) for v in lb]}


def reuse_probability(freq):
    """P(a block is accessed again | it has been accessed k times) for
    k = 1 .. len(freq) - 2, from the frequency histogram (exact below the
    tail bin): blocks with f >= k+1 over blocks with f >= k."""
    f = np.asarray(freq, np.int64)
    at_least = np.cumsum(f[::-1])[::-1]          # blocks with f >= k (tail bin counts as >= F)
    return [float(at_least[k + 1]) / float(at_least[k]) if at_least[k] else 0.0 for k in range(1, f.size - 1)]


def session_profile(blk_off, sess, ts_us, edges, fp_max, rq_max):
    """Per-session statistics from the request table.

    footprint: sessions by footprint, the largest request's block count
    (append-only contexts), bin min(fp, fp_max); requests: sessions by
    number of requests, bin min(count, rq_max); duration: histogram of
    ts(last request) - ts(first request); gap: histogram over requests with
    an earlier request of the same session of the time since that one."""
    bo = np.asarray(blk_off, np.int64)
    m = np.diff(bo)
    sess = np.asarray(sess, np.int64)
    ts = np.asarray(ts_us, np.uint64)
    fp, cnt, t0, t1, last = {}, {}, {}, {}, {}
    gaps = []
    for r in range(sess.size):
        s = int(sess[r])
        fp[s] = max(fp.get(s, 0), int(m[r]))
        cnt[s] = cnt.get(s, 0) + 1
        t0.setdefault(s, int(ts[r]))
        t1[s] = int(ts[r])
        if s in last:
            gaps.append(int(ts[r]) - last[s])
        last[s] = int(ts[r])
    ss = sorted(fp)
    return {"footprint": [int(v) for v in np.bincount(np.minimum([fp[s] for s in ss], fp_max),
                                                      minlength=fp_max + 1)],
            "requests": [int(v) for v in np.bincount(np.minimum([cnt[s] for s in ss], rq_max),
                                                     minlength=rq_max + 1)],
            "duration": _hist([t1[s] - t0[s] for s in ss], edges),
            "gap": _hist(gaps, edges)}


def lorenz_top_share(footprint_hist, frac):
    """Share of all footprint blocks held by the largest ceil(frac * S)
    sessions, from an exact footprint histogram (no tail sessions)."""
    h = np.asarray(footprint_hist, np.int64)
    total_s = int(h.sum())
    total_b = int((h * np.arange(h.size)).sum())
    want = int(np.ceil(frac * total_s))
    got_s = got_b = 0
    for v in range(h.size - 1, -1, -1):
        take = min(int(h[v]), want - got_s)
        got_s += take
        got_b += take * v
        if got_s == want:
            break
    return got_b / total_b if total_b else 0.0
