"""Pins for the CPU oracle: published values, textbook examples, brute force
and invariants that a plausible mistake in the oracle would break.  CPU only."""
import itertools
import random

import numpy as np
import pytest

import oracle
from conftest import characterization_golden, read_golden, request_golden, session_golden

NONE = oracle.NONE
G = 0x9E3779B97F4A7C15
M64 = 2 ** 64 - 1


# ---------------------------------------------------------------- hashing

def test_mix64_matches_published_splitmix64_outputs():
    for k, out in read_golden("splitmix64_seed0.txt"):
        k, out = int(k), int(out, 16)
        assert oracle.mix64((k * G) & M64) == out


def test_step_adds_golden_gamma_after_xor():
    # S(x, w) = mix64((x ^ w) + G): (0,0) -> mix64(G), (G,0) -> mix64(2G),
    # (0, 2G) -> mix64(3G); all three are published splitmix64 outputs.
    outs = {int(k): int(v, 16) for k, v in read_golden("splitmix64_seed0.txt")}
    assert oracle.step(0, 0) == outs[1]
    assert oracle.step(G, 0) == outs[2]
    assert oracle.step(0, (2 * G) & M64) == outs[3]
    assert oracle.step(5, 5) == outs[1]          # x ^ w cancels


def _req(tokens_list):
    toks = np.concatenate([np.asarray(t, np.int32) for t in tokens_list])
    lens = np.array([len(t) for t in tokens_list], np.uint32)
    starts = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.uint64)
    return toks, starts, lens


def test_only_full_blocks_count():
    toks, st, ln = _req([np.arange(33), np.arange(15), np.arange(32)])
    keys, depth = oracle.hash_requests(toks, st, ln, 16)
    assert keys.size == 2 + 0 + 2
    assert list(depth) == [0, 1, 0, 1]


def test_shared_prefix_gives_shared_keys_and_divergence_propagates():
    rng = np.random.default_rng(0)
    base = rng.integers(0, 151936, size=16 * 6).astype(np.int32)
    other = base.copy()
    other[16 * 3 + 5] += 1                      # change one token of block 3
    toks, st, ln = _req([base, other])
    keys, _ = oracle.hash_requests(toks, st, ln, 16)
    a, b = keys[:6], keys[6:]
    assert np.array_equal(a[:3], b[:3])
    assert np.all(a[3:] != b[3:])               # the change reaches every later block


def test_block_position_matters():
    # the same 16 tokens at depth 0 and at depth 1 must not collide
    blk = np.arange(100, 116, dtype=np.int32)
    toks, st, ln = _req([np.concatenate([blk, blk])])
    keys, _ = oracle.hash_requests(toks, st, ln, 16)
    assert keys[0] != keys[1]


def test_word_packing_is_order_sensitive():
    toks, st, ln = _req([[1, 2], [2, 1], [1, 2, 3, 4], [3, 4, 1, 2]])
    keys, _ = oracle.hash_requests(toks, st, ln, 2)
    assert keys[0] != keys[1]
    k4, _ = oracle.hash_requests(toks, st, ln, 4)
    assert k4[0] != k4[1]


def test_parent_chaining_equals_one_pass():
    rng = np.random.default_rng(1)
    t = rng.integers(0, 151936, size=16 * 10).astype(np.int32)
    full, _ = oracle.hash_requests(*_req([t]), 16)
    first, _ = oracle.hash_requests(*_req([t[:16 * 4]]), 16)
    rest, _ = oracle.hash_requests(*_req([t[16 * 4:]]), 16, parent=[first[-1]])
    assert np.array_equal(full, np.concatenate([first, rest]))
    rooted, _ = oracle.hash_requests(*_req([t]), 16, root=123)
    assert np.all(rooted != full)


def _split_words(words):
    """int32 tokens whose packed words (tok[2k] | tok[2k+1] << 32) are `words`."""
    toks = []
    for w in words:
        toks += [w & 0xFFFFFFFF, w >> 32]
    return np.array(toks, np.uint32).view(np.int32)


def _published():
    return {int(k): int(v, 16) for k, v in read_golden("splitmix64_seed0.txt")}


def test_four_token_block_folds_words_in_order_and_chains():
    # Published splitmix64 outputs only: out_k = mix64(k G).  With w0 = 0 the
    # first fold step is S(0, 0) = out1; with w1 = out1 ^ G the second is
    # mix64(2G) = out2, which is the digest; with root = out2 ^ 2G the key is
    # mix64(3G) = out3.  A reversed fold, a hi/lo swap inside a word, or a
    # digest that is not chained from the root would all miss out3.
    out = _published()
    toks = _split_words([0, out[1] ^ G])
    assert oracle.block_digest(toks) == out[2]
    keys, depth = oracle.hash_requests(*_req([toks]), 4, root=out[2] ^ ((2 * G) & M64))
    assert int(keys[0]) == out[3] and list(depth) == [0]
    # the same block under a parent instead of the root
    keys, _ = oracle.hash_requests(*_req([toks]), 4, parent=[out[2] ^ ((2 * G) & M64)])
    assert int(keys[0]) == out[3]


def test_sixteen_token_block_from_published_outputs():
    # Eight words chosen so that the fold visits out1, out2, out3, out1,
    # out3, out2, out2, out1: word k = d_{k-1} ^ (j - 1) G sends the digest
    # to mix64(j G) = out_j.  Then root = out1 ^ 2G gives the key out3.
    out = _published()
    path = [1, 2, 3, 1, 3, 2, 2, 1]
    words, d = [], 0
    for j in path:
        words.append(d ^ (((j - 1) * G) & M64))
        d = out[j]
    toks = _split_words(words)
    assert oracle.block_digest(toks) == out[1]
    keys, _ = oracle.hash_requests(*_req([toks]), 16, root=out[1] ^ ((2 * G) & M64))
    assert int(keys[0]) == out[3]
    # a two-block request: the second block's key chains from the first key
    keys2, depth2 = oracle.hash_requests(*_req([np.concatenate([toks, toks])]), 16,
                                         root=out[1] ^ ((2 * G) & M64))
    assert int(keys2[0]) == out[3] and list(depth2) == [0, 1]
    # reversed word order must not give the same digest
    assert oracle.block_digest(_split_words(words[::-1])) != out[1]


def test_digest_is_fold_over_words_from_zero():
    # a block of B=2 tokens is one word: digest = S(0, w); key = S(root, digest)
    w = 7 | (9 << 32)
    keys, _ = oracle.hash_requests(*_req([[7, 9]]), 2)
    assert int(keys[0]) == oracle.step(0, oracle.step(0, w))


# ---------------------------------------------------------- prev / next

def brute_prev_next(keys):
    n = len(keys)
    prev = [NONE] * n
    nxt = [NONE] * n
    for t in range(n):
        for i in range(t - 1, -1, -1):
            if keys[i] == keys[t]:
                prev[t] = i
                break
        for i in range(t + 1, n):
            if keys[i] == keys[t]:
                nxt[t] = i
                break
    return prev, nxt


def random_streams(count=60, seed=0):
    rng = random.Random(seed)
    for _ in range(count):
        n = rng.randint(0, 120)
        m = rng.randint(1, 30)
        hot = rng.random() < 0.3
        ks = []
        for _ in range(n):
            if hot and rng.random() < 0.5:
                ks.append(1)
            else:
                ks.append(rng.randrange(m) * 0x10001 + 7)
        yield np.array(ks, dtype=np.uint64)


def test_prev_next_brute_force():
    for keys in random_streams():
        p, n = oracle.prev_next(keys)
        bp, bn = brute_prev_next(list(keys))
        assert list(p) == bp and list(n) == bn


# ------------------------------------------------------ stack distances

def brute_distance(keys):
    """Distinct keys strictly between the previous use and t."""
    out = []
    for t, k in enumerate(keys):
        p = None
        for i in range(t - 1, -1, -1):
            if keys[i] == k:
                p = i
                break
        out.append(NONE if p is None else len(set(keys[p + 1:t])))
    return out


def next_form_distance(keys):
    """#{i in (prev(t), t) : next(i) > t}, cold -> NONE."""
    prev, nxt = brute_prev_next(list(keys))
    out = []
    for t in range(len(keys)):
        p = prev[t]
        if p == NONE:
            out.append(NONE)
        else:
            out.append(sum(1 for i in range(p + 1, t) if nxt[i] == NONE or nxt[i] > t))
    return out


def _golden_streams():
    for row in read_golden("stack_distance_examples.txt"):
        bar = row.index("|")
        names = row[1:bar]
        want = [NONE if v == "-" else int(v) for v in row[bar + 1:]]
        ids = {}
        keys = np.array([ids.setdefault(x, len(ids) + 100) for x in names], np.uint64)
        yield row[0], keys, want


def test_hand_worked_examples():
    for name, keys, want in _golden_streams():
        assert list(oracle.stack_distance_walk(keys)) == want, name
        p, _ = oracle.prev_next(keys)
        assert list(oracle.stack_distance_bit(p)) == want, name


def test_walk_and_fenwick_match_brute_force_and_next_form():
    for keys in random_streams(80, seed=3):
        want = brute_distance(list(keys))
        assert list(oracle.stack_distance_walk(keys)) == want
        p, _ = oracle.prev_next(keys)
        assert list(oracle.stack_distance_bit(p)) == want
        assert next_form_distance(keys) == want


# ------------------------------------------------------------- LRU / MIN

def test_textbook_page_replacement_example():
    rows = read_golden("page_replacement_textbook.txt")
    ref = np.array([int(x) + 1 for x in rows[0]], np.uint64)
    frames, lru_faults, opt_faults = (int(x) for x in rows[1])
    (h, _), = oracle.lru(ref, [frames])
    assert ref.size - h == lru_faults
    (b,) = oracle.belady(ref, [frames])
    assert ref.size - b == opt_faults


def test_lru_hit_iff_distance_below_capacity():
    for keys in random_streams(40, seed=5):
        d = oracle.stack_distance_walk(keys)
        caps = [0, 1, 2, 3, 5, 8, 13, 40]
        res = oracle.lru(keys, caps, flags=True)
        prev_flags = None
        for c, (h, _, fl) in zip(caps, res):
            want = (d != NONE) & (d < c)
            assert np.array_equal(fl.astype(bool), want), c
            assert h == int(want.sum())
            if prev_flags is not None:                  # inclusion, per access
                assert np.all(fl >= prev_flags)
            prev_flags = fl


def test_lru_special_capacities():
    for keys in random_streams(40, seed=7):
        n = keys.size
        distinct = len(set(keys.tolist()))
        (h1, _), (hbig, _) = oracle.lru(keys, [1, max(distinct, 1)])
        assert h1 == sum(1 for t in range(1, n) if keys[t] == keys[t - 1])
        assert hbig == n - distinct


def brute_min(keys, cap):
    """Exhaustive offline optimum for demand paging (tiny inputs)."""
    best = 0

    def rec(t, cache, hits):
        nonlocal best
        if t == len(keys):
            best = max(best, hits)
            return
        if hits + (len(keys) - t) <= best:
            return
        k = keys[t]
        if k in cache:
            rec(t + 1, cache, hits + 1)
        elif len(cache) < cap:
            rec(t + 1, cache | {k}, hits)
        else:
            for v in cache:
                rec(t + 1, (cache - {v}) | {k}, hits)

    if cap == 0:
        return 0
    rec(0, frozenset(), 0)
    return best


def test_belady_is_the_exhaustive_optimum():
    rng = random.Random(11)
    for _ in range(40):
        n = rng.randint(1, 11)
        keys = np.array([rng.randrange(5) + 1 for _ in range(n)], np.uint64)
        for c in range(0, 5):
            assert oracle.belady(keys, [c])[0] == brute_min(keys.tolist(), c)


def test_lru_never_beats_belady_and_meets_it_when_everything_fits():
    for keys in random_streams(40, seed=13):
        distinct = len(set(keys.tolist()))
        caps = [1, 2, 4, 8, max(distinct, 1)]
        lru_h = [h for h, _ in oracle.lru(keys, caps)]
        opt_h = oracle.belady(keys, caps)
        assert all(a <= b for a, b in zip(lru_h, opt_h))
        assert lru_h[-1] == opt_h[-1] == keys.size - distinct


# --------------------------------------------------------------- curves

def test_uniform_cost_savings_equal_hit_ratio():
    for keys in random_streams(20, seed=17):
        if keys.size == 0:
            continue
        depth = np.arange(keys.size, dtype=np.uint32) % 7
        caps = [1, 2, 3, 10, 100]
        count, dsum, cost = oracle.mrc_bins(keys, caps, depth, alpha=1, beta=0)
        assert sum(count) == keys.size
        hr, csr = oracle.curves(count, cost)
        assert hr == csr


def test_linear_cost_closed_form_on_one_session():
    # example (ii): contexts of 3, 5, 6 blocks; depth = block index.
    # At capacity 5 (> 4) every re-access hits: hits are depths 0..2 and 0..4.
    # linear cost d+1 -> saved = (1+2+3) + (1+2+3+4+5) = 21, total = 6+15+21 = 42.
    _, keys, _ = [g for g in _golden_streams() if g[0] == "ii"][0]
    depth = np.array([0, 1, 2, 0, 1, 2, 3, 4, 0, 1, 2, 3, 4, 5], np.uint32)
    count, dsum, cost = oracle.mrc_bins(keys, [3, 5], depth, alpha=1, beta=1)
    assert count == [3, 5, 6]           # D=2 re-reads, D=4 re-reads, cold blocks
    hr, csr = oracle.curves(count, cost)
    assert csr[1] == 21 / 42
    assert hr[1] == 8 / 14


def test_nextuse_histogram_brute_force():
    for keys in random_streams(30, seed=19):
        _, nxt = oracle.prev_next(keys)
        caps = [1, 2, 3, 5, 9]
        want = [0] * (len(caps) + 1)
        for t in range(keys.size):
            if nxt[t] == NONE:
                want[-1] += 1
            else:
                gap = int(nxt[t]) - t
                want[sum(1 for c in caps if c <= gap)] += 1
        assert oracle.nextuse_hist(nxt, caps) == want


# --------------------------------------------------- request-level residency

def test_request_level_hand_worked_examples():
    for name, keys, blk_off, want, hits in request_golden():
        assert list(oracle.stack_distance_req_walk(keys, blk_off)) == want, name
        assert list(oracle.stack_distance_req_bit(keys, blk_off)) == want, name
        caps = sorted(hits)
        got = oracle.lru_req(keys, blk_off, caps)
        assert [g[0] for g in got] == [hits[c] for c in caps], name


def random_requests(count, seed):
    """Small multi-turn traces: sessions re-send and extend their context,
    some start from shared prompts, some reset; keys are distinct inside a
    request (as chained prefix hashes are)."""
    rng = np.random.default_rng(seed)
    for _ in range(count):
        n_sess = int(rng.integers(1, 6))
        ctx = {s: [] for s in range(n_sess)}
        shared = {p: [1000 * (p + 1) + d for d in range(int(rng.integers(1, 4)))] for p in range(3)}
        reqs, nxt = [], 1
        for _r in range(int(rng.integers(1, 30))):
            s = int(rng.integers(n_sess))
            if not ctx[s] and rng.random() < 0.3:
                ctx[s] = list(shared[int(rng.integers(3))])
            grow = int(rng.integers(0, 5))
            ctx[s] = ctx[s] + list(range(nxt, nxt + grow))
            nxt += grow
            if rng.random() < 0.1:
                ctx[s] = []
            if ctx[s]:
                reqs.append(list(ctx[s]))
        if not reqs:
            continue
        keys = np.array([k for r in reqs for k in r], np.uint64)
        blk_off = np.concatenate([[0], np.cumsum([len(r) for r in reqs])]).astype(np.uint64)
        yield keys, blk_off


def test_request_level_walk_fenwick_and_simulation_agree():
    """Two exact distance methods agree, and the pinned-request cache hits
    exactly when D_req < c at every feasible capacity (so request-level LRU
    is a stack algorithm there, with inclusion)."""
    for keys, blk_off in random_requests(150, seed=21):
        d = oracle.stack_distance_req_walk(keys, blk_off)
        assert np.array_equal(d, oracle.stack_distance_req_bit(keys, blk_off))
        mx = oracle.max_request_blocks(blk_off)
        caps = list(range(max(mx, 1), mx + 10))
        prev_flags = None
        for c, res in zip(caps, oracle.lru_req(keys, blk_off, caps, flags=True)):
            h, _, fl = res
            want = (d != NONE) & (d < c)
            assert np.array_equal(fl.astype(bool), want), c
            assert h == int(want.sum())
            if prev_flags is not None:
                assert np.all(fl >= prev_flags)   # inclusion
            prev_flags = fl
        if mx > 1:
            assert oracle.lru_req(keys, blk_off, [mx - 1])[0] is None   # infeasible


def test_request_level_equals_per_access_for_single_block_requests():
    for keys in random_streams(60, seed=8):
        blk_off = np.arange(keys.size + 1, dtype=np.uint64)
        assert np.array_equal(oracle.stack_distance_req_walk(keys, blk_off), oracle.stack_distance_walk(keys))


def test_request_level_identity_in_recency_order():
    """In recency order (each request's blocks deepest first), the request
    distance equals the per-access distance minus the earlier accesses of the
    same request whose previous use is older (cold ones included):
    D_req(t) = D(t) - #{j in [s(t), t) : prev(j) + 1 < prev(t) + 1}."""
    for keys, blk_off in random_requests(120, seed=5):
        bo = blk_off.astype(np.int64)
        order = np.concatenate([np.arange(bo[r + 1] - 1, bo[r] - 1, -1) for r in range(bo.size - 1)])
        kp = keys[order]
        p, _ = oracle.prev_next(kp)
        d = oracle.stack_distance_walk(kp)
        v = np.where(p == NONE, 0, p.astype(np.int64) + 1)
        want_p = np.empty(kp.size, np.int64)
        for r in range(bo.size - 1):
            for t in range(bo[r], bo[r + 1]):
                want_p[t] = -1 if p[t] == NONE else int(d[t]) - int((v[bo[r]:t] < v[t]).sum())
        got = oracle.stack_distance_req_walk(keys, blk_off).astype(np.int64)
        got[got == NONE] = -1
        assert np.array_equal(got[order], want_p)


# ------------------------------------------------------- session level

def test_session_level_hand_worked_examples():
    for name, keys, blk_off, sess, want, hits in session_golden():
        assert list(oracle.stack_distance_session_walk(keys, blk_off, sess)) == want, name
        caps = sorted(hits)
        got = oracle.lru_session(keys, blk_off, sess, caps)
        assert [g[0] for g in got] == [hits[c] for c in caps], name


def random_sessions(count, seed, append_only=True):
    """Multi-turn sessions (append-only contexts, some starting from shared
    prompts), or arbitrary requests tagged with sessions; keys distinct
    inside a request."""
    rng = np.random.default_rng(seed)
    for _ in range(count):
        n_sess = int(rng.integers(1, 7))
        ctx = {s: [] for s in range(n_sess)}
        shared = {p: [1000 * (p + 1) + d for d in range(int(rng.integers(1, 4)))] for p in range(2)}
        reqs, sess, nxt = [], [], 1
        for _r in range(int(rng.integers(1, 30))):
            s = int(rng.integers(n_sess))
            if append_only:
                if not ctx[s] and rng.random() < 0.4:
                    ctx[s] = list(shared[int(rng.integers(2))])
                grow = int(rng.integers(0, 4))
                ctx[s] = ctx[s] + list(range(nxt, nxt + grow))
                nxt += grow
                req = list(ctx[s])
            else:
                req = list(rng.choice(40, size=int(rng.integers(0, 6)), replace=False) + 1)
            reqs.append(req)
            sess.append(s)
        keys = np.array([k for r in reqs for k in r], np.uint64)
        if keys.size == 0:
            continue
        blk_off = np.concatenate([[0], np.cumsum([len(r) for r in reqs])]).astype(np.uint64)
        yield keys, blk_off, np.array(sess, np.uint32)


@pytest.mark.parametrize("append_only", [True, False])
def test_session_level_simulation_hits_iff_distance_below_capacity(append_only):
    """Session-level LRU is a stack algorithm: the literal simulation hits
    exactly where the walked distance is below the capacity, per access and
    at every capacity (so inclusion holds)."""
    for keys, blk_off, sess in random_sessions(60, 31 if append_only else 32, append_only):
        d = oracle.stack_distance_session_walk(keys, blk_off, sess).astype(np.int64)
        caps = [0, 1, 2, 3, 4, 6, 9, 13, 20, 40, 1000]
        res = oracle.lru_session(keys, blk_off, sess, caps, flags=True)
        prev = None
        for c, (h, _, fl) in zip(caps, res):
            want = (d != NONE) & (d < c)
            assert np.array_equal(fl.astype(bool), want), c
            assert h == int(want.sum())
            if prev is not None:
                assert np.all(fl >= prev)
            prev = fl


def test_session_level_one_block_sessions_reduce_to_block_lru():
    """Every request one block and every session one key: sessions are
    blocks of size one, so session-level LRU is per-access LRU."""
    rng = np.random.default_rng(5)
    for _ in range(30):
        sess = rng.integers(0, int(rng.integers(1, 12)), size=int(rng.integers(1, 80))).astype(np.uint32)
        keys = sess.astype(np.uint64) * np.uint64(977) + np.uint64(3)
        blk_off = np.arange(sess.size + 1, dtype=np.uint64)
        assert np.array_equal(oracle.stack_distance_session_walk(keys, blk_off, sess),
                              oracle.stack_distance_walk(keys))


def test_session_level_everything_fits():
    """With room for every session's footprint, each block that was used
    before hits."""
    for keys, blk_off, sess in random_sessions(20, 33):
        p, _ = oracle.prev_next(keys)
        (h, _), = oracle.lru_session(keys, blk_off, sess, [int(keys.size) + 1])
        assert h == int((p != NONE).sum())


# ------------------------------------------------------- characterisation

def test_characterization_hand_worked_example():
    keys, blk_off, sess, ts, want = characterization_golden()
    edges = want["edges"]
    rp = oracle.reuse_profile(keys, blk_off, ts, edges, want["freq_max"][0])
    assert rp["interval"] == want["interval"]
    assert rp["lifetime"] == want["lifetime"]
    assert rp["freq"] == want["freq"]
    k = len(edges) + 1
    assert rp["life_by_class"][:k] == want["class0"] and rp["life_by_class"][k:2 * k] == want["class1"]
    assert not any(rp["life_by_class"][2 * k:])
    sp = oracle.session_profile(blk_off, sess, ts, edges, want["footprint_max"][0], want["requests_max"][0])
    for name in ("footprint", "requests", "duration", "gap"):
        assert sp[name] == want[name], name


def _timed_sessions(seed):
    for keys, blk_off, sess in random_sessions(30, seed):
        rng = np.random.default_rng(seed)
        ts = np.cumsum(rng.integers(0, 50, size=sess.size)).astype(np.uint64)
        yield keys, blk_off, sess, ts


def test_characterization_invariants_and_brute_force():
    edges = [1, 3, 10, 30, 100, 300]
    for keys, blk_off, sess, ts in _timed_sessions(51):
        n = keys.size
        rp = oracle.reuse_profile(keys, blk_off, ts, edges, 1000)
        at = oracle.access_times(blk_off, ts)
        # brute force per block: its accesses in order
        acc = {}
        for t, k in enumerate(keys.tolist()):
            acc.setdefault(k, []).append(t)
        assert sum(rp["freq"]) == len(acc)
        assert sum(f * c for f, c in enumerate(rp["freq"])) == n
        assert sum(rp["interval"]) == n - len(acc)
        ivals = [int(at[b]) - int(at[a]) for ts_ in acc.values() for a, b in zip(ts_, ts_[1:])]
        assert rp["interval"] == [int(v) for v in np.bincount(np.searchsorted(edges, ivals, side="right"),
                                                             minlength=len(edges) + 1)]
        lives = [int(at[v[-1]]) - int(at[v[0]]) for v in acc.values()]
        assert rp["lifetime"] == [int(v) for v in np.bincount(np.searchsorted(edges, lives, side="right"),
                                                             minlength=len(edges) + 1)]
        # further-reuse probability after k accesses, counted access by access
        p = oracle.reuse_probability(rp["freq"])
        for k in range(1, 6):
            kth = [len(v) > k for v in acc.values() if len(v) >= k]
            if kth:
                assert p[k - 1] == sum(kth) / len(kth)
        sp = oracle.session_profile(blk_off, sess, ts, edges, 1000, 1000)
        # append-only sessions: the footprint is the number of distinct blocks
        bo = blk_off.astype(np.int64)
        held = {}
        for r, s in enumerate(sess.tolist()):
            held.setdefault(s, set()).update(keys[bo[r]:bo[r + 1]].tolist())
        assert sp["footprint"] == [int(v) for v in np.bincount([len(h) for h in held.values()], minlength=1001)]
        assert sum(sp["gap"]) == sess.size - len(held)


def test_lorenz_top_share_closed_forms():
    # one session with 10 blocks and nine with 1: the top 10% hold 10/19
    h = [0, 9] + [0] * 8 + [1]
    assert oracle.lorenz_top_share(h, 0.1) == 10 / 19
    assert oracle.lorenz_top_share(h, 1.0) == 1.0
    assert oracle.lorenz_top_share([0, 0, 0, 5], 0.4) == 0.4   # equal footprints: share = fraction
