"""Parity of the HIP path (through the C ABI) against the CPU oracle.

Every stage is checked on its own, fed with the oracle's inputs, and then end
to end.  Integer outputs (keys, prev/next, distances, bins, 128-bit costs)
must be bit-exact; the float64 ratios are formed from the exact integers and
must agree to 1e-12 relative (they come out identical)."""
import sys

import numpy as np
import pytest
import torch

import oracle
import pcgen
from paper_2609_28870_amd import pc

pytestmark = pytest.mark.gpu
NONE = pc.NONE
CUSTOM_COSTS = [(1, 0), (2 * 16 * 3_000_000_000, 2 * 16 * 16), (1, 1)]   # uniform, literal, linear(d+1)


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def gpu_hash(trace, B=16, parent=None, root=0):
    up = pc.upload_trace(trace, B)
    par = pc.to_dev_u64(parent) if parent is not None else None
    keys, depth, ws = pc.hash_blocks(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"],
                                     up["n_blocks"], B, parent=par, root=root)
    assert pc.workspace_status(ws) == 0
    return pc.as_u64(keys), pc.as_u32(depth)


LAST_HIGH_KEY = [None]   # whether the last gpu_prev_next needed the high key bits


def gpu_prev_next(keys_np):
    keys = pc.to_dev_u64(keys_np)
    prev, nxt, ws = pc.prev_next_use(keys)
    assert pc.workspace_status(ws) == 0
    LAST_HIGH_KEY[0] = pc.high_key_passes_ran(ws)
    return pc.as_u32(prev), pc.as_u32(nxt)


def gpu_dist(prev_np, next_np):
    dist, ws = pc.stack_distance(pc.to_dev_u32(prev_np), pc.to_dev_u32(next_np))
    assert pc.workspace_status(ws) == 0
    return pc.as_u32(dist)


def gpu_bins(dist_np, caps, depth_np=None, next_np=None, alpha=1, beta=0):
    out, ws = pc.mrc_weighted(pc.to_dev_u32(dist_np), pc.to_dev_u64(caps),
                              pc.to_dev_u32(depth_np) if depth_np is not None else None,
                              pc.to_dev_u32(next_np) if next_np is not None else None, alpha, beta)
    assert pc.workspace_status(ws) == 0
    return pc.bins_to_host(out)


def check_keys_path(keys, depth=None, caps=None, label=""):
    """prev/next, distances and bins of a key stream against the oracle."""
    n = keys.size
    say("case", label, "n", n)
    ids = oracle.key_ids(keys)
    op, on = oracle.prev_next(keys, ids)
    gp, gn = gpu_prev_next(keys)
    assert np.array_equal(gp, op), label + " prev"
    assert np.array_equal(gn, on), label + " next"
    od = oracle.stack_distance_bit(op)
    gd = gpu_dist(op, on)
    bad = np.nonzero(gd != od)[0]
    assert bad.size == 0, "%s dist: %d mismatches, first t=%s gpu=%s want=%s" % (
        label, bad.size, bad[:5], gd[bad[:5]], od[bad[:5]])
    if caps is not None:
        dep = depth if depth is not None else np.zeros(n, np.uint32)
        for a, b in CUSTOM_COSTS:
            cnt, dsum, cost = oracle.mrc_bins(keys, caps, dep, a, b, ids)
            g = gpu_bins(od, caps, dep, on, a, b)
            assert g["count"] == cnt and g["depthsum"] == dsum and g["cost"] == cost, (label, a, b)
            assert g["nextuse"] == oracle.nextuse_hist(on, caps)
            hr, csr = pc.curves(g["count"], g["cost"])
            ohr, ocsr = oracle.curves(cnt, cost)
            np.testing.assert_allclose(hr, ohr, rtol=1e-12, atol=0)
            np.testing.assert_allclose(csr, ocsr, rtol=1e-12, atol=0)
    return od


# ------------------------------------------------------------------ stages

def test_hash_tiny_trace_bit_exact():
    tr = pcgen.make_trace("tiny")
    ok, od = oracle.hash_trace(tr)
    gk, gd = gpu_hash(tr)
    assert np.array_equal(gk, ok) and np.array_equal(gd, od)


@pytest.mark.parametrize("B", [32, 48, 64, 256])
def test_hash_multiples_of_16_aligned_and_not(B):
    # 16-byte aligned streams take 16-byte loads, streams shifted by one token
    # the scalar path; both must give the oracle's keys
    tr = pcgen.make_trace("tiny")
    ok, od = oracle.hash_trace(tr, B)
    gk, gd = gpu_hash(tr, B)
    assert np.array_equal(gk, ok) and np.array_equal(gd, od)
    tr2 = pcgen.subtrace(tr, 0, tr.n_requests)
    tr2.tok_start = tr.tok_start + np.uint64(1)
    tr2.tok_len = np.where(tr.tok_len > 0, tr.tok_len - 1, 0).astype(np.uint32)
    tr2.tokens = np.concatenate([tr.tokens, np.zeros(1, np.int32)])
    ok2, od2 = oracle.hash_trace(tr2, B)
    gk2, gd2 = gpu_hash(tr2, B)
    assert np.array_equal(gk2, ok2) and np.array_equal(gd2, od2)


@pytest.mark.parametrize("B", [2, 6, 64, 256])
def test_hash_other_block_sizes(B):
    tr = pcgen.make_trace("tiny")
    ok, od = oracle.hash_trace(tr, B)
    gk, gd = gpu_hash(tr, B)
    assert np.array_equal(gk, ok) and np.array_equal(gd, od)


def test_hash_unaligned_views_parent_and_root():
    tr = pcgen.make_trace("tiny")
    r = tr.n_requests
    # shift every request by one token (4-byte aligned only) and give parents
    tr2 = pcgen.subtrace(tr, 0, r)
    tr2.tok_start = tr.tok_start + np.uint64(1)
    tr2.tok_len = np.maximum(tr.tok_len.astype(np.int64) - 1, 0).astype(np.uint32)
    parent = (np.arange(r, dtype=np.uint64) * np.uint64(0x9E3779B97F4A7C15))
    ok, _ = oracle.hash_requests(tr2.tokens, tr2.tok_start, tr2.tok_len, 16, parent=parent)
    gk, _ = gpu_hash(tr2, 16, parent=parent)
    assert np.array_equal(gk, ok)
    ok, _ = oracle.hash_requests(tr.tokens, tr.tok_start, tr.tok_len, 16, root=77)
    gk, _ = gpu_hash(tr, 16, root=77)
    assert np.array_equal(gk, ok)


def low_byte_hist(keys):
    k = np.asarray(keys, np.uint64)
    return np.concatenate([np.bincount(((k >> np.uint64(8 * p)) & np.uint64(0xFF)).astype(np.int64),
                                       minlength=256) for p in range(4)])


def test_hash_counts_the_key_byte_histogram():
    tr = pcgen.make_trace("tiny")
    keys, _ = oracle.hash_trace(tr)
    up = pc.upload_trace(tr, 16)
    hist = torch.empty(1024, dtype=torch.int32, device="cuda")
    gk, _, ws = pc.hash_blocks(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"], 16,
                               key_hist=hist)
    assert pc.workspace_status(ws) == 0
    assert np.array_equal(pc.as_u64(gk), keys)
    assert np.array_equal(pc.as_u32(hist).astype(np.int64), low_byte_hist(keys))


@pytest.mark.parametrize("kind", ["mixed", "lowsame"])
def test_prev_next_with_a_given_histogram(kind):
    keys = stream(kind, 70001, 5)
    hist = pc.to_dev_u32(low_byte_hist(keys).astype(np.uint32))
    prev, nxt, ws = pc.prev_next_use(pc.to_dev_u64(keys), key_hist=hist)
    assert pc.workspace_status(ws) == 0
    op, on = oracle.prev_next(keys)
    assert np.array_equal(pc.as_u32(prev), op) and np.array_equal(pc.as_u32(nxt), on)


def test_prev_next_reports_a_wrong_histogram():
    keys = stream("mixed", 20000, 6)
    h = low_byte_hist(keys)
    short = h.copy()
    short[3] -= 1                       # a row that does not sum to n
    _, _, ws = pc.prev_next_use(pc.to_dev_u64(keys), key_hist=pc.to_dev_u32(short.astype(np.uint32)))
    assert pc.workspace_status(ws) == 4
    moved = h.copy()
    d = int(np.nonzero(moved[:256])[0][0])
    moved[d] -= 1
    moved[(d + 1) % 256] += 1           # sums to n, but not these keys' counts
    _, _, ws = pc.prev_next_use(pc.to_dev_u64(keys), key_hist=pc.to_dev_u32(moved.astype(np.uint32)))
    assert pc.workspace_status(ws) == 4


def test_tiny_trace_every_stage():
    tr = pcgen.make_trace("tiny")
    keys, depth = oracle.hash_trace(tr)
    od = check_keys_path(keys, depth, tr.caps(), "tiny")
    assert np.array_equal(od, oracle.stack_distance_walk(keys))


def test_tiny_trace_end_to_end_pipeline():
    tr = pcgen.make_trace("tiny")
    keys, depth = oracle.hash_trace(tr)
    caps = tr.caps()
    up = pc.upload_trace(tr)
    a, b = CUSTOM_COSTS[1]
    p = pc.Pipeline(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"],
                    pc.to_dev_u64(caps), 16, a, b)
    p.run()
    torch.cuda.synchronize()
    assert p.status() == {"hash": 0, "prev_next": 0, "stack_distance": 0, "mrc": 0}
    assert np.array_equal(pc.as_u64(p.keys), keys)
    op, on = oracle.prev_next(keys)
    assert np.array_equal(pc.as_u32(p.prev), op) and np.array_equal(pc.as_u32(p.next), on)
    assert np.array_equal(pc.as_u32(p.dist), oracle.stack_distance_walk(keys))
    g = pc.bins_to_host(p.bins)
    cnt, dsum, cost = oracle.mrc_bins(keys, caps, depth, a, b)
    assert g["count"] == cnt and g["depthsum"] == dsum and g["cost"] == cost


# -------------------------------------------------------------- edge cases

def stream(kind, n, seed=0):
    rng = np.random.default_rng(seed)
    if kind == "equal":
        return np.full(n, 0xABCDEF, np.uint64)
    if kind == "distinct":
        return (rng.permutation(n).astype(np.uint64) * np.uint64(2654435761) + np.uint64(1))
    if kind == "hot":
        return pcgen.random_keys(n, max(n // 50, 1), seed, hot=0.5)
    if kind == "few":
        return pcgen.random_keys(n, 7, seed)
    if kind == "cyclic":
        m = max(n // 7, 1)
        return (np.arange(n) % m).astype(np.uint64) + np.uint64(5)
    if kind == "lowpairs":
        # every low-32-bit value is shared by two keys: short mixed runs
        low = rng.integers(1, 2 ** 32, size=max(n // 40, 1), dtype=np.uint64)
        pick = rng.integers(0, low.size, size=n)
        high = rng.integers(1, 3, size=n).astype(np.uint64)
        return low[pick] | (high << np.uint64(32))
    if kind == "lowsame":
        # one low-32-bit value for everything, 1000 keys: one huge mixed run
        return np.uint64(0x1234ABCD) | (rng.integers(1, 1001, size=n).astype(np.uint64) << np.uint64(32))
    if kind == "lowhot":
        # a hot key and a rare key sharing its low bits among random keys
        k = pcgen.random_keys(n, max(n // 20, 1), seed)
        u = rng.random(n)
        k[u < 0.4] = np.uint64(0x77 | (5 << 32))
        k[u > 0.999] = np.uint64(0x77 | (9 << 32))
        return k
    return pcgen.random_keys(n, max(n // 10, 1), seed)


@pytest.mark.parametrize("n", [0, 1, 2, 3, 63, 64, 65, 2047, 2048, 2049, 4095, 4096, 4097, 8193, 16383, 16384,
                               16385])
def test_small_and_ragged_sizes(n):
    check_keys_path(stream("mixed", n, n), caps=np.array([1, 2, 5, 100, 1000], np.uint64),
                    label="ragged%d" % n)


@pytest.mark.parametrize("kind", ["equal", "distinct", "hot", "few", "cyclic", "mixed", "lowpairs",
                                  "lowsame", "lowhot"])
def test_degenerate_streams(kind):
    check_keys_path(stream(kind, 70001, 3), caps=np.array([0, 1, 2, 7, 10000, 10 ** 8], np.uint64),
                    label=kind)
    # 1000 keys sharing one low-32-bit value are too many to scan, so the
    # high-bit passes and the second link must have run; short mixed runs
    # (lowpairs) and a hot key sharing its low bits with a rare one (lowhot)
    # are resolved by scanning
    assert LAST_HIGH_KEY[0] == (kind == "lowsame"), kind


# 2^22 + 777 and 2^23 + 5 give the way back to time order a second
# partition pass of one and two bits after the link's eight
@pytest.mark.parametrize("n", [(1 << 20) + 12345, (1 << 21) - 1, (1 << 22) + 777, (1 << 23) + 5])
def test_two_level_sizes(n):
    check_keys_path(stream("mixed", n, 9), label="twolevel%d" % n)


def test_determinism():
    keys = stream("hot", 300000, 4)
    op, on = oracle.prev_next(keys)
    d1 = gpu_dist(op, on)
    d2 = gpu_dist(op, on)
    assert np.array_equal(d1, d2)
    caps = np.array([1, 10, 100, 1000], np.uint64)
    assert gpu_bins(d1, caps) == gpu_bins(d2, caps)


@pytest.mark.parametrize("k", [1024, 1025, 2500, 4096])
def test_many_capacities(k):
    # more edges than one launch holds in LDS (1024): each launch takes only
    # the accesses between its own edges; duplicate edges, a zero edge and
    # edges on both sides of every distance, aligned and unaligned views
    n = 70001
    keys = stream("mixed", n, 11)
    ids = oracle.key_ids(keys)
    op, on = oracle.prev_next(keys, ids)
    od = oracle.stack_distance_bit(op)
    rng = np.random.default_rng(k)
    top = int(od[od != NONE].max()) + 2
    caps = np.sort(np.concatenate([[0], rng.integers(0, top + top // 4, k - 1)])).astype(np.uint64)
    dep = rng.integers(0, 5000, n).astype(np.uint32)
    say("case many_capacities k", k, "n", n, "distinct edges", np.unique(caps).size)
    cnt, dsum, cost = oracle.mrc_bins(keys, caps, dep, 1, 1, ids, threads=16)
    nh = oracle.nextuse_hist(on, caps)
    g = gpu_bins(od, caps, dep, on, 1, 1)
    assert g["count"] == cnt and g["depthsum"] == dsum and g["cost"] == cost
    assert g["nextuse"] == nh
    # views one element past an aligned start: scalar loads throughout
    shift = lambda a: pc.to_dev_u32(np.concatenate([[7], a]).astype(np.uint32))[1:]
    out, ws = pc.mrc_weighted(shift(od), pc.to_dev_u64(caps), shift(dep), shift(on), 1, 1)
    assert pc.workspace_status(ws) == 0
    g = pc.bins_to_host(out)
    assert g["count"] == cnt and g["depthsum"] == dsum and g["cost"] == cost
    assert g["nextuse"] == nh


def layout_of(case, n, rng):
    """Request lengths summing to n for the layout cases."""
    if case == "one_request":
        return [n]
    if case == "single":
        return [1] * n
    L = []
    while sum(L) < n:
        if case == "empty_reqs" and rng.random() < 0.3:
            L.append(0)
        L.append(int(rng.integers(1, 3000 if case == "ragged" else 20)))
    L[-1] -= sum(L) - n
    if case == "empty_reqs":
        L = [0] + L + [0, 0]
    return L


@pytest.mark.parametrize("desc", [False, True])
@pytest.mark.parametrize("case,n,k", [("ragged", 70001, 20), ("short", 70001, 20), ("empty_reqs", 20003, 20),
                                      ("single", 4099, 20), ("one_request", 9, 5), ("short", 1, 5),
                                      ("short", 7, 5), ("short", 8, 5), ("short", 63, 5), ("short", 64, 5),
                                      ("short", 65, 5), ("ragged", 70001, 2500)])
def test_bins_with_depth_from_the_layout(case, n, k, desc):
    # depth[t] = t - blk_off[r] for the request r holding t (or, deepest
    # first, blk_off[r + 1] - 1 - t): the same bins as with that depth passed
    # as an array, and as the oracle's; request starts and ends fall at every
    # offset within the 8-access groups and the 64-position words
    rng = np.random.default_rng(n + k)
    L = layout_of(case, n, rng)
    off = np.concatenate([[0], np.cumsum(L)]).astype(np.uint64)
    assert int(off[-1]) == n
    pos = np.arange(n, dtype=np.int64)
    if desc:
        depth = (np.repeat(off[1:].astype(np.int64), L) - 1 - pos).astype(np.uint32)
    else:
        depth = (pos - np.repeat(off[:-1].astype(np.int64), L)).astype(np.uint32)
    keys = stream("mixed", n, 13)
    ids = oracle.key_ids(keys)
    op, on = oracle.prev_next(keys, ids)
    od = oracle.stack_distance_bit(op)
    top = int(od[od != NONE].max()) + 2 if (od != NONE).any() else 2
    caps = np.sort(rng.integers(0, top + 2, k)).astype(np.uint64)
    say("case layout", case, "n", n, "requests", len(L), "caps", k)
    a, b = 2 * 16 * 3_000_000_000, 2 * 16 * 16
    out, ws = pc.mrc_weighted_layout(pc.to_dev_u32(od), pc.to_dev_u64(caps), pc.to_dev_u64(off), pc.to_dev_u32(on),
                                     a, b, deepest_first=desc)
    assert pc.workspace_status(ws) == 0
    g = pc.bins_to_host(out)
    assert g == gpu_bins(od, caps, depth, on, a, b)
    cnt, dsum, cost = oracle.mrc_bins(keys, caps, depth, a, b, ids, threads=16)
    assert g["count"] == cnt and g["depthsum"] == dsum and g["cost"] == cost
    assert g["nextuse"] == oracle.nextuse_hist(on, caps)


def test_bins_layout_rejects_an_invalid_layout():
    od = oracle.stack_distance_bit(oracle.prev_next(stream("mixed", 5000, 2))[0])
    caps = pc.to_dev_u64(np.array([1, 10, 100], np.uint64))
    for off in ([0, 100, 4000], [1, 2500, 5000], [0, 3000, 2000, 5000]):
        for desc in (False, True):
            out, ws = pc.mrc_weighted_layout(pc.to_dev_u32(od), caps, pc.to_dev_u64(np.array(off, np.uint64)),
                                             deepest_first=desc)
            assert pc.workspace_status(ws) == 2, off


def test_decreasing_edges_set_the_status():
    # edges out of order inside one launch's edges and across two launches
    od = oracle.stack_distance_bit(oracle.prev_next(stream("mixed", 5000, 2))[0])
    for k, i in ((10, 4), (2000, 1023)):
        caps = np.arange(1, k + 1, dtype=np.uint64)
        caps[i] = caps[i + 1] + 1
        out, ws = pc.mrc_weighted(pc.to_dev_u32(od), pc.to_dev_u64(caps))
        assert pc.workspace_status(ws) == 3, (k, i)


# ------------------------------------------------------- workload-shaped

def test_agent_trace_reduced_all_stages():
    tr = pcgen.make_trace("agent", n_sessions=250)
    keys, depth = oracle.hash_trace(tr)
    gk, gd = gpu_hash(tr)
    assert np.array_equal(gk, keys) and np.array_equal(gd, depth)
    check_keys_path(keys, depth, tr.caps(), "agent250")


@pytest.mark.parametrize("B", [64, 256])
def test_agent_trace_granularity_sweep(B):
    tr = pcgen.make_trace("agent", n_sessions=250)
    keys, depth = oracle.hash_trace(tr, B)
    gk, _ = gpu_hash(tr, B)
    assert np.array_equal(gk, keys)
    check_keys_path(keys, depth, pcgen.capacities("tokens64", B), "agent250-B%d" % B)


def test_chat_trace_reduced_with_shared_prompts():
    tr = pcgen.make_trace("chat", n_sessions=1500)
    keys, depth = oracle.hash_trace(tr)
    gk, _ = gpu_hash(tr)
    assert np.array_equal(gk, keys)
    caps = tr.caps()[::6]
    check_keys_path(keys, depth, caps, "chat1500")
