"""Parity of request-level residency (Sec. 3.1, every block of a request
resident at once) through the C ABI against the CPU oracle.

The GPU path reorders each request's accesses (deepest block first), runs
prev/next and the per-access stack distance on that order and turns the
result into the request-level distance.  The oracle walks the recency list
of the pinned-request cache directly (small cases) or uses its Fenwick form
(larger ones, pinned to the walk and to the per-capacity simulation on the
CPU).  Distances and bins are integers and must be bit-exact."""
import sys

import numpy as np
import pytest
import torch

import oracle
import pcgen
from conftest import request_golden
from paper_2609_28870_amd import pc

pytestmark = pytest.mark.gpu
NONE = pc.NONE
COSTS = [(1, 0), (2 * 16 * 3_000_000_000, 2 * 16 * 16)]


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def recency_perm(blk_off, n):
    """Position q of the request order holds access perm[q] of the original
    order (each request reversed); the map is its own inverse."""
    bo = np.asarray(blk_off, np.int64)
    idx = np.arange(n, dtype=np.int64)
    r = np.searchsorted(bo, idx, side="right") - 1
    return bo[r] + bo[r + 1] - 1 - idx


def gpu_request_path(keys, blk_off, depth=None):
    """request order -> prev/next -> dist -> dist_req, all on the GPU, each
    call with its own workspace and a clean status."""
    kd = pc.to_dev_u64(keys)
    bo = pc.to_dev_u64(blk_off)
    dd = pc.to_dev_u32(depth) if depth is not None else None
    kr, dr, ws = pc.request_order(kd, bo, dd)
    assert pc.workspace_status(ws) == 0
    prev, nxt, ws = pc.prev_next_use(kr)
    assert pc.workspace_status(ws) == 0
    dist, ws = pc.stack_distance(prev, nxt)
    assert pc.workspace_status(ws) == 0
    dreq, ws = pc.stack_distance_req(prev, dist, bo)
    assert pc.workspace_status(ws) == 0
    out = dict(keys_r=pc.as_u64(kr), prev=pc.as_u32(prev), next=pc.as_u32(nxt), dist=pc.as_u32(dist),
               dist_req=pc.as_u32(dreq))
    if depth is not None:
        out["depth_r"] = pc.as_u32(dr)
    return out


def check_request_path(keys, blk_off, depth=None, label="", exact_walk=None):
    keys = np.asarray(keys, np.uint64)
    n = keys.size
    say("case", label, "n", n, "requests", len(blk_off) - 1)
    perm = recency_perm(blk_off, n)
    g = gpu_request_path(keys, blk_off, depth)
    assert np.array_equal(g["keys_r"], keys[perm]), label + " request order"
    if depth is not None:
        assert np.array_equal(g["depth_r"], np.asarray(depth, np.uint32)[perm]), label + " depth order"
    # the per-access stages on the reordered stream
    op, on = oracle.prev_next(keys[perm])
    assert np.array_equal(g["prev"], op) and np.array_equal(g["next"], on), label + " prev/next"
    assert np.array_equal(g["dist"], oracle.stack_distance_bit(op)), label + " per-access dist"
    if exact_walk is None:
        exact_walk = n <= 200_000
    want = (oracle.stack_distance_req_walk if exact_walk else oracle.stack_distance_req_bit)(keys, blk_off)
    got = g["dist_req"][perm]
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, "%s dist_req: %d mismatches, first t=%s gpu=%s want=%s" % (
        label, bad.size, bad[:5], got[bad[:5]], want[bad[:5]])
    return g


# ------------------------------------------------------------------ golden

def test_hand_worked_examples():
    """The three fixtures worked by hand from the residency rules."""
    for name, keys, blk_off, want, _hits in request_golden():
        g = check_request_path(keys, blk_off, label="golden-" + name)
        assert list(g["dist_req"][recency_perm(blk_off, keys.size)]) == want, name


@pytest.mark.parametrize("B", [16, 6])
def test_hash_deepest_first_is_the_request_order(B):
    """pc_hash_blocks with PC_HASH_DEEPEST_FIRST writes what pc_request_order
    makes of its depth-order output (aligned fast path and any-size path)."""
    tr = pcgen.make_trace("agent", n_sessions=60)
    keys, depth = oracle.hash_trace(tr, B)
    bo = tr.blk_off(B)
    up = pc.upload_trace(tr, B)
    h1 = torch.empty(1024, dtype=torch.int32, device="cuda")
    h2 = torch.empty(1024, dtype=torch.int32, device="cuda")
    k1, d1, ws = pc.hash_blocks(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"], B,
                                key_hist=h1, deepest_first=True)
    assert pc.workspace_status(ws) == 0
    _, _, ws = pc.hash_blocks(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"], B,
                              key_hist=h2)
    perm = recency_perm(bo, keys.size)
    assert np.array_equal(pc.as_u64(k1), keys[perm])
    assert np.array_equal(pc.as_u32(d1), depth[perm])
    assert torch.equal(h1, h2)


# --------------------------------------------------------------- structure

def random_requests(count, seed, sessions=(1, 6), turns=(1, 30)):
    """Multi-turn sessions re-sending and extending their context, some from
    shared prompts, some reset; keys distinct inside a request."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(count):
        n_sess = int(rng.integers(*sessions))
        ctx = {s: [] for s in range(n_sess)}
        shared = {p: [10 ** 9 * (p + 1) + d for d in range(int(rng.integers(1, 4)))] for p in range(3)}
        reqs, nxt = [], 1
        for _r in range(int(rng.integers(*turns))):
            s = int(rng.integers(n_sess))
            if not ctx[s] and rng.random() < 0.3:
                ctx[s] = list(shared[int(rng.integers(3))])
            grow = int(rng.integers(0, 5))
            ctx[s] = ctx[s] + list(range(nxt, nxt + grow))
            nxt += grow
            if rng.random() < 0.1:
                ctx[s] = []
            reqs.append(list(ctx[s]))   # empty requests stay in the table
        keys = np.array([k for r in reqs for k in r], np.uint64)
        blk_off = np.concatenate([[0], np.cumsum([len(r) for r in reqs])]).astype(np.uint64)
        out.append((keys, blk_off))
    return out


def test_random_small_sessions_with_empty_requests():
    for i, (keys, bo) in enumerate(random_requests(40, 11)):
        if keys.size == 0:
            continue
        check_request_path(keys, bo, label="rand%d" % i, exact_walk=True)


def many_requests(n_req, seed, max_grow=3):
    """Many short requests over many sessions (request table past one and
    two sort digits); keys (session, depth) are distinct inside a request,
    the first few depths shared by groups of sessions."""
    rng = np.random.default_rng(seed)
    n_sess = max(n_req // 6, 1)
    sess = rng.integers(0, n_sess, n_req)
    grow = rng.integers(0, max_grow + 1, n_req)
    reset = rng.random(n_req) < 0.05
    length = np.zeros(n_sess, np.int64)
    lens = np.empty(n_req, np.int64)
    for r in range(n_req):
        s = sess[r]
        if reset[r]:
            length[s] = 0
        length[s] += grow[r]
        lens[r] = length[s]
    blk_off = np.concatenate([[0], np.cumsum(lens)]).astype(np.uint64)
    s_of = np.repeat(sess, lens).astype(np.uint64)
    d_of = (np.arange(int(blk_off[-1]), dtype=np.int64) - np.repeat(blk_off[:-1].astype(np.int64), lens))
    group = s_of % np.uint64(97)
    owner = np.where(d_of < 2, group | np.uint64(1 << 40), s_of)
    keys = (owner * np.uint64(0x9E3779B97F4A7C15)) ^ (d_of.astype(np.uint64) << np.uint64(44)) ^ np.uint64(12345)
    return keys, blk_off, d_of.astype(np.uint32)


@pytest.mark.parametrize("n_req", [300, 70000])
def test_many_requests_sort_digits(n_req):
    keys, bo, depth = many_requests(n_req, n_req)
    check_request_path(keys, bo, depth, label="many%d" % n_req)


def test_single_block_requests_equal_per_access():
    keys = pcgen.random_keys(50000, 3000, 5, hot=0.3)
    bo = np.arange(keys.size + 1, dtype=np.uint64)
    g = check_request_path(keys, bo, label="single-block")
    assert np.array_equal(g["dist_req"], g["dist"])


def test_one_request_is_all_cold():
    keys = np.arange(1, 9000, dtype=np.uint64) * np.uint64(0x10001)
    bo = np.array([0, keys.size], np.uint64)
    g = check_request_path(keys, bo, label="one-request")
    assert np.all(g["dist_req"] == NONE)


def test_repeated_request_reuses_from_the_top():
    """The same request twice in a row: on its return every block is
    resident and the block at depth j has the j shallower blocks above it."""
    m = 5000
    keys = np.tile(np.arange(1, m + 1, dtype=np.uint64) * np.uint64(977), 2)
    bo = np.array([0, m, 2 * m], np.uint64)
    g = check_request_path(keys, bo, label="repeat")
    got = g["dist_req"][recency_perm(bo, 2 * m)]
    assert np.array_equal(got[m:], np.arange(m, dtype=np.uint32))


def test_scrambled_reuse_takes_the_direct_count():
    """Keys that are not prefix chains: later requests re-read earlier blocks
    in shuffled order, so their previous uses are out of order inside the
    request and the kernel counts them directly (large requests included)."""
    rng = np.random.default_rng(21)
    pool = np.arange(1, 20001, dtype=np.uint64) * np.uint64(0x9E3779B1)
    reqs = [pool[:6000], rng.permutation(pool[:6000]), pool[3000:9000],
            rng.permutation(pool[:12000])[:7000], rng.permutation(pool[5000:20000])]
    keys = np.concatenate(reqs)
    bo = np.concatenate([[0], np.cumsum([r.size for r in reqs])]).astype(np.uint64)
    check_request_path(keys, bo, label="scrambled", exact_walk=False)


@pytest.mark.parametrize("n", [0, 1, 2, 4095, 4096, 4097, 8193])
def test_ragged_sizes(n):
    keys = pcgen.random_keys(max(n, 1), max(n // 4, 1), n)[:n]
    rng = np.random.default_rng(n)
    cuts = np.sort(rng.integers(0, n + 1, size=max(n // 20, 1)))
    bo = np.unique(np.concatenate([[0], cuts, [n]])).astype(np.uint64)
    # make keys distinct inside each request: tag with the position's depth
    d = np.arange(n, dtype=np.int64) - np.repeat(bo[:-1].astype(np.int64), np.diff(bo).astype(np.int64))
    keys = keys ^ (d.astype(np.uint64) << np.uint64(48))
    if n == 0:
        g = gpu_request_path(keys, np.array([0, 0], np.uint64))
        assert g["dist_req"].size == 0
        return
    check_request_path(keys, bo, label="ragged%d" % n, exact_walk=True)


def test_two_level_size():
    keys, bo, depth = many_requests(260000, 7, max_grow=4)
    say("two-level n", keys.size)
    assert keys.size > (1 << 20)
    check_request_path(keys, bo, depth, label="twolevel")


def test_bad_layout_is_reported():
    keys = np.arange(1, 101, dtype=np.uint64)
    prev, nxt, _ = pc.prev_next_use(pc.to_dev_u64(keys))
    dist, _ = pc.stack_distance(prev, nxt)
    for bo in ([0, 50, 99], [0, 60, 40, 100], [1, 50, 100]):
        _, ws = pc.stack_distance_req(prev, dist, pc.to_dev_u64(np.array(bo, np.uint64)))
        assert pc.workspace_status(ws) == 2, bo
    _, _, ws = pc.request_order(pc.to_dev_u64(keys), pc.to_dev_u64(np.array([0, 60, 40, 100], np.uint64)))
    assert pc.workspace_status(ws) == 2


# ------------------------------------------------------- workload-shaped

def pipeline_request(tr, caps, a, b, B=16):
    up = pc.upload_trace(tr, B)
    p = pc.Pipeline(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"],
                    pc.to_dev_u64(caps), B, a, b, residency="request")
    p.run()
    torch.cuda.synchronize()
    assert p.status() == {"hash": 0, "prev_next": 0, "stack_distance": 0, "stack_distance_req": 0, "mrc": 0}
    return p


def test_tiny_trace_pipeline_bins_against_simulation():
    tr = pcgen.make_trace("tiny")
    keys, depth = oracle.hash_trace(tr)
    bo = tr.blk_off(16)
    caps = tr.caps()
    for a, b in COSTS:
        p = pipeline_request(tr, caps, a, b)
        perm = recency_perm(bo, keys.size)
        assert np.array_equal(pc.as_u64(p.keys_r), keys[perm])
        want = oracle.stack_distance_req_walk(keys, bo)
        assert np.array_equal(pc.as_u32(p.dist_req)[perm], want)
        g = pc.bins_to_host(p.bins)
        cnt, dsum, cost, feas = oracle.mrc_bins_req(keys, bo, caps, depth, a, b)
        assert any(feas) and not all(feas)
        assert g["count"] == cnt and g["depthsum"] == dsum and g["cost"] == cost, (a, b)
        assert g["nextuse"] == [0] * (caps.size + 1)


def test_agent_trace_reduced_against_simulation():
    tr = pcgen.make_trace("agent", n_sessions=250)
    keys, depth = oracle.hash_trace(tr)
    bo = tr.blk_off(16)
    check_request_path(keys, bo, depth, label="agent250")
    caps = tr.caps()[::8]
    a, b = COSTS[1]
    p = pipeline_request(tr, caps, a, b)
    g = pc.bins_to_host(p.bins)
    cnt, dsum, cost, feas = oracle.mrc_bins_req(keys, bo, caps, depth, a, b)
    assert any(feas)
    assert g["count"] == cnt and g["depthsum"] == dsum and g["cost"] == cost


def test_chat_trace_reduced_distances():
    tr = pcgen.make_trace("chat", n_sessions=1500)
    keys, depth = oracle.hash_trace(tr)
    check_request_path(keys, tr.blk_off(16), depth, label="chat1500")
