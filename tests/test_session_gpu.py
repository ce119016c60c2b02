"""Parity of session-level eviction (Sec. 5.3, whole sessions evicted at
once) through the C ABI against the CPU oracle.

The GPU turns per-access prev links, the request table and the session of
every request into a size-weighted session distance; the oracle walks the
session recency list directly, and its literal per-capacity simulation is
pinned to that walk on the CPU.  Distances and bins are integers and must be
bit-exact."""
import sys

import numpy as np
import pytest
import torch

import oracle
import pcgen
from conftest import session_golden
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


def gpu_session_dist(keys, blk_off, sess):
    prev, _, ws = pc.prev_next_use(pc.to_dev_u64(keys))
    assert pc.workspace_status(ws) == 0
    d, ws = pc.stack_distance_session(prev, pc.to_dev_u64(blk_off), pc.to_dev_u32(sess))
    assert pc.workspace_status(ws) == 0
    return pc.as_u32(d)


def check_session(keys, blk_off, sess, label=""):
    keys = np.asarray(keys, np.uint64)
    say("case", label, "n", keys.size, "requests", len(blk_off) - 1, "sessions", len(np.unique(sess)))
    got = gpu_session_dist(keys, blk_off, sess)
    want = oracle.stack_distance_session_walk(keys, blk_off, sess)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, "%s: %d mismatches, first t=%s gpu=%s want=%s" % (
        label, bad.size, bad[:5], got[bad[:5]], want[bad[:5]])
    return got


def test_hand_worked_examples():
    for name, keys, blk_off, sess, want, _hits in session_golden():
        assert list(check_session(keys, blk_off, sess, "golden-" + name)) == want, name


def random_sessions(count, seed, append_only):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(count):
        n_sess = int(rng.integers(1, 9))
        ctx = {s: [] for s in range(n_sess)}
        shared = {p: [10 ** 9 * (p + 1) + d for d in range(int(rng.integers(1, 4)))] for p in range(2)}
        reqs, sess, nxt = [], [], 1
        for _r in range(int(rng.integers(1, 40))):
            s = int(rng.integers(n_sess))
            if append_only:
                if not ctx[s] and rng.random() < 0.4:
                    ctx[s] = list(shared[int(rng.integers(2))])
                grow = int(rng.integers(0, 4))
                ctx[s] = ctx[s] + list(range(nxt, nxt + grow))
                nxt += grow
                req = list(ctx[s])
            else:
                req = list(rng.choice(60, size=int(rng.integers(0, 7)), replace=False) + 1)
            reqs.append(req)
            sess.append(s * 7919 + 3)          # arbitrary session ids
        keys = np.array([k for r in reqs for k in r], np.uint64)
        if keys.size == 0:
            continue
        blk_off = np.concatenate([[0], np.cumsum([len(r) for r in reqs])]).astype(np.uint64)
        out.append((keys, blk_off, np.array(sess, np.uint32)))
    return out


@pytest.mark.parametrize("append_only", [True, False])
def test_random_small_sessions(append_only):
    for i, (keys, bo, sess) in enumerate(random_sessions(40, 41 if append_only else 42, append_only)):
        check_session(keys, bo, sess, "rand%d" % i)


def many_session_requests(n_req, seed, max_grow=3):
    """Many short append-only sessions (thousands of requests between a
    session's turns at the larger size), first two depths shared by groups."""
    rng = np.random.default_rng(seed)
    n_sess = max(n_req // 6, 1)
    sess = rng.integers(0, n_sess, n_req)
    grow = rng.integers(0, max_grow + 1, n_req)
    length = np.zeros(n_sess, np.int64)
    lens = np.empty(n_req, np.int64)
    for r in range(n_req):
        length[sess[r]] += grow[r]
        lens[r] = length[sess[r]]
    blk_off = np.concatenate([[0], np.cumsum(lens)]).astype(np.uint64)
    s_of = np.repeat(sess, lens).astype(np.uint64)
    d_of = np.arange(int(blk_off[-1]), dtype=np.int64) - np.repeat(blk_off[:-1].astype(np.int64), lens)
    owner = np.where(d_of < 2, (s_of % np.uint64(97)) | np.uint64(1 << 40), s_of)
    keys = (owner * np.uint64(0x9E3779B97F4A7C15)) ^ (d_of.astype(np.uint64) << np.uint64(44)) ^ np.uint64(99)
    return keys, blk_off, sess.astype(np.uint32), d_of.astype(np.uint32)


@pytest.mark.parametrize("n_req", [300, 70000])
def test_many_sessions(n_req):
    keys, bo, sess, _ = many_session_requests(n_req, n_req)
    check_session(keys, bo, sess, "many%d" % n_req)


def test_one_block_sessions_equal_per_access():
    rng = np.random.default_rng(8)
    sess = rng.integers(0, 3000, size=60000).astype(np.uint32)
    keys = sess.astype(np.uint64) * np.uint64(977) + np.uint64(3)
    bo = np.arange(sess.size + 1, dtype=np.uint64)
    got = check_session(keys, bo, sess, "one-block")
    assert np.array_equal(got, oracle.stack_distance_bit(oracle.prev_next(keys)[0]))


def test_edge_layouts():
    # no accesses; one request; one session only; empty requests in between
    d = gpu_session_dist(np.zeros(0, np.uint64), np.array([0, 0], np.uint64), np.array([4], np.uint32))
    assert d.size == 0
    keys = np.arange(1, 5000, dtype=np.uint64)
    check_session(keys, np.array([0, keys.size], np.uint64), np.array([1], np.uint32), "one-request")
    keys = np.concatenate([np.arange(1, 300, dtype=np.uint64)] * 3)
    bo = np.array([0, 299, 299, 598, 598, 598, 897], np.uint64)
    check_session(keys, bo, np.array([5, 6, 5, 7, 8, 5], np.uint32), "empty-requests")
    check_session(keys, np.array([0, 299, 598, 897], np.uint64), np.array([2, 2, 2], np.uint32), "one-session")


def test_two_level_size():
    keys, bo, sess, _ = many_session_requests(260000, 13, max_grow=4)
    assert keys.size > (1 << 20)
    check_session(keys, bo, sess, "twolevel")


def test_bad_layout_is_reported():
    keys = np.arange(1, 101, dtype=np.uint64)
    prev, _, _ = pc.prev_next_use(pc.to_dev_u64(keys))
    for bo in ([0, 50, 99], [0, 60, 40, 100], [1, 50, 100]):
        ns = len(bo) - 1
        _, ws = pc.stack_distance_session(prev, pc.to_dev_u64(np.array(bo, np.uint64)),
                                          pc.to_dev_u32(np.arange(ns, dtype=np.uint32)))
        assert pc.workspace_status(ws) == 2, bo


# ------------------------------------------------------- workload-shaped

def pipeline_session(tr, caps, a, b, B=16):
    up = pc.upload_trace(tr, B)
    p = pc.Pipeline(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"],
                    pc.to_dev_u64(caps), B, a, b, residency="session", session=up["session"])
    p.run()
    torch.cuda.synchronize()
    assert p.status() == {"hash": 0, "prev_next": 0, "stack_distance": 0, "mrc": 0}
    return p


def test_tiny_trace_pipeline_bins_against_simulation():
    tr = pcgen.make_trace("tiny")
    keys, depth = oracle.hash_trace(tr)
    bo = tr.blk_off(16)
    sess = tr.session.astype(np.uint32)
    caps = tr.caps()
    want = oracle.stack_distance_session_walk(keys, bo, sess)
    for a, b in COSTS:
        p = pipeline_session(tr, caps, a, b)
        assert np.array_equal(pc.as_u32(p.dist), want)
        g = pc.bins_to_host(p.bins)
        cnt, dsum, cost = oracle.mrc_bins_session(keys, bo, sess, caps, depth, a, b)
        assert g["count"] == cnt and g["depthsum"] == dsum and g["cost"] == cost, (a, b)
        assert g["nextuse"] == [0] * (caps.size + 1)


def test_agent_trace_reduced_against_simulation():
    tr = pcgen.make_trace("agent", n_sessions=250)
    keys, depth = oracle.hash_trace(tr)
    bo = tr.blk_off(16)
    sess = tr.session.astype(np.uint32)
    check_session(keys, bo, sess, "agent250")
    caps = tr.caps()[::8]
    a, b = COSTS[1]
    p = pipeline_session(tr, caps, a, b)
    g = pc.bins_to_host(p.bins)
    cnt, dsum, cost = oracle.mrc_bins_session(keys, bo, sess, caps, depth, a, b)
    assert g["count"] == cnt and g["depthsum"] == dsum and g["cost"] == cost


def test_chat_trace_reduced_with_shared_prompts():
    tr = pcgen.make_trace("chat", n_sessions=1500)
    keys, _ = oracle.hash_trace(tr)
    check_session(keys, tr.blk_off(16), tr.session.astype(np.uint32), "chat1500")
