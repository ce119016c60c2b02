"""Exact parity on the full agent-shaped trace (5,000 sessions with up to
2,000 turns, ~2.8e7 block accesses at B = 16) and on its eviction-granularity
sweep (B = 16, 64, 256 with capacities at 64 log-spaced token counts from
1e2 to 1e8), through the same Pipeline bench.py times.  At this size the
oracle redoes every stage, so every output is compared element by element:
keys, prev / next, distances, bins with the depth-weighted miss cost
2 B (P_lin + B d) and the next-use gaps; the request-level and session-level
modes likewise at B = 16."""
import sys

import numpy as np
import pytest
import torch

import oracle
import pcgen
from paper_2609_28870_amd import pc

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]
NONE = pc.NONE
P_LIN = 3_000_000_000


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def agent():
    assert torch.cuda.is_available()
    tr = pcgen.make_trace("agent")
    say("agent trace:", tr.n_requests, "requests", tr.n_blocks(), "accesses at B = 16")
    return tr


def bucket(dist, caps, weight):
    """Histogram of distances on the capacity edges (bin k: caps[k-1] <= d <
    caps[k]; PC_NONE and d >= caps[-1] in the last bin), counts and weight
    sums, as exact integers."""
    d = dist.astype(np.int64)
    b = np.searchsorted(caps.astype(np.int64), d, side="right")
    b[dist == NONE] = caps.size
    cnt = np.bincount(b, minlength=caps.size + 1)
    wsum = np.zeros(caps.size + 1, np.int64)
    np.add.at(wsum, b, weight.astype(np.int64))
    return [int(x) for x in cnt], [int(x) for x in wsum]


def run_pipeline(tr, B, caps, residency="access"):
    up = pc.upload_trace(tr, B)
    a, b = 2 * B * P_LIN, 2 * B * B
    p = pc.Pipeline(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"],
                    pc.to_dev_u64(caps), B, a, b, residency=residency,
                    session=up["session"] if residency == "session" else None)
    p.run()
    torch.cuda.synchronize()
    return p, a, b


@pytest.mark.parametrize("B", [16, 64, 256])
def test_access_level_every_output(agent, B):
    tr = agent
    caps = pcgen.capacities("tokens64", B)
    p, a, b = run_pipeline(tr, B, caps)
    assert p.status() == {"hash": 0, "prev_next": 0, "stack_distance": 0, "mrc": 0}
    keys, depth = oracle.hash_trace(tr, B)
    say("B", B, "accesses", keys.size)
    assert np.array_equal(pc.as_u64(p.keys), keys)
    # the pipeline takes depths from the request layout (checked through the
    # depth sums below); the hash kernel's own depth output against the oracle
    up = pc.upload_trace(tr, B)
    _, gdep, _ = pc.hash_blocks(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"], B)
    assert np.array_equal(pc.as_u32(gdep), depth)
    del up, gdep
    ids = oracle.key_ids(keys)
    op, on = oracle.prev_next(keys, ids)
    assert np.array_equal(pc.as_u32(p.prev), op)
    assert np.array_equal(pc.as_u32(p.next), on)
    od = oracle.stack_distance_bit(op)
    gd = pc.as_u32(p.dist)
    bad = np.nonzero(gd != od)[0]
    assert bad.size == 0, (bad.size, bad[:5])
    cnt, dsum, cost = oracle.mrc_bins(keys, caps, depth, a, b, ids)
    g = pc.bins_to_host(p.bins)
    assert g["count"] == cnt and g["depthsum"] == dsum and g["cost"] == cost
    assert g["nextuse"] == oracle.nextuse_hist(on, caps)
    hr, csr = pc.curves(g["count"], g["cost"])
    ohr, ocsr = oracle.curves(cnt, cost)
    np.testing.assert_allclose(hr, ohr, rtol=1e-12, atol=0)
    np.testing.assert_allclose(csr, ocsr, rtol=1e-12, atol=0)
    del p
    torch.cuda.empty_cache()


def test_request_level_every_output(agent):
    tr = agent
    B = 16
    caps = tr.caps(B)
    p, a, b = run_pipeline(tr, B, caps, "request")
    assert p.status() == {"hash": 0, "prev_next": 0, "stack_distance": 0, "stack_distance_req": 0, "mrc": 0}
    keys, depth = oracle.hash_trace(tr, B)
    off = tr.blk_off(B).astype(np.uint64)
    # the oracle's request-level distances are in depth order; the pipeline
    # hashed every request deepest block first
    want = oracle.stack_distance_req_bit(keys, off)
    pos = np.arange(keys.size, dtype=np.int64)
    r = np.searchsorted(off.astype(np.int64), pos, side="right") - 1
    perm = off[r].astype(np.int64) + off[r + 1].astype(np.int64) - 1 - pos   # recency slot -> depth slot
    assert np.array_equal(pc.as_u64(p.keys), keys[perm])
    got = pc.as_u32(p.dist_req)[np.argsort(perm)]
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, (bad.size, bad[:5])
    cnt, wsum = bucket(want, caps, depth)
    g = pc.bins_to_host(p.bins)
    assert g["count"] == cnt and g["depthsum"] == wsum
    assert g["cost"] == [a * c + b * d for c, d in zip(cnt, wsum)]
    del p
    torch.cuda.empty_cache()


def test_session_level_every_output(agent):
    tr = agent
    B = 16
    caps = tr.caps(B)
    p, a, b = run_pipeline(tr, B, caps, "session")
    assert all(v == 0 for v in p.status().values()), p.status()
    keys, depth = oracle.hash_trace(tr, B)
    off = tr.blk_off(B).astype(np.uint64)
    want = oracle.stack_distance_session_walk(keys, off, tr.session.astype(np.uint32))
    got = pc.as_u32(p.dist)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, (bad.size, bad[:5])
    cnt, wsum = bucket(want, caps, depth)
    g = pc.bins_to_host(p.bins)
    assert g["count"] == cnt and g["depthsum"] == wsum
    assert g["cost"] == [a * c + b * d for c, d in zip(cnt, wsum)]
    del p
    torch.cuda.empty_cache()
