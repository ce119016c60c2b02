"""Session-level eviction at the benchmark's full size.

The full-scale mixed trace runs through the session mode of the Pipeline
(``bench.py --residency session``).  The oracle cannot redo the whole trace,
so it checks:

* exact windows of whole requests: the synthetic sessions are append-only,
  so a session's footprint after a request is that request's block count,
  and the distance of a block whose previous use lies inside a window only
  involves requests inside it; the oracle's walk over the window is exact
  for those blocks;
* properties that hold at any size, with plain torch ops on the GPU: none
  exactly for cold accesses, and bins equal to a torch bucketize of the
  distances.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import pcgen
from paper_2609_28870_amd import pc

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(1500)]
NONE = pc.NONE
P_LIN = 3_000_000_000
B = 16


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def full():
    assert torch.cuda.is_available()
    tr = pcgen.make_trace("full")
    say("full trace generated:", tr.n_requests, "requests", tr.n_blocks(), "accesses")
    caps = tr.caps()
    up = pc.upload_trace(tr, B)
    p = pc.Pipeline(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"],
                    pc.to_dev_u64(caps), B, 2 * B * P_LIN, 2 * B * B, residency="session",
                    session=up["session"])
    p.run()
    torch.cuda.synchronize()
    say("session-level pipeline done, status", p.status())
    yield tr, caps, p
    del p
    torch.cuda.empty_cache()


def test_device_status_clean(full):
    _, _, p = full
    assert p.status() == {"hash": 0, "prev_next": 0, "stack_distance": 0, "mrc": 0}


@pytest.mark.parametrize("where", ["start", "middle", "end"])
def test_exact_request_windows(full, where):
    tr, _, p = full
    off = tr.blk_off()
    n = p.n
    m = 3_000_000
    a0 = {"start": 0, "middle": n // 2, "end": n - m}[where]
    r0 = int(np.searchsorted(off, a0, side="left"))
    r1 = int(np.searchsorted(off, int(off[r0]) + m, side="right")) - 1
    a, b = int(off[r0]), int(off[r1])
    keys, _ = oracle.hash_requests(tr.tokens, tr.tok_start[r0:r1], tr.tok_len[r0:r1], B)
    wo = (off[r0:r1 + 1] - off[r0]).astype(np.uint64)
    want = oracle.stack_distance_session_walk(keys, wo, tr.session[r0:r1].astype(np.uint32))
    got = pc.as_u32(p.dist[a:b])
    gp = pc.as_u32(p.prev[a:b]).astype(np.int64)
    inside = want != NONE
    say(where, "window of requests", r0, r1, "accesses", b - a, "with in-window reuse", int(inside.sum()))
    assert np.array_equal(got[inside], want[inside])
    assert np.all((gp[~inside] == NONE) | (gp[~inside] < a))
    if a == 0:
        assert np.all(got[~inside] == NONE)


def test_cold_exactly_none(full):
    _, _, p = full
    n = p.n
    chunk = 1 << 27
    for lo in range(0, n, chunk):
        hi = min(n, lo + chunk)
        d = p.dist[lo:hi].to(torch.int64) & 0xFFFFFFFF
        cold = (p.prev[lo:hi].to(torch.int64) & 0xFFFFFFFF) == NONE
        assert bool(((d == NONE) == cold).all())


def test_bins_match_torch_bucketize(full):
    tr, caps, p = full
    n = p.n
    k = caps.size
    edges = torch.tensor(caps.astype(np.int64), device="cuda")
    count = torch.zeros(k + 1, dtype=torch.int64, device="cuda")
    dsum = torch.zeros(k + 1, dtype=torch.int64, device="cuda")
    off = torch.tensor(tr.blk_off().astype(np.int64), device="cuda")
    chunk = 1 << 27
    for lo in range(0, n, chunk):
        hi = min(n, lo + chunk)
        d = p.dist[lo:hi].to(torch.int64) & 0xFFFFFFFF
        bk = torch.bucketize(d, edges, right=True)
        bk[d == NONE] = k
        count += torch.bincount(bk, minlength=k + 1)
        # depth = position in the request, from the offsets with torch
        t = torch.arange(lo, hi, device="cuda", dtype=torch.int64)
        dep = t - off[torch.searchsorted(off, t, right=True) - 1]
        dsum.scatter_add_(0, bk, dep)
    g = pc.bins_to_host(p.bins)
    assert g["count"] == count.cpu().tolist()
    assert g["depthsum"] == dsum.cpu().tolist()
    a, b = 2 * B * P_LIN, 2 * B * B
    assert g["cost"] == [a * c + b * d for c, d in zip(g["count"], g["depthsum"])]
