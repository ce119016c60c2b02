"""Request-level residency at the benchmark's full size.

The full-scale mixed trace (~2.1e9 block accesses) runs through the request
mode of the Pipeline (``bench.py --residency request``).  The oracle cannot
redo the whole trace, so it checks:

* the request order of sampled requests (each request reversed);
* exact windows of whole requests: what a block finds above it when its
  request arrives depends only on the accesses since its previous use, so
  the oracle's request-level distances over a window [a, b) of requests are
  exact for every access whose previous use lies inside the window;
* properties that hold at any size, with plain torch ops on the GPU:
  dist_req <= dist, equality for the first (deepest) access of each request,
  none exactly for cold accesses, and bins equal to a torch bucketize of
  dist_req weighted by depth in the same order.
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
                    pc.to_dev_u64(caps), B, 2 * B * P_LIN, 2 * B * B, residency="request")
    p.run()
    torch.cuda.synchronize()
    say("request-level pipeline done, status", p.status())
    # the pipeline takes depths from the request layout; the hash kernel's
    # depth output (deepest first), for the checks of the depth array
    _, p.depth_out, _ = pc.hash_blocks(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"],
                                       B, keys=p.keys_r, ws=p.ws_hash, deepest_first=True)
    torch.cuda.synchronize()
    yield tr, caps, p
    del p
    torch.cuda.empty_cache()


def test_device_status_clean(full):
    _, _, p = full
    assert p.status() == {"hash": 0, "prev_next": 0, "stack_distance": 0, "stack_distance_req": 0, "mrc": 0}


def test_sampled_requests_reversed(full):
    tr, _, p = full
    off = tr.blk_off()
    rng = np.random.default_rng(1)
    for r in np.unique(np.concatenate([np.arange(100), rng.integers(0, tr.n_requests, 200),
                                       [tr.n_requests - 1]])):
        lo, hi = int(off[r]), int(off[r + 1])
        if hi == lo:
            continue
        want, wd = oracle.hash_requests(tr.tokens, tr.tok_start[r:r + 1], tr.tok_len[r:r + 1], B)
        assert np.array_equal(pc.as_u64(p.keys_r[lo:hi]), want[::-1]), r
        assert np.array_equal(pc.as_u32(p.depth_out[lo:hi]), wd[::-1]), r


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
    assert keys.size == b - a
    wo = (off[r0:r1 + 1] - off[r0]).astype(np.uint64)
    want = oracle.stack_distance_req_bit(keys, wo)          # depth order inside each request
    # the GPU arrays are in request order: reverse each request back
    idx = np.arange(b - a, dtype=np.int64)
    rr = np.searchsorted(wo.astype(np.int64), idx, side="right") - 1
    perm = wo.astype(np.int64)[rr] + wo.astype(np.int64)[rr + 1] - 1 - idx
    got = pc.as_u32(p.dist_req[a:b])[perm]
    gp = pc.as_u32(p.prev[a:b]).astype(np.int64)[perm]
    inside = want != NONE
    say(where, "window of requests", r0, r1, "accesses", b - a, "with in-window reuse", int(inside.sum()))
    assert np.array_equal(got[inside], want[inside])
    # the rest had their previous use before the window (or none at all)
    assert np.all((gp[~inside] == NONE) | (gp[~inside] < a))
    if a == 0:
        assert np.all(got[~inside] == NONE)


def test_properties_everywhere(full):
    _, _, p = full
    n = p.n
    first = torch.zeros(n, dtype=torch.bool, device="cuda")
    first[p.blk_off[:-1][p.blk_off[:-1] < p.blk_off[1:]]] = True   # deepest block of each request
    chunk = 1 << 27
    for lo in range(0, n, chunk):
        hi = min(n, lo + chunk)
        d = p.dist[lo:hi].to(torch.int64) & 0xFFFFFFFF
        dr = p.dist_req[lo:hi].to(torch.int64) & 0xFFFFFFFF
        cold = (p.prev[lo:hi].to(torch.int64) & 0xFFFFFFFF) == NONE
        assert bool(((dr == NONE) == cold).all())
        assert bool((dr[~cold] <= d[~cold]).all())
        f = first[lo:hi] & ~cold
        assert bool((dr[f] == d[f]).all())


def test_bins_match_torch_bucketize(full):
    tr, caps, p = full
    n = p.n
    k = caps.size
    edges = torch.tensor(caps.astype(np.int64), device="cuda")
    count = torch.zeros(k + 1, dtype=torch.int64, device="cuda")
    dsum = torch.zeros(k + 1, dtype=torch.int64, device="cuda")
    chunk = 1 << 27
    for lo in range(0, n, chunk):
        hi = min(n, lo + chunk)
        d = p.dist_req[lo:hi].to(torch.int64) & 0xFFFFFFFF
        bk = torch.bucketize(d, edges, right=True)
        bk[d == NONE] = k
        count += torch.bincount(bk, minlength=k + 1)
        dsum.scatter_add_(0, bk, p.depth_out[lo:hi].to(torch.int64))   # the hash kernel's, against the layout's
    g = pc.bins_to_host(p.bins)
    assert g["count"] == count.cpu().tolist()
    assert g["depthsum"] == dsum.cpu().tolist()
    a, b = 2 * B * P_LIN, 2 * B * B
    assert g["cost"] == [a * c + b * d for c, d in zip(g["count"], g["depthsum"])]
    assert g["nextuse"] == [0] * (k + 1)
