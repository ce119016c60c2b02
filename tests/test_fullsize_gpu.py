"""Parity at the benchmark's full size and launch configuration.

Three traces run through the same Pipeline bench.py times: the chat-shaped
trace (20,000 sessions, ~2.2e8 block accesses), the full-scale mixed trace
(2e9 context tokens, ~2.1e9 block accesses) and the same mix up to 2.2e9
context tokens (~2.3e9 accesses, so positions pass 2^31).  They are checked
against the oracle's full-size references (``tests/golden/fullsize_*.txt``,
written by ``tests/golden/make_fullsize.py`` from ``oracle/`` alone):

* every array (keys, depth, prev, next, dist) through a position-keyed
  fingerprint of all its elements;
* every capacity's LRU hit count, depth sum over the hits and hit-set
  fingerprint (which accesses hit), from the GPU's bins and distances;
* the next-use histogram and the number of distinct blocks.

Besides, the oracle recomputes sampled requests' keys and three exact
windows of the trace (distances and links only depend on the past), the
distances of the runs path equal the generic dominance count's element by
element, and properties that hold at any size are checked with plain torch
ops on the GPU (prev/next are inverse links between equal keys).
"""
import os
import sys

import numpy as np
import pytest
import torch

import oracle
import pcgen
from fingerprints import array_fp, hit_fps
from paper_2609_28870_amd import pc

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(1500)]
NONE = pc.NONE
P_LIN = 3_000_000_000
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
# workload name -> (pcgen config, context-token target override)
WORKLOADS = {"chat": ("chat", None), "full": ("full", None), "full_2g2": ("full", 2_200_000_000)}


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def read_reference(name):
    g = {"caps": []}
    with open(os.path.join(GOLDEN, "fullsize_%s.txt" % name)) as f:
        for line in f:
            w = line.split("#", 1)[0].split()
            if not w:
                continue
            if w[0] == "cap":
                g["caps"].append((int(w[1]), int(w[2]), int(w[3]), int(w[4], 16)))
            elif w[0] == "nextuse":
                g["nextuse"] = [int(x) for x in w[1:]]
            elif w[0].startswith("fp_"):
                g[w[0]] = int(w[1], 16)
            elif w[0] != "workload":
                g[w[0]] = int(w[1])
    return g


@pytest.fixture(scope="module", params=["chat", "full", "full_2g2"])
def full(request):
    assert torch.cuda.is_available()
    cfg, target = WORKLOADS[request.param]
    say(request.param, "generating the trace")
    tr = pcgen.make_trace(cfg, target_tokens=target)
    say(request.param, "trace generated:", tr.n_requests, "requests", tr.n_blocks(), "accesses")
    caps = tr.caps()
    B = 16
    up = pc.upload_trace(tr, B)
    p = pc.Pipeline(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"],
                    pc.to_dev_u64(caps), B, 2 * B * P_LIN, 2 * B * B)
    p.run()
    torch.cuda.synchronize()
    say(request.param, "pipeline done, status", p.status())
    # the pipeline takes depths from the request layout; the hash kernel's
    # depth output, for the checks of the depth array
    _, p.depth_out, _ = pc.hash_blocks(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"],
                                       B, keys=p.keys, ws=p.ws_hash)
    torch.cuda.synchronize()
    p.reference = read_reference(request.param)
    p.name = request.param
    yield tr, caps, p
    del p, up
    torch.cuda.empty_cache()


def test_reference_is_for_this_trace(full):
    tr, caps, p = full
    g = p.reference
    assert g["n"] == p.n and g["requests"] == tr.n_requests
    assert [c for c, _, _, _ in g["caps"]] == [int(c) for c in caps]
    if p.name == "full_2g2":
        assert p.n > 2 ** 31


def test_all_arrays_match_the_oracle(full):
    _, _, p = full
    g = p.reference
    for name, t in (("keys", p.keys), ("depth", p.depth_out), ("prev", p.prev), ("next", p.next), ("dist", p.dist)):
        got = array_fp(t)
        say(p.name, name, "fingerprint", hex(got))
        assert got == g["fp_" + name], name


def test_every_capacity_matches_the_oracle(full):
    _, caps, p = full
    g = p.reference
    bins = pc.bins_to_host(p.bins)
    h = d = 0
    for k, (c, hits, dsum, _) in enumerate(g["caps"]):
        h += bins["count"][k]
        d += bins["depthsum"][k]
        assert (h, d) == (hits, dsum), c
    assert sum(bins["count"]) == p.n and sum(bins["depthsum"]) == g["depth_total"]
    assert bins["nextuse"] == g["nextuse"]
    # which accesses hit, at every capacity, from the GPU's distances
    got = hit_fps(p.dist, torch.tensor(caps.astype(np.int64), device="cuda"))
    assert got == [(hits, fp) for _, hits, _, fp in g["caps"]]


def test_cold_accesses_are_the_distinct_blocks(full):
    _, _, p = full
    n = p.n
    chunk = 1 << 27
    cold = 0
    for lo in range(0, n, chunk):
        cold += int((p.prev[lo:lo + chunk] == -1).sum())
    assert cold == p.reference["distinct"]


def test_runs_distances_equal_the_generic_dominance_count(full):
    _, _, p = full
    info = pc.runs_info(p.ws_sd)
    say(p.name, "stack distance over runs:", info)
    assert not info["generic"]
    ref, ws = pc.stack_distance(p.prev, p.next)
    torch.cuda.synchronize()
    assert pc.workspace_status(ws) == 0
    del ws
    chunk = 1 << 28
    for lo in range(0, p.n, chunk):
        assert torch.equal(ref[lo:lo + chunk], p.dist[lo:lo + chunk]), lo
    del ref
    torch.cuda.empty_cache()


def test_device_status_clean(full):
    _, _, p = full
    assert p.status() == {"hash": 0, "prev_next": 0, "stack_distance": 0, "mrc": 0}


def test_sampled_request_keys(full):
    tr, _, p = full
    off = tr.blk_off()
    rng = np.random.default_rng(0)
    reqs = np.unique(np.concatenate([np.arange(200), rng.integers(0, tr.n_requests, 300),
                                     [tr.n_requests - 1]]))
    for r in reqs:
        lo, hi = int(off[r]), int(off[r + 1])
        if hi == lo:
            continue
        want, wd = oracle.hash_requests(tr.tokens, tr.tok_start[r:r + 1], tr.tok_len[r:r + 1], 16)
        got = pc.as_u64(p.keys[lo:hi])
        assert np.array_equal(got, want), r
        assert np.array_equal(pc.as_u32(p.depth_out[lo:hi]), wd), r


def window_requests(tr, a, b):
    """Requests covering accesses [a, b) and the access offset of the first."""
    off = tr.blk_off()
    r0 = int(np.searchsorted(off, a, side="right")) - 1
    r1 = int(np.searchsorted(off, b, side="left"))
    return r0, r1, int(off[r0])


@pytest.mark.parametrize("where", ["start", "middle", "high", "end"])
def test_exact_windows(full, where):
    tr, _, p = full
    n = p.n
    m = 3_000_000
    if where == "high" and n < 2 ** 31 + 2 * m:
        pytest.skip("positions stay below 2^31 on this trace")
    a = {"start": 0, "middle": n // 2, "high": 2 ** 31 + m, "end": n - m}[where]
    r0, r1, base = window_requests(tr, a, a + m)
    keys, _ = oracle.hash_requests(tr.tokens, tr.tok_start[r0:r1], tr.tok_len[r0:r1], 16)
    keys = keys[a - base:a - base + m]
    assert np.array_equal(pc.as_u64(p.keys[a:a + m]), keys)
    op, on = oracle.prev_next(keys)
    od = oracle.stack_distance_bit(op)
    gp = pc.as_u32(p.prev[a:a + m]).astype(np.int64)
    gn = pc.as_u32(p.next[a:a + m]).astype(np.int64)
    gd = pc.as_u32(p.dist[a:a + m])
    inside = op != NONE
    say(where, "window", a, "accesses with in-window reuse:", int(inside.sum()))
    assert np.array_equal(gp[inside], op[inside].astype(np.int64) + a)
    assert np.array_equal(gd[inside], od[inside])
    # accesses whose previous use is before the window: GPU says so too
    outside = ~inside
    assert np.all((gp[outside] == NONE) | (gp[outside] < a))
    if a == 0:
        assert np.all(gp[outside] == NONE) and np.all(gd[outside] == NONE)
    has_next = on != NONE
    assert np.array_equal(gn[has_next], on[has_next].astype(np.int64) + a)
    assert np.all((gn[~has_next] == NONE) | (gn[~has_next] >= a + m))


def test_links_are_consistent_everywhere(full):
    _, _, p = full
    n = p.n
    chunk = 1 << 27
    cold = last = 0
    for lo in range(0, n, chunk):
        hi = min(n, lo + chunk)
        t = torch.arange(lo, hi, device="cuda", dtype=torch.int64)
        pv = p.prev[lo:hi].to(torch.int64) & 0xFFFFFFFF
        nx = p.next[lo:hi].to(torch.int64) & 0xFFFFFFFF
        hp = pv != NONE
        assert bool((pv[hp] < t[hp]).all())
        back = p.next[pv[hp]].to(torch.int64) & 0xFFFFFFFF
        assert bool((back == t[hp]).all())
        assert bool((p.keys[pv[hp]] == p.keys[lo:hi][hp]).all())
        hn = nx != NONE
        assert bool((nx[hn] > t[hn]).all())
        fwd = p.prev[nx[hn]].to(torch.int64) & 0xFFFFFFFF
        assert bool((fwd == t[hn]).all())
        cold += int((~hp).sum())
        last += int((~hn).sum())
        dd = p.dist[lo:hi].to(torch.int64) & 0xFFFFFFFF
        assert bool(((dd == NONE) == (~hp)).all())
        # D(t) counts distinct blocks strictly inside (prev, t)
        assert bool((dd[hp] <= t[hp] - pv[hp] - 1).all())
    assert cold == last   # first uses and last uses of each distinct key


def test_bins_match_torch_bucketize(full):
    tr, caps, p = full
    n = p.n
    k = caps.size
    edges = torch.tensor(caps.astype(np.int64), device="cuda")
    count = torch.zeros(k + 1, dtype=torch.int64, device="cuda")
    dsum = torch.zeros(k + 1, dtype=torch.int64, device="cuda")
    nuse = torch.zeros(k + 1, dtype=torch.int64, device="cuda")
    chunk = 1 << 27
    for lo in range(0, n, chunk):
        hi = min(n, lo + chunk)
        d = p.dist[lo:hi].to(torch.int64) & 0xFFFFFFFF
        b = torch.bucketize(d, edges, right=True)
        b[d == NONE] = k
        count += torch.bincount(b, minlength=k + 1)
        dep = p.depth_out[lo:hi].to(torch.int64)   # the hash kernel's, against the bins' layout depths
        dsum.scatter_add_(0, b, dep)
        nx = p.next[lo:hi].to(torch.int64) & 0xFFFFFFFF
        gap = nx - torch.arange(lo, hi, device="cuda", dtype=torch.int64)
        nb = torch.bucketize(gap, edges, right=True)
        nb[nx == NONE] = k
        nuse += torch.bincount(nb, minlength=k + 1)
    g = pc.bins_to_host(p.bins)
    assert g["count"] == count.cpu().tolist()
    assert g["depthsum"] == dsum.cpu().tolist()
    assert g["nextuse"] == nuse.cpu().tolist()
    a, b = 2 * 16 * P_LIN, 2 * 16 * 16
    assert g["cost"] == [a * c + b * d for c, d in zip(g["count"], g["depthsum"])]
    assert sum(g["count"]) == n
