"""Workload characterisation at the benchmark's full size.

The full-scale mixed trace (~2.1e9 block accesses, 1.39e6 requests) runs
through the Profiler (``bench.py --profile``).  Checks:

* the session histograms against the oracle, exactly (they only need the
  request table);
* the block histograms against an independent computation with plain torch
  ops on the GPU (no libpc): every access's chain start by pointer jumping
  over prev[], then per block its access count and first/last times, and per
  reuse the time since the previous access; all exact.
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
B = 16
EDGES = [10 ** k for k in range(0, 11)] + [3 * 10 ** k for k in range(0, 10)]
EDGES.sort()
FREQ_MAX = 2048


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def full():
    assert torch.cuda.is_available()
    tr = pcgen.make_trace("full")
    say("full trace generated:", tr.n_requests, "requests", tr.n_blocks(), "accesses")
    up = pc.upload_trace(tr, B)
    p = pc.Profiler(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"], up["session"],
                    up["ts_us"], pc.to_dev_u64(np.array(EDGES, np.uint64)), B, freq_max=FREQ_MAX,
                    fp_max=1 << 16, rq_max=2048)
    p.run()
    torch.cuda.synchronize()
    say("profiler done, status", p.status())
    yield tr, up, p
    del p
    torch.cuda.empty_cache()


def test_device_status_clean(full):
    _, _, p = full
    assert p.status() == {"hash": 0, "prev_next": 0, "reuse_profile": 0, "session_profile": 0}


def test_session_histograms_exact(full):
    tr, _, p = full
    want = oracle.session_profile(tr.blk_off(B), tr.session, tr.ts_us.astype(np.uint64), EDGES, 1 << 16, 2048)
    assert pc.hists_to_host(p.sessions) == want


def test_block_histograms_against_torch(full):
    tr, up, p = full
    n = p.n
    assert n < 2 ** 31
    dev = torch.device("cuda")
    prev = p.prev.to(torch.int64) & 0xFFFFFFFF
    cold = prev == NONE
    # chain start of every access by pointer jumping
    head = torch.where(cold, torch.arange(n, device=dev), prev).to(torch.int32)
    del prev
    for rounds in range(40):
        nxt = head[head.to(torch.int64)]
        if torch.equal(nxt, head):
            break
        head = nxt
    del nxt
    say("pointer jumping converged after", rounds, "rounds")
    blk_off = up["blk_off"]
    ts = up["ts_us"]
    edges = torch.tensor(EDGES, dtype=torch.int64, device=dev)
    k = len(EDGES)
    K = k + 1
    count = torch.zeros(n, dtype=torch.int32, device=dev)
    chunk = 1 << 27
    interval = torch.zeros(K, dtype=torch.int64, device=dev)
    for lo in range(0, n, chunk):
        hi = min(n, lo + chunk)
        h = head[lo:hi].to(torch.int64)
        count.index_add_(0, h, torch.ones(hi - lo, dtype=torch.int32, device=dev))
        pos = torch.arange(lo, hi, device=dev)
        pv = p.prev[lo:hi].to(torch.int64) & 0xFFFFFFFF
        has = pv != NONE
        r_t = torch.searchsorted(blk_off, pos[has], right=True) - 1
        r_p = torch.searchsorted(blk_off, pv[has], right=True) - 1
        gap = ts[r_t] - ts[r_p]
        interval += torch.bincount(torch.bucketize(gap, edges, right=True), minlength=K)
    # per block: first = its chain start, last = the access with no next
    lifetime = torch.zeros(K, dtype=torch.int64, device=dev)
    freq = torch.zeros(FREQ_MAX + 1, dtype=torch.int64, device=dev)
    by_class = torch.zeros(32 * K, dtype=torch.int64, device=dev)
    for lo in range(0, n, chunk):
        hi = min(n, lo + chunk)
        nx = p.next[lo:hi].to(torch.int64) & 0xFFFFFFFF
        last = torch.nonzero(nx == NONE).squeeze(1) + lo
        first = head[last].to(torch.int64)
        f = count[first].to(torch.int64)
        life = ts[torch.searchsorted(blk_off, last, right=True) - 1] - \
            ts[torch.searchsorted(blk_off, first, right=True) - 1]
        lb = torch.bucketize(life, edges, right=True)
        lifetime += torch.bincount(lb, minlength=K)
        freq += torch.bincount(torch.clamp(f, max=FREQ_MAX), minlength=FREQ_MAX + 1)
        cls = torch.floor(torch.log2(f.to(torch.float64))).to(torch.int64)   # exact for f < 2^31
        by_class += torch.bincount(cls * K + lb, minlength=32 * K)
    g = pc.hists_to_host(p.reuse)
    assert g["interval"] == interval.cpu().tolist()
    assert g["lifetime"] == lifetime.cpu().tolist()
    assert g["freq"] == freq.cpu().tolist()
    assert g["life_by_class"] == by_class.cpu().tolist()
    assert sum(g["freq"]) == int(cold.sum())
