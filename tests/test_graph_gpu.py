"""One Pipeline step captured into a HIP graph and replayed.

Every path decision inside a step (the chained prev/next or the generic one
over all keys; the stack distance over runs or the dominance count over
accesses) is taken on the device, so the whole step can be captured once and
replayed on new inputs of the same shape.  One graph is replayed, in turn,
over two traces with the same request lengths: in one every request copies a
prefix of an earlier request's blocks (the chain and the runs paths hold), in
the other each block is one of two and requests branch at every depth (too
many unresolved accesses and too many runs: the generic prev/next and the
dominance count run).  Every replay must equal the eager run of the same
trace, and both must equal the oracle."""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2609_28870_amd import pc

pytestmark = pytest.mark.gpu
B = 16
CAPS = np.array([1, 2, 5, 10, 50, 100, 500, 1000, 5000, 20000, 100000], np.uint64)
ALPHA, BETA = 2 * 16 * 3_000_000_000, 2 * 16 * 16


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def two_traces(n_req=2000, seed=3):
    """Token buffers of the two traces over one layout (request r's tokens at
    16 * blk_off[r], length 16 * L[r])."""
    rng = np.random.default_rng(seed)
    L = rng.integers(16, 49, n_req)
    table = rng.integers(0, 1 << 31, (int(L.sum()) + 2, B)).astype(np.int32)   # one row per fresh block
    fresh = 2
    copy_reqs = []
    for r in range(n_req):
        if r and rng.random() < 0.95:
            # the longest of four earlier requests, cut a few blocks short
            cand = [copy_reqs[int(i)] for i in rng.integers(0, r, 4)]
            src = max(cand, key=lambda c: c.size)
            cut = max(0, min(int(L[r]), src.size) - int(rng.integers(0, 4)))
        else:
            src, cut = np.empty(0, np.int64), 0
        new = np.arange(fresh, fresh + L[r] - cut)
        fresh += L[r] - cut
        copy_reqs.append(np.concatenate([src[:cut], new]))
    branch_reqs = [rng.integers(0, 2, l) for l in L]   # rows 0 and 1 only
    tok_copy = table[np.concatenate(copy_reqs)].reshape(-1)
    tok_branch = table[np.concatenate(branch_reqs)].reshape(-1)
    tok_len = (L * B).astype(np.uint32)
    tok_start = np.concatenate([[0], np.cumsum(tok_len.astype(np.uint64))[:-1]]).astype(np.uint64)
    return tok_copy, tok_branch, tok_start, tok_len


def run_count(prev):
    """Runs of the prev stream: warm accesses that do not continue the previous
    access's run (t - 1 warm and prev(t) = prev(t - 1) + 1)."""
    warm = prev != pc.NONE
    cont = np.zeros(prev.size, bool)
    cont[1:] = warm[1:] & warm[:-1] & (prev[1:] == prev[:-1] + np.uint32(1))
    return int((warm & ~cont).sum())


def snapshot(p):
    torch.cuda.synchronize()
    return {"keys": pc.as_u64(p.keys).copy(),
            "prev": pc.as_u32(p.prev).copy(), "next": pc.as_u32(p.next).copy(),
            "dist": pc.as_u32(p.dist).copy(), "bins": pc.bins_to_host(p.bins),
            "chain": pc.chained_info(p.ws_pn), "runs": pc.runs_info(p.ws_sd), "status": p.status()}


def clobber(p):
    for t in (p.keys, p.prev, p.next, p.dist):
        t.fill_(-1)
    for t in p.bins.values():
        t.fill_(-1)


def check_oracle(snap, tokens, tok_start, tok_len, label):
    keys, depth = oracle.hash_requests(tokens, tok_start, tok_len, B)
    assert np.array_equal(snap["keys"], keys), label + " keys"
    ids = oracle.key_ids(keys)
    op, on = oracle.prev_next(keys, ids)
    assert np.array_equal(snap["prev"], op) and np.array_equal(snap["next"], on), label + " prev/next"
    assert np.array_equal(snap["dist"], oracle.stack_distance_bit(op)), label + " dist"
    cnt, dsum, cost = oracle.mrc_bins(keys, CAPS, depth, ALPHA, BETA, ids)
    g = snap["bins"]
    assert g["count"] == cnt and g["depthsum"] == dsum and g["cost"] == cost, label + " bins"
    assert g["nextuse"] == oracle.nextuse_hist(on, CAPS), label + " next-use bins"
    return op


def same(a, b, label):
    for k in ("keys", "prev", "next", "dist"):
        assert np.array_equal(a[k], b[k]), "%s: %s differs from eager" % (label, k)
    assert a["bins"] == b["bins"], label + ": bins differ from eager"
    assert a["chain"] == b["chain"] and a["runs"] == b["runs"], label + ": path words differ from eager"
    assert a["status"] == b["status"], label + ": status differs from eager"


def test_pipeline_step_replays_as_a_graph():
    tok_copy, tok_branch, tok_start, tok_len = two_traces()
    blk_off = np.concatenate([[0], np.cumsum(tok_len // B)]).astype(np.uint64)
    n = int(blk_off[-1])
    rmax = n // 16 + 1024   # the runs path's capacity in runs
    say("graph: n", n, "requests", tok_len.size)
    dev = torch.device("cuda:0")
    tokens = torch.from_numpy(tok_copy.copy()).to(dev)
    srcs = {"copy": torch.from_numpy(tok_copy).to(dev), "branch": torch.from_numpy(tok_branch).to(dev)}
    p = pc.Pipeline(tokens, pc.to_dev_u64(tok_start), pc.to_dev_u32(tok_len), pc.to_dev_u64(blk_off), n,
                    pc.to_dev_u64(CAPS), B, ALPHA, BETA)

    eager = {}
    for name, host in (("copy", tok_copy), ("branch", tok_branch)):
        tokens.copy_(srcs[name])
        clobber(p)
        p.run()
        eager[name] = snap = snapshot(p)
        say(name, "chain", snap["chain"], "runs", snap["runs"])
        assert snap["status"] == {"hash": 0, "prev_next": 0, "stack_distance": 0, "mrc": 0}, name
        op = check_oracle(snap, host, tok_start, tok_len, name)
        R = run_count(op)
        assert snap["runs"]["runs"] == R, name
        assert snap["runs"]["generic"] == (R > rmax), name
    # the two traces take different paths at both decisions
    assert not eager["copy"]["chain"]["generic"] and not eager["copy"]["runs"]["generic"]
    assert eager["branch"]["chain"]["generic"] and eager["branch"]["runs"]["generic"]

    # capture (after a warm-up on the capture's side stream)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        p.run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        p.run()
    torch.cuda.synchronize()

    for i, name in enumerate(["copy", "branch", "branch", "copy", "branch", "copy"]):
        clobber(p)
        tokens.copy_(srcs[name])
        torch.cuda.synchronize()
        g.replay()
        snap = snapshot(p)
        say("replay", i, name, "chain", snap["chain"], "runs", snap["runs"])
        same(snap, eager[name], "replay %d (%s)" % (i, name))
