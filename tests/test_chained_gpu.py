"""pc_prev_next_chained against the oracle's prev / next (element by element)
on chained traces in both block layouts, and on key streams that break the
chain structure, where the call must take the generic path and still be
exact.  Also the invalid block layouts it must reject to the generic path."""
import sys

import numpy as np
import pytest
import torch

import oracle
import pcgen
from paper_2609_28870_amd import pc

pytestmark = pytest.mark.gpu
NONE = pc.NONE


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def deepest_first(keys, off):
    """Each request's keys in descending depth order (the PC_HASH_DEEPEST_FIRST
    layout), built on the host from the ascending layout."""
    L = np.diff(off)
    r = np.repeat(np.arange(L.size), L)
    perm = off[r] + off[r + 1] - 1 - np.arange(keys.size, dtype=np.int64)
    return keys[perm]


def run(keys, off, deepest=False):
    kd = pc.to_dev_u64(keys)
    od = pc.to_dev_u64(off.astype(np.uint64))
    prev, nxt, ws = pc.prev_next_chained(kd, od, deepest_first=deepest)
    info = pc.chained_info(ws)
    status = pc.workspace_status(ws)
    return pc.as_u32(prev), pc.as_u32(nxt), info, status


def exact(keys, off, deepest=False):
    p, q, info, status = run(keys, off, deepest)
    op, on = oracle.prev_next(keys)
    bad = np.nonzero((p != op) | (q != on))[0]
    assert bad.size == 0, (bad.size, bad[:5], info)
    return info, status


@pytest.fixture(scope="module", params=[("tiny", None), ("agent", 300), ("chat", 400)])
def chained(request):
    assert torch.cuda.is_available()
    name, ns = request.param
    tr = pcgen.make_trace(name, n_sessions=ns) if ns else pcgen.make_trace(name)
    keys, _ = oracle.hash_trace(tr)
    return name, keys, tr.blk_off(16).astype(np.int64)


def test_chained_trace_takes_the_chain_path(chained):
    name, keys, off = chained
    info, status = exact(keys, off)
    say(name, keys.size, info)
    assert status == 0 and not info["generic"], info
    op, on = oracle.prev_next(keys)
    # exactly the first and last uses stay unresolved on these traces
    assert info["unresolved"] == int(((op == NONE) | (on == NONE)).sum())


def test_deepest_first_layout(chained):
    name, keys, off = chained
    info, status = exact(deepest_first(keys, off), off, deepest=True)
    assert status == 0 and not info["generic"], info


@pytest.mark.parametrize("kinds", [1, 3, 1000, None])
def test_unchained_keys_fall_back_exactly(kinds):
    rng = np.random.default_rng(7)
    L = rng.integers(0, 400, 300)
    L[::17] = 0                                   # empty requests
    off = np.concatenate([[0], np.cumsum(L)]).astype(np.int64)
    n = int(off[-1])
    keys = (rng.integers(0, kinds, n) if kinds else rng.integers(0, 2 ** 63, n)).astype(np.uint64)
    for deepest in (False, True):
        info, status = exact(keys, off, deepest)
        assert status == 0
        say("kinds", kinds, "deepest", deepest, info)


def test_chains_with_planted_collisions():
    tr = pcgen.make_trace("agent", n_sessions=60)
    keys, _ = oracle.hash_trace(tr)
    off = tr.blk_off(16).astype(np.int64)
    rng = np.random.default_rng(3)
    for trial in range(4):
        k = keys.copy()
        i, j = rng.integers(0, k.size, 2)
        k[i] = k[j]                               # one key copied to an unrelated place
        info, status = exact(k, off)
        say("collision", i, j, info)


def chain_keys(word_seqs):
    """Chained keys (equal keys mean equal prefixes) of per-request word
    sequences, and the block layout."""
    out = []
    for k in word_seqs:
        c = np.empty(k.size, np.uint64)
        x = 0
        for d, w in enumerate(k):
            x = oracle.step(x, int(w))
            c[d] = x
        out.append(c)
    off = np.concatenate([[0], np.cumsum([r.size for r in out])]).astype(np.int64)
    return np.concatenate(out), off


def ragged_requests(rng, n_req, tail):
    """Requests that copy a prefix of an earlier request (cut just before, at
    and after 64-depth anchor boundaries) and add `tail` fresh blocks."""
    reqs = [rng.integers(0, 2 ** 63, 300).astype(np.uint64)]
    for t in range(n_req):
        src = reqs[int(rng.integers(0, len(reqs)))]
        cut = min(int(rng.choice([0, 1, 63, 64, 65, 127, 128, 129, 200, 255, 256, 257])), src.size)
        new = int(rng.integers(0, tail + 1))
        reqs.append(np.concatenate([src[:cut], rng.integers(0, 2 ** 63, new).astype(np.uint64)]))
    return reqs


@pytest.mark.parametrize("tail", [0, 3, 100])
def test_ragged_requests_and_anchor_boundaries(tail):
    rng = np.random.default_rng(11 + tail)
    keys, off = chain_keys(ragged_requests(rng, 400, tail))
    for deepest in (False, True):
        info, status = exact(deepest_first(keys, off) if deepest else keys, off, deepest)
        say("tail", tail, "deepest", deepest, keys.size, info)
        assert status == 0
        if tail <= 3:
            # mostly reuse: the unresolved accesses fit, the chain path holds
            assert not info["generic"], info


@pytest.mark.parametrize("case", ["decreasing", "short", "long", "start"])
def test_invalid_layout_takes_the_generic_path(case):
    rng = np.random.default_rng(5)
    L = rng.integers(1, 100, 50)
    off = np.concatenate([[0], np.cumsum(L)]).astype(np.int64)
    n = int(off[-1])
    keys = rng.integers(0, 50, n).astype(np.uint64)
    bad = off.copy()
    if case == "decreasing":
        bad[10] = bad[12]
    elif case == "short":
        bad[-1] = n - 1
    elif case == "long":
        bad[-1] = n + 5
    else:
        bad[0] = 1
    kd = pc.to_dev_u64(keys)
    prev, nxt, ws = pc.prev_next_chained(kd, pc.to_dev_u64(bad.astype(np.uint64)))
    info = pc.chained_info(ws)
    assert info["generic"] and info["reason"] == 1
    assert pc.workspace_status(ws) == 2
    op, on = oracle.prev_next(keys)
    assert np.array_equal(pc.as_u32(prev), op) and np.array_equal(pc.as_u32(nxt), on)


def test_empty_and_single():
    for L in ([0], [1], [0, 0, 3], [64], [65]):
        off = np.concatenate([[0], np.cumsum(L)]).astype(np.int64)
        keys = np.arange(int(off[-1]), dtype=np.uint64)
        if keys.size == 0:
            continue
        exact(keys, off)


@pytest.mark.parametrize("residency", ["access", "request", "session"])
def test_pipeline_chained_equals_generic(residency):
    # the same trace through both prev/next and stack-distance paths: every
    # output equal (each path is also checked against the oracle elsewhere)
    tr = pcgen.make_trace("agent", n_sessions=80)
    up = pc.upload_trace(tr, 16)
    caps = pc.to_dev_u64(tr.caps(16))
    outs = []
    for chained in (True, False):
        p = pc.Pipeline(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"], caps, 16,
                        7, 3, residency=residency, session=up["session"], chained=chained)
        p.run()
        torch.cuda.synchronize()
        assert all(v == 0 for v in p.status().values()), p.status()
        o = {"prev": pc.as_u32(p.prev), "next": pc.as_u32(p.next), "dist": pc.as_u32(p.dist),
             "bins": pc.bins_to_host(p.bins)}
        if residency == "request":
            o["dist_req"] = pc.as_u32(p.dist_req)
        outs.append(o)
    a, b = outs
    for k in a:
        if k == "bins":
            assert a[k] == b[k]
        elif k == "next" and residency == "session":
            continue   # the chained session pipeline asks for prev only
        else:
            assert np.array_equal(a[k], b[k]), k


@pytest.mark.parametrize("kind", ["chained", "unchained"])
def test_prev_only_gives_the_same_prev(kind):
    # PC_PREV_ONLY skips the next links of the chain path; prev stays exact,
    # also when the generic path over all keys runs
    tr = pcgen.make_trace("chat", n_sessions=300)
    keys, _ = oracle.hash_trace(tr)
    off = tr.blk_off(16).astype(np.int64)
    if kind == "unchained":
        keys = np.random.default_rng(5).integers(0, 1000, keys.size).astype(np.uint64)
    op, on = oracle.prev_next(keys)
    kd, od = pc.to_dev_u64(keys), pc.to_dev_u64(off.astype(np.uint64))
    prev, nxt, ws = pc.prev_next_chained(kd, od, prev_only=True)
    info = pc.chained_info(ws)
    say(kind, info)
    assert pc.workspace_status(ws) == 0
    assert info["generic"] == (kind == "unchained"), info
    assert np.array_equal(pc.as_u32(prev), op)


def test_profiler_chained_equals_generic():
    tr = pcgen.make_trace("chat", n_sessions=150)
    up = pc.upload_trace(tr, 16)
    edges = pc.to_dev_u64(np.array([10 ** k for k in range(1, 11)], np.uint64))
    outs = []
    for chained in (True, False):
        p = pc.Profiler(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"], up["session"],
                        up["ts_us"], edges, 16, chained=chained)
        p.run()
        torch.cuda.synchronize()
        assert all(v == 0 for v in p.status().values()), p.status()
        outs.append((pc.as_u32(p.prev), pc.as_u32(p.next), pc.hists_to_host(p.reuse), pc.hists_to_host(p.sessions)))
    (pa, na, ra, sa), (pb, nb, rb, sb) = outs
    assert np.array_equal(pa, pb) and np.array_equal(na, nb)
    assert ra == rb and sa == sb


@pytest.mark.timeout(900)
def test_mid_size_trace_equals_generic():
    # 5.8e8 accesses: between 2^29 and 2^30 the staircase takes eight slots
    # per wave iteration (two below, as on the chat-shaped trace, sixteen
    # above, as on the full-scale one); chained and generic prev / next on
    # the GPU, element by element (both are checked against the oracle on
    # smaller traces)
    tr = pcgen.make_trace("chat", n_sessions=50000)
    up = pc.upload_trace(tr, 16)
    n = up["n_blocks"]
    say("mid-size chat trace:", n, "accesses")
    assert (1 << 29) <= n < (1 << 30), n
    keys, _, _ = pc.hash_blocks(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], n, 16,
                                want_depth=False)
    del up["tokens"]
    prev, nxt, ws = pc.prev_next_chained(keys, up["blk_off"])
    torch.cuda.synchronize()
    info = pc.chained_info(ws)
    say("chained:", info)
    assert pc.workspace_status(ws) == 0 and not info["generic"], info
    del ws
    gp, gn, gws = pc.prev_next_use(keys)
    torch.cuda.synchronize()
    assert pc.workspace_status(gws) == 0
    assert torch.equal(prev, gp) and torch.equal(nxt, gn)
