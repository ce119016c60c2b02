"""Belady's MIN on the GPU (pc_belady) against the oracle's demand-paging
MIN simulation (a max-heap on next use, pinned by exhaustive search and the
textbook example): hit counts, depth sums and per-access hit flags at every
capacity, from one block (every batch walked access by access, evictions
reaching into the batch's own window) to capacities that hold everything
(bulk batches only), on random streams, looping scans, chained traces, the
full agent-shaped trace and the edge cases; and the relations the paper
relies on (LRU never beats MIN; both hit every reuse once the cache holds
every block)."""
import numpy as np
import pytest
import torch

import oracle
import pcgen
from conftest import read_golden
from paper_2609_28870_amd import pc

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]
NONE = pc.NONE
# tiny to huge: window evictions, buffer refills and spills, bulk-only batches
CAPS = [0, 1, 2, 3, 7, 63, 64, 65, 100, 128, 129, 191, 200, 256, 257, 500, 512, 513, 1000, 1024, 1025, 1100, 1500,
        2048, 3000, 5000, 10000, 40000, 10 ** 7]


def gpu_belady(nxt, caps, depth=None, flags=True):
    dev_caps = pc.to_dev_u64(np.asarray(caps, np.uint64))
    out, ws = pc.belady(pc.to_dev_u32(nxt), dev_caps, pc.to_dev_u32(depth) if depth is not None else None,
                        flags=flags)
    torch.cuda.synchronize()
    assert pc.workspace_status(ws) == 0
    res = {"hits": [int(x) for x in pc.as_u64(out["hits"])], "depthsum": [int(x) for x in pc.as_u64(out["depthsum"])]}
    if flags:
        res["flags"] = out["flags"].cpu().numpy()
    return res


def check_against_oracle(keys, caps, depth=None, threads=8):
    keys = np.asarray(keys, np.uint64)
    ids = oracle.key_ids(keys)
    _, nxt = oracle.prev_next(keys, ids)
    want = oracle.belady(keys, caps, ids, nxt, flags=True, threads=threads)
    got = gpu_belady(nxt, caps, depth)
    for k, c in enumerate(caps):
        h, fl = want[k]
        assert got["hits"][k] == h, (c, got["hits"][k], h)
        assert np.array_equal(got["flags"][k], fl), c
        if depth is not None:
            assert got["depthsum"][k] == int(np.asarray(depth, np.uint64)[fl.astype(bool)].sum()), c
    return got, want


def test_textbook_example():
    rows = read_golden("page_replacement_textbook.txt")
    ref = np.array([int(x) for x in rows[0]], np.uint64) + 1
    frames, _, opt_faults = (int(x) for x in rows[1])
    _, nxt = oracle.prev_next(ref)
    got = gpu_belady(nxt, [frames])
    assert got["hits"][0] == ref.size - opt_faults


@pytest.mark.parametrize("seed", range(8))
def test_random_streams(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 60000))
    distinct = int(rng.integers(1, 30000))
    keys = rng.integers(0, distinct, size=n).astype(np.uint64)
    if seed % 2:
        keys[rng.random(n) < 0.2] = 3        # a hot block
    depth = rng.integers(0, 5000, size=n).astype(np.uint32)
    check_against_oracle(keys, CAPS, depth)


def test_looping_scan_and_degenerate_streams():
    # a cyclic scan one block larger than the cache: MIN keeps c - 1 of the
    # loop's blocks per round
    for loop in (65, 1025, 3000):
        keys = np.tile(np.arange(loop, dtype=np.uint64), 20)
        check_against_oracle(keys, [loop - 1, loop, 64, 1024, 1025, 2999])
    check_against_oracle(np.zeros(0, np.uint64), [1, 2000])
    check_against_oracle(np.array([5], np.uint64), [0, 1, 5000])
    check_against_oracle(np.arange(1000, dtype=np.uint64), [1, 2000])        # all cold
    check_against_oracle(np.full(777, 9, np.uint64), [1, 1500])              # one block


@pytest.mark.parametrize("name,sessions", [("tiny", None), ("agent", 200), ("chat", 600)])
def test_chained_traces(name, sessions):
    tr = pcgen.make_trace(name, n_sessions=sessions)
    keys, depth = oracle.hash_trace(tr)
    caps = [int(c) for c in tr.caps()][::3] + [1024, 1025]
    got, _ = check_against_oracle(keys, caps, depth)
    # LRU never beats MIN; with room for every block both hit every reuse
    lru = oracle.lru(keys, caps, depth, threads=8)
    distinct = oracle.key_ids(keys)[1]
    for k, c in enumerate(caps):
        assert lru[k][0] <= got["hits"][k], c
        if c >= distinct:
            assert got["hits"][k] == lru[k][0] == keys.size - distinct


def test_full_agent_trace_table_capacities():
    # the agent-shaped trace at full size (2.8e7 accesses), the paper's
    # cache-size points and a few around them; hits and depth sums
    tr = pcgen.make_trace("agent")
    keys, depth = oracle.hash_trace(tr, threads=8)
    caps = [1000, 5000] + list(pcgen.GIB_BLOCKS.values()) + [10 ** 6]
    ids = oracle.key_ids(keys)
    _, nxt = oracle.prev_next(keys, ids)
    want = oracle.belady(keys, caps, ids, nxt, threads=8)
    up_next = pc.to_dev_u32(nxt)
    out, ws = pc.belady(up_next, pc.to_dev_u64(np.asarray(caps, np.uint64)), pc.to_dev_u32(depth))
    torch.cuda.synchronize()
    assert pc.workspace_status(ws) == 0
    assert [int(x) for x in pc.as_u64(out["hits"])] == want


def test_invalid_next_is_reported_and_stays_in_bounds():
    nxt = np.array([5, 1, 0xFFFFFFFF, 2, 100, 0xFFFFFFFF], np.uint32)   # t=1 points at itself, t=3 back, t=4 past n
    out, ws = pc.belady(pc.to_dev_u32(nxt), pc.to_dev_u64(np.array([1, 2000], np.uint64)))
    torch.cuda.synchronize()
    assert pc.workspace_status(ws) == 2
