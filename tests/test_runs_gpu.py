"""pc_stack_distance_runs against the oracle's stack distance (element by
element): chained traces in both block layouts, streams built from copied
segments (many runs of every length, still on the runs path), streams
without run structure (the call must take pc_stack_distance), degenerate
streams, ragged sizes and an unaligned view."""
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


def runs_dist(prev, nxt, offset=0):
    """Distances through the C ABI; `offset` shifts the device views by that
    many elements (an unaligned start)."""
    n = prev.size
    pd = torch.empty(n + offset, dtype=torch.int32, device="cuda")[offset:]
    nd = torch.empty(n + offset, dtype=torch.int32, device="cuda")[offset:]
    pd.copy_(torch.from_numpy(prev.view(np.int32)))
    nd.copy_(torch.from_numpy(nxt.view(np.int32)))
    dd = torch.empty(n + offset, dtype=torch.int32, device="cuda")[offset:]
    _, ws = pc.stack_distance_runs(pd, nd, dd)
    info = pc.runs_info(ws)
    return pc.as_u32(dd), info, pc.workspace_status(ws)


def exact(keys, offset=0):
    p, q = oracle.prev_next(keys)
    want = oracle.stack_distance_bit(p)
    got, info, status = runs_dist(p, q, offset)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, (bad.size, bad[:5], info)
    assert status == 0
    # the runs path holds up to n/16 + 1024 runs
    assert info["runs"] == runs_of(p)
    assert info["generic"] == (info["runs"] > keys.size // 16 + 1024), info
    return info


def runs_of(prev):
    p = prev.astype(np.int64)
    warm = prev != NONE
    cont = np.zeros(prev.size, bool)
    cont[1:] = warm[1:] & warm[:-1] & (p[1:] == p[:-1] + 1)
    return int((warm & ~cont).sum())


@pytest.fixture(scope="module", params=[("tiny", None), ("agent", 300), ("chat", 400)])
def trace_keys(request):
    assert torch.cuda.is_available()
    name, ns = request.param
    tr = pcgen.make_trace(name, n_sessions=ns) if ns else pcgen.make_trace(name)
    keys, _ = oracle.hash_trace(tr)
    return name, keys, tr.blk_off(16).astype(np.int64)


def test_chained_traces_take_the_runs_path(trace_keys):
    name, keys, off = trace_keys
    info = exact(keys)
    say(name, keys.size, info)
    assert not info["generic"]


def test_deepest_first_layout(trace_keys):
    name, keys, off = trace_keys
    L = np.diff(off)
    r = np.repeat(np.arange(L.size), L)
    perm = off[r] + off[r + 1] - 1 - np.arange(keys.size, dtype=np.int64)
    info = exact(keys[perm])
    assert not info["generic"]


def copied_segments(rng, n, max_len, fresh):
    """A key stream that repeatedly copies a random earlier segment (or emits
    fresh keys with probability `fresh`)."""
    out = []
    size = 0
    nxt_key = 0
    while size < n:
        ln = int(rng.integers(1, max_len + 1))
        if size == 0 or rng.random() < fresh:
            seg = np.arange(nxt_key, nxt_key + ln, dtype=np.uint64)
            nxt_key += ln
        else:
            a = int(rng.integers(0, size))
            allk = np.concatenate(out)
            seg = allk[a:a + ln]
        out.append(seg)
        size += seg.size
    return np.concatenate(out)[:n]


@pytest.mark.parametrize("n,max_len,fresh", [(50_000, 200, 0.2), (300_001, 64, 0.1), (123_457, 1000, 0.5),
                                             (400_000, 4000, 0.3)])
def test_copied_segments(n, max_len, fresh):
    rng = np.random.default_rng(n)
    keys = copied_segments(rng, n, max_len, fresh)
    info = exact(keys)
    say(n, info)


@pytest.mark.parametrize("kinds", [3, 1000, None])
def test_streams_without_runs_fall_back(kinds):
    rng = np.random.default_rng(9)
    n = 200_003
    keys = (rng.integers(0, kinds, n) if kinds else rng.integers(0, 2 ** 63, n)).astype(np.uint64)
    info = exact(keys)
    say(kinds, info)


@pytest.mark.parametrize("case", ["one", "cold", "same", "alternate", "ragged", "ragged_unaligned"])
def test_degenerate_and_ragged(case):
    rng = np.random.default_rng(4)
    if case == "one":
        keys = np.array([7], np.uint64)
    elif case == "cold":
        keys = np.arange(10_000, dtype=np.uint64)
    elif case == "same":
        keys = np.zeros(9_999, np.uint64)          # one run: prev(t) = t - 1
    elif case == "alternate":
        keys = (np.arange(10_001) % 2).astype(np.uint64)   # one run: prev(t) = t - 2
    else:
        keys = copied_segments(rng, 4096 * 3 + 17, 300, 0.3)
    info = exact(keys, offset=1 if case == "ragged_unaligned" else 0)
    say(case, info)
