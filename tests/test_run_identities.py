"""The identities the stack distance over runs rests on, checked with the
oracle's distances on the CPU: along a run (prev(t) = prev(t-1) + 1, both
warm) the distance does not change, and at a run head the count of earlier
warm accesses with an older previous use is the summed length of the earlier
runs whose previous-use range starts lower (those ranges are disjoint)."""
import numpy as np
import pytest

import oracle
import pcgen

NONE = oracle.NONE


def runs(prev):
    p = prev.astype(np.int64)
    warm = prev != NONE
    cont = np.zeros(prev.size, bool)
    cont[1:] = warm[1:] & warm[:-1] & (p[1:] == p[:-1] + 1)
    heads = np.nonzero(warm & ~cont)[0]
    ends = np.empty_like(heads)
    for i, h in enumerate(heads):
        e = h
        while e + 1 < prev.size and cont[e + 1]:
            e += 1
        ends[i] = e
    return cont, heads, ends


def streams():
    rng = np.random.default_rng(2)
    yield "random 40", rng.integers(0, 40, 3000).astype(np.uint64)
    yield "random 3", rng.integers(0, 3, 2000).astype(np.uint64)
    # copied segments
    out = [np.arange(50, dtype=np.uint64)]
    nxt = 50
    for _ in range(120):
        allk = np.concatenate(out)
        if rng.random() < 0.3:
            ln = int(rng.integers(1, 30))
            out.append(np.arange(nxt, nxt + ln, dtype=np.uint64))
            nxt += ln
        else:
            a = int(rng.integers(0, allk.size))
            out.append(allk[a:a + int(rng.integers(1, 80))])
    yield "copied segments", np.concatenate(out)
    tr = pcgen.make_trace("tiny")
    yield "tiny trace", oracle.hash_trace(tr)[0][:20000]


@pytest.mark.parametrize("name,keys", list(streams()))
def test_distance_is_constant_along_runs(name, keys):
    prev, _ = oracle.prev_next(keys)
    d = oracle.stack_distance_walk(keys)
    cont, _, _ = runs(prev)
    assert cont.any() or name.startswith("random")
    assert np.array_equal(d[1:][cont[1:]], d[:-1][cont[1:]])


@pytest.mark.parametrize("name,keys", list(streams()))
def test_head_distance_from_earlier_runs(name, keys):
    prev, _ = oracle.prev_next(keys)
    d = oracle.stack_distance_walk(keys)
    _, heads, ends = runs(prev)
    p = prev[heads].astype(np.int64)
    ln = (ends - heads + 1).astype(np.int64)
    cold_before = np.concatenate([[0], np.cumsum(prev == NONE)])
    for i, h in enumerate(heads):
        # previous-use ranges of different runs never overlap
        if i:
            lo, hi = p[:i], p[:i] + ln[:i]
            assert np.all((hi <= p[i]) | (lo >= p[i] + ln[i]))
        c = int(ln[:i][p[:i] < p[i]].sum())
        assert d[h] == cold_before[h] + c - p[i] - 1, (name, h)
