"""The lookup the bins kernel uses to take each block's depth from the request
layout, against the depth computed directly (CPU, numpy).

The map: a bitmap with a bit at every request start (deepest-first layout:
at every request's last position) and, per 64 positions, the start of the
request holding the word's first position (deepest first: the last position
of the request holding the word's last position).  A thread of PER
consecutive accesses starting at t0 (a multiple of PER) takes the last start
at or below t0 in its 64-position word, else the word's entry, and follows
the start bits up; deepest first, the first end at or above its last access,
else the word's entry, and follows the end bits down."""
import numpy as np
import pytest


def direct(off, desc):
    L = np.diff(off)
    n = int(off[-1])
    pos = np.arange(n, dtype=np.int64)
    if desc:
        return np.repeat(off[1:] - 1, L) - pos
    return pos - np.repeat(off[:-1], L)


def build_map(off, desc):
    n = int(off[-1])
    words = (n + 63) // 64
    bits = np.zeros(words * 64, bool)
    table = np.full(words, -1, np.int64)
    for r in range(off.size - 1):
        a, b = int(off[r]), int(off[r + 1])
        if a == b:
            continue
        if not desc:
            bits[a] = True
            w = (a + 63) // 64
            while w * 64 < b:
                table[w] = a
                w += 1
        else:
            bits[b - 1] = True
            w = a // 64
            while w < words:
                last = min(64 * w + 63, n - 1)
                if last >= b:
                    break
                table[w] = b - 1
                w += 1
    assert (table >= 0).all()
    return bits, table


def lookup(bits, table, n, per, desc):
    out = np.zeros(n, np.int64)
    for t0 in range(0, n, per):
        wd, sh = t0 // 64, t0 % 64
        word = bits[wd * 64:(wd + 1) * 64]
        if not desc:
            upto = np.nonzero(word[:sh + 1])[0]
            st = wd * 64 + upto[-1] if upto.size else table[wd]
            for j in range(per):
                if j and word[sh + j]:
                    st = t0 + j
                if t0 + j < n:
                    out[t0 + j] = t0 + j - st
        else:
            frm = np.nonzero(word[sh + per - 1:])[0]
            en = wd * 64 + sh + per - 1 + frm[0] if frm.size else table[wd]
            for j in range(per - 1, -1, -1):
                if j < per - 1 and word[sh + j]:
                    en = t0 + j
                if t0 + j < n:
                    out[t0 + j] = en - (t0 + j)
    return out


def random_layout(rng, n, kind):
    L = []
    while sum(L) < n:
        if kind == "empty" and rng.random() < 0.3:
            L.append(0)
        L.append(int(rng.integers(1, {"short": 12, "mixed": 200, "empty": 70}[kind])))
    L[-1] -= sum(L) - n
    if kind == "empty":
        L = [0] + L + [0]
    return np.concatenate([[0], np.cumsum(L)]).astype(np.int64)


@pytest.mark.parametrize("desc", [False, True])
@pytest.mark.parametrize("per", [8, 16])
@pytest.mark.parametrize("kind", ["short", "mixed", "empty"])
def test_lookup_equals_the_direct_depth(kind, per, desc):
    rng = np.random.default_rng(["short", "mixed", "empty"].index(kind) * 4 + (per // 8) * 2 + int(desc))
    for n in (1, 7, 8, 15, 16, 63, 64, 65, 127, 128, 129, 1000, 4099):
        off = random_layout(rng, n, kind)
        bits, table = build_map(off, desc)
        assert np.array_equal(lookup(bits, table, n, per, desc), direct(off, desc)), (kind, per, desc, n)


@pytest.mark.parametrize("desc", [False, True])
def test_one_request_and_single_blocks(desc):
    for off in (np.array([0, 300]), np.arange(0, 201), np.array([0, 0, 64, 64, 128, 129, 300, 300])):
        n = int(off[-1])
        bits, table = build_map(off, desc)
        for per in (8, 16):
            assert np.array_equal(lookup(bits, table, n, per, desc), direct(off, desc)), (off[:5], per)
