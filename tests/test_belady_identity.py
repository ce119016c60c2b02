"""The closed form the Belady kernel uses to decide a batch's evictions at
once, against the access-by-access greedy it replaces (CPU, pure Python).

A batch is up to 64 accesses.  An eviction (a miss once the cache is full)
takes a dead block (no further use) while there is one, else the largest
candidate present: the buffer's candidates are present from the start, an
insert of the batch from the access after its own.  Candidates are named by
their joint rank (0 = largest).  The closed form: the evictions left after
the dead blocks are where the running maximum of (evictions so far) − (dead
blocks available) grows; for each rank k, R(k) = min(E, A(k) + E + m(k)) is
the number of evictions that take a candidate ranked below k (A(k): buffer
candidates below k, m(k): lowest prefix sum of "−1 per eviction, then +1 per
insert ranked below k"), and rank k is taken iff R(k + 1) > R(k).  The batch
needs the general walk when an eviction finds no candidate below `nhigh`."""
import random

import pytest


def greedy(nb, ev, dm, d0, b_ranks, pend, nhigh):
    """Access by access (the kernel's former walk)."""
    present = set(b_ranks)
    gone = set()
    d = d0
    for j in range(nb):
        if (ev >> j) & 1:
            if d:
                d -= 1
            else:
                cand = sorted(present - gone)
                if not cand or cand[0] >= nhigh:
                    return False, None, None
                gone.add(cand[0])
        if (dm >> j) & 1:
            d += 1
        elif j in pend:
            present.add(pend[j])
    return True, gone, d


def closed_form(nb, ev, dm, d0, b_ranks, pend, nhigh):
    popc = lambda x: bin(x).count("1")
    real = 0
    best = 0
    for j in range(nb):
        gap = popc(ev & ((2 << j) - 1)) - d0 - popc(dm & ((1 << j) - 1))
        if gap > best:
            real |= 1 << j
            best = gap
    E = popc(real)
    d = d0 + popc(dm) - (popc(ev) - E)

    def R(k):
        a = sum(1 for r in b_ranks if r < k)
        ins = 0
        for j, r in pend.items():
            if r < k:
                ins |= 1 << j
        run = low = 0
        for j in range(nb):
            run -= (real >> j) & 1
            low = min(low, run)
            run += (ins >> j) & 1
        return min(E, a + E + low)

    Rs = [R(k) for k in range(129)]
    if Rs[min(nhigh, 128)] != E:
        return False, None, None
    return True, {k for k in range(128) if Rs[k + 1] > Rs[k]}, d


def random_batch(rng):
    nb = rng.randint(1, 64)
    nbt = rng.randint(0, 64)
    steps = list(range(nb))
    dead_steps = set(rng.sample(steps, rng.randint(0, nb // 3)))
    pend_steps = [j for j in steps if j not in dead_steps and rng.random() < 0.7]
    ranks = list(range(nbt + len(pend_steps)))
    rng.shuffle(ranks)
    b_ranks = sorted(ranks[:nbt])
    pend = dict(zip(pend_steps, ranks[nbt:]))
    p = rng.choice([0.2, 0.6, 0.95, 1.0])
    ev = sum(1 << j for j in steps if rng.random() < p)
    dm = sum(1 << j for j in dead_steps)
    d0 = rng.choice([0, 0, 1, 3, 10])
    tot = len(ranks)
    nhigh = rng.randint(0, tot) if rng.random() < 0.5 else tot
    return nb, ev, dm, d0, b_ranks, pend, nhigh


@pytest.mark.parametrize("seed", range(4))
def test_closed_form_equals_the_greedy(seed):
    rng = random.Random(seed)
    for _ in range(500):
        batch = random_batch(rng)
        assert closed_form(*batch) == greedy(*batch), batch


def test_hand_worked_batch():
    # three evictions, no dead block: the buffer's candidate (rank 1) goes
    # first, then the first access's insert (rank 0); the third finds nothing
    # ranked below nhigh, and the walk takes over
    assert greedy(3, 0b111, 0, 0, [1], {0: 0}, 2) == (False, None, None)
    assert closed_form(3, 0b111, 0, 0, [1], {0: 0}, 2) == (False, None, None)
    # one dead block waiting: it serves the first eviction, the second takes
    # the first access's insert (rank 0, larger than the buffer's), the third
    # the buffer's candidate
    assert greedy(3, 0b111, 0, 1, [1], {0: 0}, 2) == (True, {0, 1}, 0)
    assert closed_form(3, 0b111, 0, 1, [1], {0: 0}, 2) == (True, {0, 1}, 0)
