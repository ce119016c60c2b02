"""The torch fingerprints used by the full-size GPU tests agree with the
oracle's (CPU, torch on the host)."""
import numpy as np
import torch

import oracle
from conftest import read_golden
from fingerprints import array_fp, hit_fps, mix64, to_u64


def test_torch_mix64_matches_published_splitmix64_outputs():
    G = 0x9E3779B97F4A7C15
    for k, out in read_golden("splitmix64_seed0.txt"):
        z = torch.tensor([((int(k) * G) % (1 << 64)) - ((1 << 64) if (int(k) * G) % (1 << 64) >= 1 << 63 else 0)])
        assert to_u64(mix64(z)[0]) == int(out, 16)


def test_array_fingerprints_match_oracle():
    rng = np.random.default_rng(3)
    a32 = rng.integers(0, 2 ** 32, size=100_003, dtype=np.uint64).astype(np.uint32)
    a32[::7] = 0xFFFFFFFF
    a64 = rng.integers(0, 2 ** 63, size=50_001, dtype=np.int64).astype(np.uint64) * np.uint64(3)
    assert array_fp(torch.from_numpy(a32.view(np.int32))) == oracle.fingerprint(a32)
    assert array_fp(torch.from_numpy(a64.view(np.int64))) == oracle.fingerprint(a64)
    # pieces add up
    assert (oracle.fingerprint(a32[:1000]) + oracle.fingerprint(a32[1000:], t0=1000)) % 2 ** 64 == \
        oracle.fingerprint(a32)
    # one changed element changes the fingerprint
    b = a32.copy()
    b[500] ^= 1
    assert oracle.fingerprint(b) != oracle.fingerprint(a32)


def test_hit_fingerprints_match_oracle_simulation():
    # a small chained trace: LRU simulations per capacity (with hit-set
    # fingerprints) against the torch binning of the oracle's distances
    import pcgen
    tr = pcgen.make_trace("tiny")
    keys, depth = oracle.hash_trace(tr)
    caps = tr.caps()
    prev, _ = oracle.prev_next(keys)
    d = oracle.stack_distance_bit(prev)
    want = [(h, fp) for h, _, fp in oracle.lru(keys, [int(c) for c in caps], depth, fingerprints=True, threads=4)]
    got = hit_fps(torch.from_numpy(d.view(np.int32)), torch.from_numpy(caps.astype(np.int64)))
    assert got == want
    # and the oracle's own binning of the distances
    cnt, fp = oracle.dist_bins(d, caps)
    assert [int(x) for x in np.cumsum(cnt[:-1])] == [h for h, _ in want]
    assert [int(x) for x in np.cumsum(fp[:-1], dtype=np.uint64)] == [f for _, f in want]
    # the fingerprint names which accesses hit: sum of mix64(t + 1) over the
    # flagged accesses of a simulation
    (h, _, fp, fl), = oracle.lru(keys, [int(caps[20])], depth, flags=True, fingerprints=True)
    t = np.nonzero(fl)[0]
    assert h == t.size and fp == sum(oracle.mix64(int(x) + 1) for x in t) % 2 ** 64
