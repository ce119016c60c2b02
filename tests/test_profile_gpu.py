"""Parity of the workload characterisation (Sec. 4) through the C ABI
against the CPU oracle: reuse-interval, lifetime, frequency and
lifetime-by-frequency-class histograms over blocks, and footprint,
request-count, duration and gap histograms over sessions.  All integer,
all bit-exact."""
import sys

import numpy as np
import pytest
import torch

import oracle
import pcgen
from conftest import characterization_golden
from paper_2609_28870_amd import pc

pytestmark = pytest.mark.gpu
EDGES = [1, 10, 100, 1000, 10 ** 4, 10 ** 5, 10 ** 6, 10 ** 7, 10 ** 8, 10 ** 9, 10 ** 10]


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def gpu_profiles(keys, blk_off, sess, ts, edges, freq_max, fp_max, rq_max):
    kd = pc.to_dev_u64(keys)
    bo = pc.to_dev_u64(blk_off)
    td = pc.to_dev_u64(ts)
    ed = pc.to_dev_u64(np.asarray(edges, np.uint64))
    prev, nxt, ws = pc.prev_next_use(kd)
    assert pc.workspace_status(ws) == 0
    rp, ws = pc.reuse_profile(prev, nxt, bo, td, ed, freq_max)
    assert pc.workspace_status(ws) == 0
    sp, ws = pc.session_profile(bo, pc.to_dev_u32(sess), td, keys.size, ed, fp_max, rq_max)
    assert pc.workspace_status(ws) == 0
    return pc.hists_to_host(rp), pc.hists_to_host(sp)


def check_profiles(keys, blk_off, sess, ts, edges=EDGES, freq_max=64, fp_max=20000, rq_max=64, label=""):
    keys = np.asarray(keys, np.uint64)
    say("case", label, "n", keys.size, "requests", len(blk_off) - 1)
    g_rp, g_sp = gpu_profiles(keys, blk_off, sess, ts, edges, freq_max, fp_max, rq_max)
    o_rp = oracle.reuse_profile(keys, blk_off, ts, edges, freq_max)
    o_sp = oracle.session_profile(blk_off, sess, ts, edges, fp_max, rq_max)
    for name in o_rp:
        assert g_rp[name] == o_rp[name], (label, name)
    for name in o_sp:
        assert g_sp[name] == o_sp[name], (label, name)
    return g_rp, g_sp


def test_hand_worked_example():
    keys, blk_off, sess, ts, want = characterization_golden()
    rp, sp = gpu_profiles(keys, blk_off, sess, ts, want["edges"], want["freq_max"][0], want["footprint_max"][0],
                          want["requests_max"][0])
    assert rp["interval"] == want["interval"] and rp["lifetime"] == want["lifetime"]
    assert rp["freq"] == want["freq"]
    k = len(want["edges"]) + 1
    assert rp["life_by_class"][:k] == want["class0"] and rp["life_by_class"][k:2 * k] == want["class1"]
    for name in ("footprint", "requests", "duration", "gap"):
        assert sp[name] == want[name], name


@pytest.mark.parametrize("config,sessions", [("tiny", None), ("agent", 250), ("chat", 1500)])
def test_trace_profiles(config, sessions):
    tr = pcgen.make_trace(config, n_sessions=sessions) if sessions else pcgen.make_trace(config)
    keys, _ = oracle.hash_trace(tr)
    check_profiles(keys, tr.blk_off(16), tr.session.astype(np.uint32), tr.ts_us.astype(np.uint64),
                   label="%s%s" % (config, sessions or ""))


def test_small_bins_and_tails():
    tr = pcgen.make_trace("agent", n_sessions=250)
    keys, _ = oracle.hash_trace(tr)
    # one edge, frequency and request tails at 1 and 3, footprint tail at 2
    check_profiles(keys, tr.blk_off(16), tr.session.astype(np.uint32), tr.ts_us.astype(np.uint64),
                   edges=[1000000], freq_max=3, fp_max=2, rq_max=1, label="tails")


def test_long_chains_next_to_short_ones():
    """One block read 200,000 times among many one-off and short-lived
    blocks: the lane walking it must not hold up the others' results."""
    rng = np.random.default_rng(3)
    n = 600000
    keys = rng.integers(1, 2 ** 62, size=n, dtype=np.uint64)
    keys[rng.random(n) < 1 / 3] = np.uint64(42)
    mid = rng.random(n) < 0.2
    keys[mid] = np.uint64(1000) + rng.integers(0, 50, size=int(mid.sum()), dtype=np.uint64)
    bo = np.arange(0, n + 1, 100, dtype=np.uint64)
    ns = bo.size - 1
    sess = (np.arange(ns) % 37).astype(np.uint32)
    ts = np.cumsum(rng.integers(0, 5000, size=ns)).astype(np.uint64)
    g_rp, _ = check_profiles(keys, bo, sess, ts, freq_max=2048, label="long-chain")
    assert g_rp["freq"][2048] >= 1


def test_edge_cases():
    e = [5]
    # no accesses at all (requests present but empty)
    check_profiles(np.zeros(0, np.uint64), np.array([0, 0, 0], np.uint64), np.array([1, 1], np.uint32),
                   np.array([3, 9], np.uint64), edges=e, label="empty")
    # a single access; a single request; equal timestamps
    check_profiles(np.array([9], np.uint64), np.array([0, 1], np.uint64), np.array([0], np.uint32),
                   np.array([0], np.uint64), edges=e, label="one")
    keys = np.tile(np.arange(1, 501, dtype=np.uint64), 4)
    check_profiles(keys, np.array([0, 500, 1000, 1500, 2000], np.uint64), np.array([3, 3, 4, 3], np.uint32),
                   np.array([7, 7, 7, 7], np.uint64), edges=[1, 2], label="same-time")


def test_bad_arguments_reported():
    keys = np.arange(1, 101, dtype=np.uint64)
    prev, nxt, _ = pc.prev_next_use(pc.to_dev_u64(keys))
    bo = pc.to_dev_u64(np.array([0, 50, 100], np.uint64))
    ts = pc.to_dev_u64(np.array([0, 1], np.uint64))
    sess = pc.to_dev_u32(np.array([0, 1], np.uint32))
    bad_edges = pc.to_dev_u64(np.array([10, 5], np.uint64))
    _, ws = pc.reuse_profile(prev, nxt, bo, ts, bad_edges, 8)
    assert pc.workspace_status(ws) == 3
    _, ws = pc.session_profile(bo, sess, ts, 100, bad_edges, 8, 8)
    assert pc.workspace_status(ws) == 3
    good = pc.to_dev_u64(np.array([5], np.uint64))
    _, ws = pc.reuse_profile(prev, nxt, pc.to_dev_u64(np.array([0, 50, 99], np.uint64)), ts, good, 8)
    assert pc.workspace_status(ws) == 2


def test_profiler_pipeline_matches_the_stages():
    tr = pcgen.make_trace("tiny")
    up = pc.upload_trace(tr)
    edges = pc.to_dev_u64(np.array(EDGES, np.uint64))
    p = pc.Profiler(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"], up["session"],
                    up["ts_us"], edges, freq_max=64, fp_max=20000, rq_max=64)
    p.run()
    torch.cuda.synchronize()
    assert p.status() == {"hash": 0, "prev_next": 0, "reuse_profile": 0, "session_profile": 0}
    keys, _ = oracle.hash_trace(tr)
    o_rp = oracle.reuse_profile(keys, tr.blk_off(16), tr.ts_us.astype(np.uint64), EDGES, 64)
    o_sp = oracle.session_profile(tr.blk_off(16), tr.session, tr.ts_us.astype(np.uint64), EDGES, 20000, 64)
    assert pc.hists_to_host(p.reuse) == o_rp
    assert pc.hists_to_host(p.sessions) == o_sp
