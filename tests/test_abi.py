"""The C ABI: libpc loads, exports every function include/pc.h declares, and
rejects bad arguments before touching the device.  CPU only (no compute)."""
import ctypes
import os
import re

import pytest

from paper_2609_28870_amd import pc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "pc.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(pc_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(pc.LIB_PATH):
        pytest.fail("libpc.so is not built (run __graft_entry__.build())")
    return pc.lib()


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert len(names) >= 15
    for name in names:
        assert hasattr(L, name), name


def test_status_strings(L):
    for code in (0, -1, -2, -3, -4, -5):
        assert L.pc_status_string(code)
    assert L.pc_version() >= 100


def test_workspace_queries_grow_with_n(L):
    a = L.pc_prev_next_use_ws(1000)
    b = L.pc_prev_next_use_ws(10 ** 6)
    assert 0 < a < b
    assert L.pc_stack_distance_ws(10 ** 6) > L.pc_stack_distance_ws(1000) > 0
    assert L.pc_hash_blocks_ws(10) >= 256
    assert L.pc_mrc_weighted_ws(10, 69) >= 256


FAKE = ctypes.c_void_p(0x1000)   # never dereferenced: every call below fails validation


def test_hash_rejects_bad_arguments(L):
    ws = L.pc_hash_blocks_ws(4)
    args = lambda B=16, n_seqs=4, nb=100, wsz=ws, tokens=FAKE, w=FAKE: (
        tokens, 1000, FAKE, FAKE, n_seqs, B, None, 0, FAKE, nb, FAKE, None, None, 0, w, wsz, None)
    assert L.pc_hash_blocks(*args(B=15)) == -1
    assert L.pc_hash_blocks(*args(B=0)) == -1
    assert L.pc_hash_blocks(*args(B=2048)) == -1
    assert L.pc_hash_blocks(*args(n_seqs=0x80000000)) == -2
    assert L.pc_hash_blocks(*args(nb=0xFFFFFFFF)) == -2
    assert L.pc_hash_blocks(*args(tokens=None)) == -1
    assert L.pc_hash_blocks(*args(w=None)) == -3
    assert L.pc_hash_blocks(*args(wsz=ws - 1)) == -3


def test_prev_next_rejects_bad_arguments(L):
    n = 1000
    ws = L.pc_prev_next_use_ws(n)
    assert L.pc_prev_next_use(FAKE, 0xFFFFFFFF, FAKE, FAKE, None, FAKE, 1 << 40, None) == -2
    assert L.pc_prev_next_use(None, n, FAKE, FAKE, None, FAKE, ws, None) == -1
    assert L.pc_prev_next_use(FAKE, n, FAKE, None, None, FAKE, ws, None) == -1
    assert L.pc_prev_next_use(FAKE, n, FAKE, FAKE, None, None, ws, None) == -3
    assert L.pc_prev_next_use(FAKE, n, FAKE, FAKE, None, FAKE, ws - 1, None) == -3


def test_prev_next_chained_rejects_bad_arguments(L):
    n, seqs = 1000, 10
    ws = L.pc_prev_next_chained_ws(n, seqs)
    assert ws > L.pc_prev_next_use_ws(n)
    assert L.pc_prev_next_chained(FAKE, 0xFFFFFFFF, FAKE, seqs, 0, FAKE, FAKE, None, FAKE, 1 << 40, None) == -2
    assert L.pc_prev_next_chained(None, n, FAKE, seqs, 0, FAKE, FAKE, None, FAKE, ws, None) == -1
    assert L.pc_prev_next_chained(FAKE, n, None, seqs, 0, FAKE, FAKE, None, FAKE, ws, None) == -1
    assert L.pc_prev_next_chained(FAKE, n, FAKE, seqs, 0, FAKE, None, None, FAKE, ws, None) == -1
    assert L.pc_prev_next_chained(FAKE, n, FAKE, seqs, 4, FAKE, FAKE, None, FAKE, ws, None) == -1   # unknown flag
    assert L.pc_prev_next_chained(FAKE, n, FAKE, seqs, 2, FAKE, None, None, FAKE, ws, None) == -1   # prev-only: next still required
    assert L.pc_prev_next_chained(FAKE, n, FAKE, seqs, 0, FAKE, FAKE, None, None, ws, None) == -3
    assert L.pc_prev_next_chained(FAKE, n, FAKE, seqs, 0, FAKE, FAKE, None, FAKE, ws - 1, None) == -3


def test_stack_distance_runs_rejects_bad_arguments(L):
    n = 1000
    ws = L.pc_stack_distance_runs_ws(n)
    assert ws >= L.pc_stack_distance_ws(n)
    assert L.pc_stack_distance_runs(FAKE, FAKE, 0xFFFFFFFF, FAKE, FAKE, 1 << 40, None) == -2
    assert L.pc_stack_distance_runs(None, FAKE, n, FAKE, FAKE, ws, None) == -1
    assert L.pc_stack_distance_runs(FAKE, None, n, FAKE, FAKE, ws, None) == -1
    assert L.pc_stack_distance_runs(FAKE, FAKE, n, None, FAKE, ws, None) == -1
    assert L.pc_stack_distance_runs(FAKE, FAKE, n, FAKE, None, ws, None) == -3
    assert L.pc_stack_distance_runs(FAKE, FAKE, n, FAKE, FAKE, ws - 1, None) == -3


def test_stack_distance_rejects_bad_arguments(L):
    n = 5000
    ws = L.pc_stack_distance_ws(n)
    assert L.pc_stack_distance(FAKE, FAKE, 0xFFFFFFFF, FAKE, FAKE, 1 << 40, None) == -2
    assert L.pc_stack_distance(FAKE, None, n, FAKE, FAKE, ws, None) == -1
    assert L.pc_stack_distance(FAKE, FAKE, n, None, FAKE, ws, None) == -1
    assert L.pc_stack_distance(FAKE, FAKE, n, FAKE, FAKE, ws - 1, None) == -3


def test_request_order_rejects_bad_arguments(L):
    ws = L.pc_request_order_ws()
    assert ws >= 256
    call = lambda keys=FAKE, depth=None, bo=FAKE, ns=4, n=10, ko=ctypes.c_void_p(0x2000), do=None, w=FAKE, \
        wsz=ws: L.pc_request_order(keys, depth, bo, ns, n, ko, do, w, wsz, None)
    assert call(n=0xFFFFFFFF) == -2
    assert call(keys=None) == -1
    assert call(bo=None) == -1
    assert call(ko=None) == -1
    assert call(depth=FAKE) == -1                     # depth without depth_out
    assert call(ko=FAKE) == -1                        # output aliases input
    assert call(depth=FAKE, do=FAKE) == -1
    assert call(w=None) == -3
    assert call(wsz=ws - 1) == -3


def test_stack_distance_req_rejects_bad_arguments(L):
    n = 5000
    ws = L.pc_stack_distance_req_ws()
    assert ws >= 256
    call = lambda prev=FAKE, ns=40, n=n, out=FAKE, w=FAKE, wsz=ws: L.pc_stack_distance_req(
        prev, FAKE, FAKE, ns, n, out, w, wsz, None)
    assert call(n=0xFFFFFFFF) == -2
    assert call(ns=0x80000000) == -2
    assert call(prev=None) == -1
    assert call(out=None) == -1
    assert call(ns=0) == -1
    assert call(w=None) == -3
    assert call(wsz=ws - 1) == -3


def test_stack_distance_session_rejects_bad_arguments(L):
    n = 5000
    ws = L.pc_stack_distance_session_ws(n, 40)
    assert ws >= L.pc_prev_next_use_ws(40)
    assert L.pc_stack_distance_session_ws(10 ** 8, 40) > ws
    call = lambda prev=FAKE, bo=FAKE, sess=FAKE, ns=40, n=n, out=FAKE, w=FAKE, wsz=ws: \
        L.pc_stack_distance_session(prev, bo, sess, ns, n, out, w, wsz, None)
    assert call(n=0xFFFFFFFF) == -2
    assert call(ns=0x80000000) == -2
    assert call(prev=None) == -1
    assert call(bo=None) == -1
    assert call(sess=None) == -1
    assert call(out=None) == -1
    assert call(ns=0) == -1
    assert call(w=None) == -3
    assert call(wsz=ws - 1) == -3


def test_profiles_reject_bad_arguments(L):
    n = 5000
    ws = L.pc_reuse_profile_ws(n)
    assert ws >= 8 * n
    rp = lambda prev=FAKE, ns=40, n=n, k=4, fm=16, out=FAKE, w=FAKE, wsz=ws: L.pc_reuse_profile(
        prev, FAKE, FAKE, FAKE, ns, n, FAKE, k, fm, out, FAKE, FAKE, FAKE, w, wsz, None)
    assert rp(n=0xFFFFFFFF) == -2
    assert rp(ns=0x80000000) == -2
    assert rp(k=0) == -1
    assert rp(k=129) == -1
    assert rp(fm=0) == -1
    assert rp(fm=2049) == -1
    assert rp(prev=None) == -1
    assert rp(out=None) == -1
    assert rp(ns=0) == -1
    assert rp(w=None) == -3
    assert rp(wsz=ws - 1) == -3
    ws = L.pc_session_profile_ws(40)
    sp = lambda bo=FAKE, ns=40, k=4, fp=16, rq=16, out=FAKE, w=FAKE, wsz=ws: L.pc_session_profile(
        bo, FAKE, FAKE, ns, n, FAKE, k, fp, rq, out, FAKE, FAKE, FAKE, w, wsz, None)
    assert sp(ns=0x80000000) == -2
    assert sp(k=0) == -1
    assert sp(rq=2049) == -1
    assert sp(fp=0) == -1
    assert sp(fp=(1 << 24) + 1) == -1
    assert sp(bo=None) == -1
    assert sp(out=None) == -1
    assert sp(w=None) == -3
    assert sp(wsz=ws - 1) == -3


def test_mrc_rejects_bad_arguments(L):
    ws = L.pc_mrc_weighted_ws(10, 4)
    ok = lambda **kw: dict(dict(dist=FAKE, depth=None, nxt=None, n=10, caps=FAKE, k=4, a=1, b=0,
                                cnt=FAKE, ds=FAKE, lo=FAKE, hi=FAKE, nh=None, w=FAKE, wsz=ws), **kw)
    call = lambda d: L.pc_mrc_weighted(d["dist"], d["depth"], d["nxt"], d["n"], d["caps"], d["k"],
                                       d["a"], d["b"], d["cnt"], d["ds"], d["lo"], d["hi"], d["nh"],
                                       d["w"], d["wsz"], None)
    assert call(ok(k=0)) == -1
    assert call(ok(k=4097)) == -1
    assert call(ok(caps=None)) == -1
    assert call(ok(nxt=FAKE)) == -1          # next without nextuse_hist
    assert call(ok(n=0xFFFFFFFF)) == -2
    assert call(ok(w=None)) == -3


def test_mrc_layout_rejects_bad_arguments(L):
    ws = L.pc_mrc_weighted_layout_ws(10, 4)
    assert ws > L.pc_mrc_weighted_layout_ws(0, 4)
    ok = lambda **kw: dict(dict(dist=FAKE, off=FAKE, seqs=2, fl=0, nxt=None, n=10, caps=FAKE, k=4, a=1, b=0,
                                cnt=FAKE, ds=FAKE, lo=FAKE, hi=FAKE, nh=None, w=FAKE, wsz=ws), **kw)
    call = lambda d: L.pc_mrc_weighted_layout(d["dist"], d["off"], d["seqs"], d["fl"], d["nxt"], d["n"], d["caps"],
                                              d["k"],
                                              d["a"], d["b"], d["cnt"], d["ds"], d["lo"], d["hi"], d["nh"],
                                              d["w"], d["wsz"], None)
    assert call(ok(off=None)) == -1
    assert call(ok(fl=2)) == -1
    assert call(ok(k=0)) == -1
    assert call(ok(k=4097)) == -1
    assert call(ok(nxt=FAKE)) == -1
    assert call(ok(n=0xFFFFFFFF)) == -2
    assert call(ok(w=None)) == -3
    assert call(ok(wsz=ws - 1)) == -3


def test_belady_rejects_bad_arguments(L):
    ws = L.pc_belady_ws(1000, 4)
    assert ws > L.pc_belady_ws(10, 4) > 0
    ok = lambda **kw: dict(dict(nxt=FAKE, depth=None, n=1000, caps=FAKE, k=4, hits=FAKE, ds=FAKE, fl=None,
                                w=FAKE, wsz=ws), **kw)
    call = lambda d: L.pc_belady(d["nxt"], d["depth"], d["n"], d["caps"], d["k"], d["hits"], d["ds"], d["fl"],
                                 d["w"], d["wsz"], None)
    assert call(ok(k=0)) == -1
    assert call(ok(k=4097)) == -1
    assert call(ok(caps=None)) == -1
    assert call(ok(hits=None)) == -1
    assert call(ok(nxt=None)) == -1
    assert call(ok(n=0xFFFFFFFF)) == -2
    assert call(ok(w=None)) == -3
    assert call(ok(wsz=ws - 1)) == -3


def test_stack_distance_noalloc_rejects_bad_arguments(L):
    m = L.pc_stack_distance_noalloc_max_n()
    assert 1_000_000 < m < 2 ** 32
    assert L.pc_stack_distance_ws(m) <= 128 << 20 < L.pc_stack_distance_ws(m + 1)
    assert L.pc_stack_distance_noalloc(FAKE, FAKE, m + 1, FAKE, None) == -2
    assert L.pc_stack_distance_noalloc(FAKE, FAKE, 0xFFFFFFFF, FAKE, None) == -2
    assert L.pc_stack_distance_noalloc(None, FAKE, 10, FAKE, None) == -1
    assert L.pc_stack_distance_noalloc(FAKE, FAKE, 10, None, None) == -1


def test_workspace_status_rejects_null(L):
    code = ctypes.c_int32(0)
    assert L.pc_workspace_status(None, 256, None, ctypes.byref(code)) == -1
    assert L.pc_workspace_status(FAKE, 16, None, ctypes.byref(code)) == -3


def test_profiling_table(L):
    n = L.pc_prof_kernel_count()
    names = [L.pc_prof_kernel_name(i).decode() for i in range(n)]
    assert "hash_blocks" in names and "sd_dominance_pass" in names and "mrc_hist" in names
    assert all(names) and len(set(names)) == n
    assert names[-1] == "mrc_map" and "belady" in names and "chain_stair" in names and "runs_merge" in names
    assert "runs_fill" in names
    assert pc.prof_read() is not None
