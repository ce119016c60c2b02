"""pc_stack_distance_noalloc (no allocation, the library's fixed scratch)
against pc_stack_distance (caller workspace) through the C ABI, on two calls
in a row, the second with a smaller input, and against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import pcgen
from paper_2609_28870_amd import pc

pytestmark = pytest.mark.gpu


def _links(tr):
    keys, _ = oracle.hash_trace(tr)
    prev, nxt = oracle.prev_next(keys)
    return prev, nxt, oracle.stack_distance_bit(prev)


def _check(prev, nxt, want):
    p, q = pc.to_dev_u32(prev), pc.to_dev_u32(nxt)
    got = torch.full((prev.size,), -7, dtype=torch.int32, device="cuda")
    pc.stack_distance_noalloc(p, q, got)
    ref, ws = pc.stack_distance(p, q)
    torch.cuda.synchronize()
    assert pc.workspace_status(ws) == 0
    assert torch.equal(got, ref)
    assert np.array_equal(pc.as_u32(got), want)


def test_two_calls_in_a_row_second_smaller():
    assert torch.cuda.is_available()
    big = pcgen.make_trace("agent", n_sessions=400)          # a few million accesses
    small = pcgen.make_trace("tiny")
    pb, nb, db = _links(big)
    ps, ns, ds = _links(small)
    assert ps.size < pb.size <= pc.stack_distance_noalloc_max_n()
    _check(pb, nb, db)
    _check(ps, ns, ds)
    # a ragged cut of the small one, and the largest size the scratch takes
    # rejected above it before anything is enqueued
    _check(ps[:12345].copy(), np.where(ns[:12345] >= 12345, 0xFFFFFFFF, ns[:12345]).astype(np.uint32),
           ds[:12345])


def test_sizes_beyond_the_scratch_are_rejected():
    m = pc.stack_distance_noalloc_max_n()
    x = torch.empty(1, dtype=torch.int32, device="cuda")
    L = pc.lib()
    assert L.pc_stack_distance_noalloc(x.data_ptr(), x.data_ptr(), m + 1, x.data_ptr(), None) == -2
    assert L.pc_stack_distance_noalloc(None, None, 0, None, None) == 0
