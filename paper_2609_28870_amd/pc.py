"""Thin ctypes binding of libpc (include/pc.h).

Argument marshalling only: every step of the hot path runs in the HIP
kernels of ``libpc.so``.  PyTorch provides device memory and the current HIP
stream.  Unsigned arrays travel in signed torch tensors of the same width
(uint64 bit patterns in int64, uint32 in int32); ``as_u64`` / ``as_u32``
reinterpret them on the host.

There is no fallback: if ``libpc.so`` is missing or no GPU is visible, calls
raise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "_lib", "libpc.so")
NONE = 0xFFFFFFFF
DEEPEST_FIRST = 1   # PC_HASH_DEEPEST_FIRST
PREV_ONLY = 2       # PC_PREV_ONLY

_lib = None

_vp = ctypes.c_void_p
_u64 = ctypes.c_uint64
_u32 = ctypes.c_uint32
_sz = ctypes.c_size_t
_st = ctypes.c_int


class PcError(RuntimeError):
    pass


def lib():
    """Load libpc.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise PcError("libpc.so not built: run paper_2609_28870_amd/build.py (or __graft_entry__.build())")
    L = ctypes.CDLL(LIB_PATH)
    L.pc_status_string.restype = ctypes.c_char_p
    L.pc_status_string.argtypes = [_st]
    L.pc_version.restype = ctypes.c_int
    L.pc_hash_blocks_ws.restype = _sz
    L.pc_hash_blocks_ws.argtypes = [_u32]
    L.pc_hash_blocks.restype = _st
    L.pc_hash_blocks.argtypes = [_vp, _u64, _vp, _vp, _u32, _u32, _vp, _u64, _vp, _u64, _vp, _vp,
                                 _vp, _u32, _vp, _sz, _vp]
    L.pc_prev_next_use_ws.restype = _sz
    L.pc_prev_next_use_ws.argtypes = [_u64]
    L.pc_prev_next_use.restype = _st
    L.pc_prev_next_use.argtypes = [_vp, _u64, _vp, _vp, _vp, _vp, _sz, _vp]
    L.pc_prev_next_chained_ws.restype = _sz
    L.pc_prev_next_chained_ws.argtypes = [_u64, _u32]
    L.pc_prev_next_chained.restype = _st
    L.pc_prev_next_chained.argtypes = [_vp, _u64, _vp, _u32, _u32, _vp, _vp, _vp, _vp, _sz, _vp]
    L.pc_stack_distance_runs_ws.restype = _sz
    L.pc_stack_distance_runs_ws.argtypes = [_u64]
    L.pc_stack_distance_runs.restype = _st
    L.pc_stack_distance_runs.argtypes = [_vp, _vp, _u64, _vp, _vp, _sz, _vp]
    L.pc_stack_distance_noalloc_max_n.restype = _u64
    L.pc_stack_distance_noalloc_max_n.argtypes = []
    L.pc_stack_distance_noalloc.restype = _st
    L.pc_stack_distance_noalloc.argtypes = [_vp, _vp, _u64, _vp, _vp]
    L.pc_stack_distance_ws.restype = _sz
    L.pc_stack_distance_ws.argtypes = [_u64]
    L.pc_stack_distance.restype = _st
    L.pc_stack_distance.argtypes = [_vp, _vp, _u64, _vp, _vp, _sz, _vp]
    L.pc_request_order_ws.restype = _sz
    L.pc_request_order_ws.argtypes = []
    L.pc_request_order.restype = _st
    L.pc_request_order.argtypes = [_vp, _vp, _vp, _u32, _u64, _vp, _vp, _vp, _sz, _vp]
    L.pc_stack_distance_req_ws.restype = _sz
    L.pc_stack_distance_req_ws.argtypes = []
    L.pc_stack_distance_req.restype = _st
    L.pc_stack_distance_req.argtypes = [_vp, _vp, _vp, _u32, _u64, _vp, _vp, _sz, _vp]
    L.pc_stack_distance_session_ws.restype = _sz
    L.pc_stack_distance_session_ws.argtypes = [_u64, _u32]
    L.pc_stack_distance_session.restype = _st
    L.pc_stack_distance_session.argtypes = [_vp, _vp, _vp, _u32, _u64, _vp, _vp, _sz, _vp]
    L.pc_reuse_profile_ws.restype = _sz
    L.pc_reuse_profile_ws.argtypes = [_u64]
    L.pc_reuse_profile.restype = _st
    L.pc_reuse_profile.argtypes = [_vp, _vp, _vp, _vp, _u32, _u64, _vp, _u32, _u32, _vp, _vp, _vp, _vp, _vp,
                                   _sz, _vp]
    L.pc_session_profile_ws.restype = _sz
    L.pc_session_profile_ws.argtypes = [_u32]
    L.pc_session_profile.restype = _st
    L.pc_session_profile.argtypes = [_vp, _vp, _vp, _u32, _u64, _vp, _u32, _u32, _u32, _vp, _vp, _vp, _vp, _vp,
                                     _sz, _vp]
    L.pc_mrc_weighted_ws.restype = _sz
    L.pc_mrc_weighted_ws.argtypes = [_u64, _u32]
    L.pc_mrc_weighted.restype = _st
    L.pc_mrc_weighted.argtypes = [_vp, _vp, _vp, _u64, _vp, _u32, _u64, _u64, _vp, _vp, _vp, _vp,
                                  _vp, _vp, _sz, _vp]
    L.pc_mrc_weighted_layout_ws.restype = _sz
    L.pc_mrc_weighted_layout_ws.argtypes = [_u64, _u32]
    L.pc_mrc_weighted_layout.restype = _st
    L.pc_mrc_weighted_layout.argtypes = [_vp, _vp, _u32, _u32, _vp, _u64, _vp, _u32, _u64, _u64, _vp, _vp, _vp,
                                         _vp, _vp, _vp, _sz, _vp]
    L.pc_belady_ws.restype = _sz
    L.pc_belady_ws.argtypes = [_u64, _u32]
    L.pc_belady.restype = _st
    L.pc_belady.argtypes = [_vp, _vp, _u64, _vp, _u32, _vp, _vp, _vp, _vp, _sz, _vp]
    L.pc_workspace_status.restype = _st
    L.pc_workspace_status.argtypes = [_vp, _sz, _vp, ctypes.POINTER(ctypes.c_int32)]
    L.pc_prof_enable.restype = None
    L.pc_prof_enable.argtypes = [ctypes.c_int]
    L.pc_prof_kernel_count.restype = ctypes.c_int
    L.pc_prof_kernel_name.restype = ctypes.c_char_p
    L.pc_prof_kernel_name.argtypes = [ctypes.c_int]
    L.pc_prof_read.restype = _st
    L.pc_prof_read.argtypes = [ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(ctypes.c_double),
                               ctypes.c_int]
    _lib = L
    return L


def check(status: int) -> None:
    if status != 0:
        raise PcError("libpc: %s (%d)" % (lib().pc_status_string(status).decode(), status))


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise PcError("expected a GPU tensor")
    if not t.is_contiguous():
        raise PcError("expected a contiguous tensor")
    return t.data_ptr()


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _dev():
    if not torch.cuda.is_available():
        raise PcError("no GPU visible: libpc needs an MI355X (gfx950)")
    return torch.device("cuda", torch.cuda.current_device())


def workspace(nbytes: int) -> torch.Tensor:
    """Device scratch for one call (torch's allocator aligns to >= 256 B)."""
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=_dev())


def workspace_status(ws: torch.Tensor) -> int:
    """Device-side status code of a workspace (synchronises the stream)."""
    code = ctypes.c_int32(0)
    check(lib().pc_workspace_status(_ptr(ws), ws.numel(), _stream(), ctypes.byref(code)))
    return int(code.value)


def as_u64(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy().view(np.uint64)


def as_u32(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy().view(np.uint32)


def to_dev_u64(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint64).view(np.int64)).to(_dev())


def to_dev_u32(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint32).view(np.int32)).to(_dev())


# ------------------------------------------------------------------ stages

def hash_blocks(tokens: torch.Tensor, tok_start: torch.Tensor, tok_len: torch.Tensor,
                blk_off: torch.Tensor, n_blocks: int, block_size: int = 16,
                parent: Optional[torch.Tensor] = None, root: int = 0, want_depth: bool = True,
                keys: Optional[torch.Tensor] = None, depth: Optional[torch.Tensor] = None,
                ws: Optional[torch.Tensor] = None, key_hist: Optional[torch.Tensor] = None,
                deepest_first: bool = False):
    """pc_hash_blocks: keys (int64 bits of uint64) and depth (int32 bits);
    with ``key_hist`` (int32[1024]) also the byte histograms of the keys'
    low four bytes, which prev_next_use can take instead of counting them.
    ``deepest_first`` writes each request's blocks in descending depth order
    (the recency order of request-level residency)."""
    L = lib()
    dev = _dev()
    n_seqs = tok_len.numel()
    if keys is None:
        keys = torch.empty(n_blocks, dtype=torch.int64, device=dev)
    if want_depth and depth is None:
        depth = torch.empty(n_blocks, dtype=torch.int32, device=dev)
    if ws is None:
        ws = workspace(L.pc_hash_blocks_ws(n_seqs))
    check(L.pc_hash_blocks(_ptr(tokens), tokens.numel(), _ptr(tok_start), _ptr(tok_len), n_seqs,
                           block_size, _ptr(parent), root & (2 ** 64 - 1), _ptr(blk_off), n_blocks,
                           _ptr(keys), _ptr(depth) if want_depth else None, _ptr(key_hist),
                           1 if deepest_first else 0, _ptr(ws), ws.numel(), _stream()))
    return keys, (depth if want_depth else None), ws


def prev_next_use(keys: torch.Tensor, prev: Optional[torch.Tensor] = None,
                  nxt: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                  key_hist: Optional[torch.Tensor] = None):
    L = lib()
    n = keys.numel()
    dev = _dev()
    if prev is None:
        prev = torch.empty(n, dtype=torch.int32, device=dev)
    if nxt is None:
        nxt = torch.empty(n, dtype=torch.int32, device=dev)
    if ws is None:
        ws = workspace(L.pc_prev_next_use_ws(n))
    check(L.pc_prev_next_use(_ptr(keys), n, _ptr(prev), _ptr(nxt), _ptr(key_hist), _ptr(ws), ws.numel(),
                             _stream()))
    return prev, nxt, ws


def high_key_passes_ran(ws: torch.Tensor) -> bool:
    """Whether the last pc_prev_next_use call on this workspace also sorted by
    the high 32 key bits (workspace word 1, decided on the device).
    Synchronises the current stream."""
    torch.cuda.current_stream().synchronize()
    return bool(int(ws[4:8].view(torch.int32).item()))


def prev_next_chained(keys: torch.Tensor, blk_off: torch.Tensor, prev: Optional[torch.Tensor] = None,
                      nxt: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                      key_hist: Optional[torch.Tensor] = None, deepest_first: bool = False,
                      prev_only: bool = False):
    """pc_prev_next_chained: the same prev / next as prev_next_use for keys
    laid out per request as hash_blocks writes them; the path is chosen on
    the device (no synchronisation).  With ``prev_only`` (PC_PREV_ONLY) next
    is scratch and unspecified afterwards."""
    L = lib()
    n = keys.numel()
    n_seqs = blk_off.numel() - 1
    dev = _dev()
    if prev is None:
        prev = torch.empty(n, dtype=torch.int32, device=dev)
    if nxt is None:
        nxt = torch.empty(n, dtype=torch.int32, device=dev)
    if ws is None:
        ws = workspace(L.pc_prev_next_chained_ws(n, n_seqs))
    check(L.pc_prev_next_chained(_ptr(keys), n, _ptr(blk_off), n_seqs,
                                 (PREV_ONLY if prev_only else 0) | (DEEPEST_FIRST if deepest_first else 0),
                                 _ptr(prev), _ptr(nxt), _ptr(key_hist), _ptr(ws), ws.numel(), _stream()))
    return prev, nxt, ws


def chained_info(ws: torch.Tensor) -> dict:
    """What the last pc_prev_next_chained call on this workspace did: whether
    the generic prev/next ran over all keys (and why), and how many accesses
    went through the generic prev/next of the unresolved ones.  Synchronises."""
    torch.cuda.current_stream().synchronize()
    w = ws[:32].view(torch.int32).cpu().tolist()
    return {"generic": bool(w[1]), "unresolved": w[2] & 0xFFFFFFFF, "reason": w[3],
            "high_anchor": bool(w[6]), "high_unresolved": bool(w[7])}


def stack_distance(prev: torch.Tensor, nxt: torch.Tensor, dist: Optional[torch.Tensor] = None,
                   ws: Optional[torch.Tensor] = None):
    L = lib()
    n = prev.numel()
    if dist is None:
        dist = torch.empty(n, dtype=torch.int32, device=_dev())
    if ws is None:
        ws = workspace(L.pc_stack_distance_ws(n))
    check(L.pc_stack_distance(_ptr(prev), _ptr(nxt), n, _ptr(dist), _ptr(ws), ws.numel(), _stream()))
    return dist, ws


def stack_distance_noalloc(prev: torch.Tensor, nxt: torch.Tensor, dist: torch.Tensor):
    """pc_stack_distance_noalloc: the same distances as stack_distance into a
    caller-provided ``dist``, with the library's own fixed device scratch
    (nothing is allocated; calls on one GPU must not overlap)."""
    check(lib().pc_stack_distance_noalloc(_ptr(prev), _ptr(nxt), prev.numel(), _ptr(dist), _stream()))
    return dist


def stack_distance_noalloc_max_n() -> int:
    return int(lib().pc_stack_distance_noalloc_max_n())


def stack_distance_runs(prev: torch.Tensor, nxt: torch.Tensor, dist: Optional[torch.Tensor] = None,
                        ws: Optional[torch.Tensor] = None):
    """pc_stack_distance_runs: the same distances as stack_distance, counted
    over the runs of the prev stream, or by the dominance count when there
    are too many runs (chosen on the device; no synchronisation)."""
    L = lib()
    n = prev.numel()
    if dist is None:
        dist = torch.empty(n, dtype=torch.int32, device=_dev())
    if ws is None:
        ws = workspace(L.pc_stack_distance_runs_ws(n))
    check(L.pc_stack_distance_runs(_ptr(prev), _ptr(nxt), n, _ptr(dist), _ptr(ws), ws.numel(), _stream()))
    return dist, ws


def runs_info(ws: torch.Tensor) -> dict:
    """What the last pc_stack_distance_runs call on this workspace did.
    Synchronises."""
    torch.cuda.current_stream().synchronize()
    w = ws[:16].view(torch.int32).cpu().tolist()
    return {"generic": bool(w[1]), "runs": w[2] & 0xFFFFFFFF, "cold": w[3] & 0xFFFFFFFF}


def request_order(keys: torch.Tensor, blk_off: torch.Tensor, depth: Optional[torch.Tensor] = None,
                  keys_out: Optional[torch.Tensor] = None, depth_out: Optional[torch.Tensor] = None,
                  ws: Optional[torch.Tensor] = None):
    """pc_request_order: every request's accesses reversed (deepest block
    first), the recency order of request-level residency."""
    L = lib()
    n = keys.numel()
    n_seqs = blk_off.numel() - 1
    dev = _dev()
    if keys_out is None:
        keys_out = torch.empty(n, dtype=torch.int64, device=dev)
    if depth is not None and depth_out is None:
        depth_out = torch.empty(n, dtype=torch.int32, device=dev)
    if ws is None:
        ws = workspace(L.pc_request_order_ws())
    check(L.pc_request_order(_ptr(keys), _ptr(depth), _ptr(blk_off), n_seqs, n, _ptr(keys_out),
                             _ptr(depth_out) if depth is not None else None, _ptr(ws), ws.numel(),
                             _stream()))
    return keys_out, depth_out, ws


def stack_distance_req(prev: torch.Tensor, dist: torch.Tensor, blk_off: torch.Tensor,
                       dist_req: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None):
    """pc_stack_distance_req: request-level stack distances from prev and
    dist of the request-ordered accesses."""
    L = lib()
    n = prev.numel()
    n_seqs = blk_off.numel() - 1
    if dist_req is None:
        dist_req = torch.empty(n, dtype=torch.int32, device=_dev())
    if ws is None:
        ws = workspace(L.pc_stack_distance_req_ws())
    check(L.pc_stack_distance_req(_ptr(prev), _ptr(dist), _ptr(blk_off), n_seqs, n,
                                  _ptr(dist_req), _ptr(ws), ws.numel(), _stream()))
    return dist_req, ws


def stack_distance_session(prev: torch.Tensor, blk_off: torch.Tensor, session: torch.Tensor,
                           dist_sess: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None):
    """pc_stack_distance_session: session-level distances from prev (request
    order), the request table and the session of every request."""
    L = lib()
    n = prev.numel()
    n_seqs = blk_off.numel() - 1
    if session.numel() != n_seqs:
        raise PcError("one session id per request expected")
    if dist_sess is None:
        dist_sess = torch.empty(n, dtype=torch.int32, device=_dev())
    if ws is None:
        ws = workspace(L.pc_stack_distance_session_ws(n, n_seqs))
    check(L.pc_stack_distance_session(_ptr(prev), _ptr(blk_off), _ptr(session), n_seqs, n, _ptr(dist_sess),
                                      _ptr(ws), ws.numel(), _stream()))
    return dist_sess, ws


FREQ_CLASSES = 32


def reuse_profile(prev: torch.Tensor, nxt: torch.Tensor, blk_off: torch.Tensor, ts_us: torch.Tensor,
                  edges: torch.Tensor, freq_max: int, out: Optional[dict] = None, ws: Optional[torch.Tensor] = None):
    """pc_reuse_profile: reuse-interval, lifetime, frequency and
    lifetime-by-frequency-class histograms (int64 tensors of uint64)."""
    L = lib()
    n = prev.numel()
    n_seqs = blk_off.numel() - 1
    k = edges.numel()
    dev = _dev()
    if out is None:
        out = {"interval": torch.empty(k + 1, dtype=torch.int64, device=dev),
               "lifetime": torch.empty(k + 1, dtype=torch.int64, device=dev),
               "freq": torch.empty(freq_max + 1, dtype=torch.int64, device=dev),
               "life_by_class": torch.empty(FREQ_CLASSES * (k + 1), dtype=torch.int64, device=dev)}
    if ws is None:
        ws = workspace(L.pc_reuse_profile_ws(n))
    check(L.pc_reuse_profile(_ptr(prev), _ptr(nxt), _ptr(blk_off), _ptr(ts_us), n_seqs, n, _ptr(edges), k,
                             freq_max, _ptr(out["interval"]), _ptr(out["lifetime"]), _ptr(out["freq"]),
                             _ptr(out["life_by_class"]), _ptr(ws), ws.numel(), _stream()))
    return out, ws


def session_profile(blk_off: torch.Tensor, session: torch.Tensor, ts_us: torch.Tensor, n: int,
                    edges: torch.Tensor, fp_max: int, rq_max: int, out: Optional[dict] = None,
                    ws: Optional[torch.Tensor] = None):
    """pc_session_profile: footprint, request-count, duration and gap
    histograms over sessions (int64 tensors of uint64)."""
    L = lib()
    n_seqs = blk_off.numel() - 1
    k = edges.numel()
    dev = _dev()
    if out is None:
        out = {"footprint": torch.empty(fp_max + 1, dtype=torch.int64, device=dev),
               "requests": torch.empty(rq_max + 1, dtype=torch.int64, device=dev),
               "duration": torch.empty(k + 1, dtype=torch.int64, device=dev),
               "gap": torch.empty(k + 1, dtype=torch.int64, device=dev)}
    if ws is None:
        ws = workspace(L.pc_session_profile_ws(n_seqs))
    check(L.pc_session_profile(_ptr(blk_off), _ptr(session), _ptr(ts_us), n_seqs, n, _ptr(edges), k, fp_max,
                               rq_max, _ptr(out["footprint"]), _ptr(out["requests"]), _ptr(out["duration"]),
                               _ptr(out["gap"]), _ptr(ws), ws.numel(), _stream()))
    return out, ws


def hists_to_host(out: dict) -> dict:
    """Device histograms -> lists of python ints."""
    return {name: [int(x) for x in as_u64(t).tolist()] for name, t in out.items()}


def mrc_weighted(dist: torch.Tensor, caps: torch.Tensor, depth: Optional[torch.Tensor] = None,
                 nxt: Optional[torch.Tensor] = None, alpha: int = 1, beta: int = 0,
                 out: Optional[dict] = None, ws: Optional[torch.Tensor] = None):
    """pc_mrc_weighted: per-bin count, depthsum, cost (lo/hi) and next-use
    histogram as int64 tensors of n_caps+1 entries (uint64 bit patterns);
    the next-use histogram is all zero when ``nxt`` is None."""
    L = lib()
    n = dist.numel()
    k = caps.numel()
    dev = _dev()
    if out is None:
        out = {name: torch.empty(k + 1, dtype=torch.int64, device=dev)
               for name in ("count", "depthsum", "cost_lo", "cost_hi", "nextuse")}
    if ws is None:
        ws = workspace(L.pc_mrc_weighted_ws(n, k))
    check(L.pc_mrc_weighted(_ptr(dist), _ptr(depth), _ptr(nxt), n, _ptr(caps), k,
                            alpha & (2 ** 64 - 1), beta & (2 ** 64 - 1), _ptr(out["count"]),
                            _ptr(out["depthsum"]), _ptr(out["cost_lo"]), _ptr(out["cost_hi"]),
                            _ptr(out["nextuse"]), _ptr(ws), ws.numel(),
                            _stream()))
    return out, ws


def mrc_weighted_layout(dist: torch.Tensor, caps: torch.Tensor, blk_off: torch.Tensor,
                        nxt: Optional[torch.Tensor] = None, alpha: int = 1, beta: int = 0,
                        out: Optional[dict] = None, ws: Optional[torch.Tensor] = None, deepest_first: bool = False):
    """pc_mrc_weighted_layout: as mrc_weighted with depth[t] = t - blk_off[r]
    for the request r holding t (the ascending layout of hash_blocks), or
    blk_off[r + 1] - 1 - t with ``deepest_first``."""
    L = lib()
    n = dist.numel()
    k = caps.numel()
    dev = _dev()
    if out is None:
        out = {name: torch.empty(k + 1, dtype=torch.int64, device=dev)
               for name in ("count", "depthsum", "cost_lo", "cost_hi", "nextuse")}
    if ws is None:
        ws = workspace(L.pc_mrc_weighted_layout_ws(n, k))
    check(L.pc_mrc_weighted_layout(_ptr(dist), _ptr(blk_off), blk_off.numel() - 1,
                                   DEEPEST_FIRST if deepest_first else 0, _ptr(nxt), n, _ptr(caps), k,
                                   alpha & (2 ** 64 - 1), beta & (2 ** 64 - 1), _ptr(out["count"]),
                                   _ptr(out["depthsum"]), _ptr(out["cost_lo"]), _ptr(out["cost_hi"]),
                                   _ptr(out["nextuse"]), _ptr(ws), ws.numel(), _stream()))
    return out, ws


def belady(nxt: torch.Tensor, caps: torch.Tensor, depth: Optional[torch.Tensor] = None, flags: bool = False,
           out: Optional[dict] = None, ws: Optional[torch.Tensor] = None):
    """pc_belady: hits and depth sums of Belady's MIN at every capacity
    (int64 tensors of uint64); with ``flags`` also the per-access hit flags
    (uint8 [n_caps, n])."""
    L = lib()
    n = nxt.numel()
    k = caps.numel()
    dev = _dev()
    if out is None:
        out = {"hits": torch.empty(k, dtype=torch.int64, device=dev),
               "depthsum": torch.empty(k, dtype=torch.int64, device=dev)}
    if flags and "flags" not in out:
        out["flags"] = torch.empty((k, n), dtype=torch.uint8, device=dev)
    if ws is None:
        ws = workspace(L.pc_belady_ws(n, k))
    check(L.pc_belady(_ptr(nxt), _ptr(depth), n, _ptr(caps), k, _ptr(out["hits"]), _ptr(out["depthsum"]),
                      _ptr(out.get("flags")) if flags else None, _ptr(ws), ws.numel(), _stream()))
    return out, ws


def bins_to_host(out: dict) -> dict:
    """Device bins -> python ints (cost as exact 128-bit integers)."""
    c = as_u64(out["count"]).tolist()
    d = as_u64(out["depthsum"]).tolist()
    lo = as_u64(out["cost_lo"]).tolist()
    hi = as_u64(out["cost_hi"]).tolist()
    nu = as_u64(out["nextuse"]).tolist()
    return {"count": [int(x) for x in c], "depthsum": [int(x) for x in d],
            "cost": [int(h) << 64 | int(l) for l, h in zip(lo, hi)], "nextuse": [int(x) for x in nu]}


def curves(count, cost):
    """Hit ratio and compute-savings ratio at each capacity edge from exact
    integer bins: hits(c_k) = sum count[0..k], saved(c_k) = sum cost[0..k];
    each ratio is one float64 division of exactly rounded integers."""
    n = sum(count)
    total = sum(cost)
    hr, csr = [], []
    h = s = 0
    for k in range(len(count) - 1):
        h += count[k]
        s += cost[k]
        hr.append(float(h) / float(n) if n else 0.0)
        csr.append(float(s) / float(total) if total else 0.0)
    return hr, csr


# --------------------------------------------------------------- profiling

def prof_enable(on: bool = True) -> None:
    lib().pc_prof_enable(1 if on else 0)


def prof_read() -> dict:
    """{kernel: (launches, total_ms)} since the last read (caller syncs)."""
    L = lib()
    n = L.pc_prof_kernel_count()
    la = (ctypes.c_uint64 * n)()
    ms = (ctypes.c_double * n)()
    check(L.pc_prof_read(la, ms, n))
    return {L.pc_prof_kernel_name(i).decode(): (int(la[i]), float(ms[i])) for i in range(n)}


# ---------------------------------------------------------------- pipeline

class Pipeline:
    """All four stages over one trace with buffers and workspaces allocated
    once; ``run()`` enqueues hash -> prev/next -> stack distance -> bins.

    ``residency="access"`` bins the per-access LRU stack distance.
    ``residency="session"`` (whole sessions evicted at once, Sec. 5.3) bins
    the session-level distance instead; it needs ``session``, the session of
    every request, and takes no next-use histogram.
    ``residency="request"`` (every block of a request resident at once,
    Sec. 3.1) hashes each request's blocks straight into recency order
    (deepest block first; ``keys_r`` and ``depth_r`` alias ``keys`` and
    ``depth``), runs prev/next and the stack distance on that order, turns
    the result into the request-level distance and bins that, with depth in
    the same order; the next-use histogram is not taken in that mode.  Its
    bins are valid at capacities of at least the largest request.
    ``with_belady`` (per-access mode) also runs Belady's MIN at every
    capacity on the step's next-use index (``belady_out``).

    The bins take each block's depth from the request layout
    (``mrc_weighted_layout``) and the hash writes no depth (``depth`` and
    ``depth_r`` are None); ``depth_array=True``, and Belady's MIN, keep the
    depth array."""

    def __init__(self, tokens, tok_start, tok_len, blk_off, n_blocks: int, caps,
                 block_size: int = 16, alpha: int = 1, beta: int = 0, with_nextuse: bool = True,
                 residency: str = "access", session: Optional[torch.Tensor] = None, chained: bool = True,
                 with_belady: bool = False, depth_array: bool = False):
        if residency not in ("access", "request", "session"):
            raise PcError("residency must be 'access', 'request' or 'session'")
        if residency == "session" and session is None:
            raise PcError("session-level residency needs the session of every request")
        L = lib()
        dev = _dev()
        self.tokens, self.tok_start, self.tok_len, self.blk_off = tokens, tok_start, tok_len, blk_off
        self.n = int(n_blocks)
        self.B = block_size
        self.caps = caps
        self.alpha, self.beta = alpha, beta
        self.residency = residency
        self.request = residency == "request"
        self.session = session
        self.with_nextuse = with_nextuse and residency == "access"
        self.with_belady = with_belady and residency == "access"
        self.layout_depth = not (depth_array or self.with_belady)
        n = self.n
        self.keys = torch.empty(n, dtype=torch.int64, device=dev)
        self.key_hist = torch.empty(4 * 256, dtype=torch.int32, device=dev)
        self.depth = None if self.layout_depth else torch.empty(n, dtype=torch.int32, device=dev)
        self.prev = torch.empty(n, dtype=torch.int32, device=dev)
        self.next = torch.empty(n, dtype=torch.int32, device=dev)
        self.dist = torch.empty(n, dtype=torch.int32, device=dev)
        k = caps.numel()
        self.bins = {name: torch.empty(k + 1, dtype=torch.int64, device=dev)
                     for name in ("count", "depthsum", "cost_lo", "cost_hi", "nextuse")}
        self.ws_hash = workspace(L.pc_hash_blocks_ws(tok_len.numel()))
        self.chained = chained
        self.ws_pn = workspace(L.pc_prev_next_chained_ws(n, tok_len.numel()) if chained
                               else L.pc_prev_next_use_ws(n))
        if residency == "session":
            self.ws_sd = workspace(L.pc_stack_distance_session_ws(n, tok_len.numel()))
        else:
            self.ws_sd = workspace(L.pc_stack_distance_runs_ws(n) if chained else L.pc_stack_distance_ws(n))
        if self.request:
            self.keys_r, self.depth_r = self.keys, self.depth   # hashed in recency order
            self.dist_req = torch.empty(n, dtype=torch.int32, device=dev)
            self.ws_req = workspace(L.pc_stack_distance_req_ws())
        self.ws_mrc = workspace(L.pc_mrc_weighted_layout_ws(n, k) if self.layout_depth
                                else L.pc_mrc_weighted_ws(n, k))
        if self.with_belady:
            self.belady_out = {"hits": torch.empty(k, dtype=torch.int64, device=dev),
                               "depthsum": torch.empty(k, dtype=torch.int64, device=dev)}
            self.ws_bel = workspace(L.pc_belady_ws(n, k))

    def run(self):
        hash_blocks(self.tokens, self.tok_start, self.tok_len, self.blk_off, self.n, self.B,
                    want_depth=not self.layout_depth, keys=self.keys, depth=self.depth, ws=self.ws_hash,
                    key_hist=self.key_hist, deepest_first=self.request)
        if self.residency == "session":
            self._prev_next(self.keys)
            stack_distance_session(self.prev, self.blk_off, self.session, dist_sess=self.dist, ws=self.ws_sd)
            self._bins(None)
            return
        if not self.request:
            self._prev_next(self.keys)
            self._stack_distance()
            self._bins(self.next if self.with_nextuse else None)
            if self.with_belady:
                belady(self.next, self.caps, self.depth, out=self.belady_out, ws=self.ws_bel)
            return
        self._prev_next(self.keys_r)
        self._stack_distance()
        stack_distance_req(self.prev, self.dist, self.blk_off, dist_req=self.dist_req, ws=self.ws_req)
        if self.layout_depth:
            mrc_weighted_layout(self.dist_req, self.caps, self.blk_off, None, self.alpha, self.beta, out=self.bins,
                                ws=self.ws_mrc, deepest_first=True)
        else:
            mrc_weighted(self.dist_req, self.caps, self.depth_r, None, self.alpha, self.beta,
                         out=self.bins, ws=self.ws_mrc)

    def _bins(self, nxt):
        if self.layout_depth:
            mrc_weighted_layout(self.dist, self.caps, self.blk_off, nxt, self.alpha, self.beta, out=self.bins,
                                ws=self.ws_mrc)
        else:
            mrc_weighted(self.dist, self.caps, self.depth, nxt, self.alpha, self.beta, out=self.bins, ws=self.ws_mrc)

    def _prev_next(self, keys):
        if self.chained:
            # session-level eviction reads no next use
            prev_next_chained(keys, self.blk_off, self.prev, self.next, ws=self.ws_pn, key_hist=self.key_hist,
                              deepest_first=self.request, prev_only=self.residency == "session")
        else:
            prev_next_use(keys, self.prev, self.next, ws=self.ws_pn, key_hist=self.key_hist)

    def _stack_distance(self):
        if self.chained:
            stack_distance_runs(self.prev, self.next, self.dist, ws=self.ws_sd)
        else:
            stack_distance(self.prev, self.next, self.dist, ws=self.ws_sd)

    def high_key_passes_ran(self) -> bool:
        """Whether the last generic prev/next call also sorted by the high 32
        key bits (decided on the device; see pc_prev_next_use).  Synchronises."""
        return high_key_passes_ran(self.ws_pn)

    def chained_info(self) -> dict:
        """What the last chained prev/next did (see chained_info)."""
        return chained_info(self.ws_pn)

    def status(self) -> dict:
        stages = [("hash", self.ws_hash), ("prev_next", self.ws_pn), ("stack_distance", self.ws_sd),
                  ("mrc", self.ws_mrc)]
        if self.request:
            stages.append(("stack_distance_req", self.ws_req))
        if self.with_belady:
            stages.append(("belady", self.ws_bel))
        return {name: workspace_status(ws) for name, ws in stages}


class Profiler:
    """Workload characterisation over one trace (Sec. 4): hash -> prev/next
    -> reuse profile (intervals, lifetimes, frequencies) and session profile
    (footprints, requests, durations, gaps), buffers allocated once."""

    def __init__(self, tokens, tok_start, tok_len, blk_off, n_blocks: int, session, ts_us, edges,
                 block_size: int = 16, freq_max: int = 2048, fp_max: int = 1 << 16, rq_max: int = 2048,
                 chained: bool = True):
        L = lib()
        dev = _dev()
        self.tokens, self.tok_start, self.tok_len, self.blk_off = tokens, tok_start, tok_len, blk_off
        self.session, self.ts_us, self.edges = session, ts_us, edges
        self.n = int(n_blocks)
        self.B = block_size
        self.freq_max, self.fp_max, self.rq_max = freq_max, fp_max, rq_max
        n = self.n
        self.keys = torch.empty(n, dtype=torch.int64, device=dev)
        self.key_hist = torch.empty(4 * 256, dtype=torch.int32, device=dev)
        self.prev = torch.empty(n, dtype=torch.int32, device=dev)
        self.next = torch.empty(n, dtype=torch.int32, device=dev)
        self.ws_hash = workspace(L.pc_hash_blocks_ws(tok_len.numel()))
        self.chained = chained
        self.ws_pn = workspace(L.pc_prev_next_chained_ws(n, tok_len.numel()) if chained
                               else L.pc_prev_next_use_ws(n))
        self.ws_rp = workspace(L.pc_reuse_profile_ws(n))
        self.ws_sp = workspace(L.pc_session_profile_ws(tok_len.numel()))
        k = edges.numel()
        self.reuse = {"interval": torch.empty(k + 1, dtype=torch.int64, device=dev),
                      "lifetime": torch.empty(k + 1, dtype=torch.int64, device=dev),
                      "freq": torch.empty(freq_max + 1, dtype=torch.int64, device=dev),
                      "life_by_class": torch.empty(FREQ_CLASSES * (k + 1), dtype=torch.int64, device=dev)}
        self.sessions = {"footprint": torch.empty(fp_max + 1, dtype=torch.int64, device=dev),
                         "requests": torch.empty(rq_max + 1, dtype=torch.int64, device=dev),
                         "duration": torch.empty(k + 1, dtype=torch.int64, device=dev),
                         "gap": torch.empty(k + 1, dtype=torch.int64, device=dev)}

    def run(self):
        hash_blocks(self.tokens, self.tok_start, self.tok_len, self.blk_off, self.n, self.B,
                    want_depth=False, keys=self.keys, ws=self.ws_hash, key_hist=self.key_hist)
        if self.chained:
            prev_next_chained(self.keys, self.blk_off, self.prev, self.next, ws=self.ws_pn, key_hist=self.key_hist)
        else:
            prev_next_use(self.keys, self.prev, self.next, ws=self.ws_pn, key_hist=self.key_hist)
        reuse_profile(self.prev, self.next, self.blk_off, self.ts_us, self.edges, self.freq_max,
                      out=self.reuse, ws=self.ws_rp)
        session_profile(self.blk_off, self.session, self.ts_us, self.n, self.edges, self.fp_max, self.rq_max,
                        out=self.sessions, ws=self.ws_sp)

    def status(self) -> dict:
        return {name: workspace_status(ws) for name, ws in
                (("hash", self.ws_hash), ("prev_next", self.ws_pn), ("reuse_profile", self.ws_rp),
                 ("session_profile", self.ws_sp))}


def upload_trace(trace, block_size: Optional[int] = None):
    """Copy a pcgen.Trace's arrays to the GPU (input preparation, untimed)."""
    B = block_size or trace.block_size
    off = trace.blk_off(B)
    dev = _dev()
    return dict(tokens=torch.from_numpy(trace.tokens).to(dev),
                tok_start=to_dev_u64(trace.tok_start), tok_len=to_dev_u32(trace.tok_len),
                blk_off=to_dev_u64(off), n_blocks=int(off[-1]), block_size=B,
                session=to_dev_u32(trace.session.astype(np.uint32)),
                ts_us=to_dev_u64(trace.ts_us.astype(np.uint64)))
