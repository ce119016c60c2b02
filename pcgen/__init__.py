"""Seeded synthetic multi-turn request traces for the prefix-cache hot path.

This module only *draws inputs*: session/turn tables, token streams and the
capacity lists the curves are evaluated at.  It holds none of the method's
arithmetic (no block hashing, no reuse indexing, no stack distances, no
binning), so both the CPU oracle and the GPU path can consume its output
without sharing any of the computation under test.

Workload shapes follow the paper's setting: 16-token KV blocks and a
151,936-entry tokenizer vocabulary (Sec. 3.1 "Traces"), append-only
multi-turn sessions that re-send the full prior context every turn
(Sec. 2.3 "Sessions"), requests over the context cap skipped (Sec. 3.1),
steady per-session pacing with session concurrency as the knob
(Appendix B), and the HBM / pool capacity points of Table "Cache sizes we
evaluate".  The paper's production traces are not available; these seeded
synthetic traces stand in for them.

Generator readings (the distributions themselves leave these open):

* single-turn status is Bernoulli(p); multi-turn turn counts are
  ``1 + Geometric(p)`` (tiny), ``1 + Zipf(s)`` truncated by rejection to
  ``<= cap`` turns (chat), ``min(floor(Pareto_I(x_m=1, alpha)), cap)``
  (agent);
* lengths are ``max(1, rint(exp(Normal(mu, sigma))))`` tokens;
* a turn whose context would exceed the cap ends the session (a session
  whose *first* request is over the cap has no requests);
* a shared system prompt (chat only) is placed before the first prompt;
* gaps between turns: Exponential(mean) (chat / tiny), Gamma(k, mean/k)
  (agent); session starts are a Poisson process with rate
  ``concurrency / mean(session duration)``;
* timestamps are integer microseconds; requests are ordered by
  ``(ts, session, turn)``;
* each session owns one token stream (its final context); request ``r``
  is the prefix ``stream[0:ctx_len[r]]`` and is described by
  ``(tok_start[r], tok_len[r])`` into one flat int32 token buffer whose
  session streams start on 16-byte boundaries.
"""
from __future__ import annotations

import dataclasses
import math
from concurrent.futures import ThreadPoolExecutor
from typing import Optional

import numpy as np

VOCAB = 151936          # Qwen3 tokenizer vocabulary (Sec. 3.1 "Traces")
SYS_PROMPT_LEN = 2048   # shared system-prompt prefix length (tokens)
N_SYS_PROMPTS = 32
TOKEN_CHUNK = 1 << 24   # tokens per independent generator stream
ALIGN_TOKENS = 4        # session streams start on 16-byte boundaries
GIB_BLOCKS = {"24GiB": 16384, "48GiB": 32768, "96GiB": 65536, "1TiB": 699051}


@dataclasses.dataclass(frozen=True)
class SessionShape:
    """Distributions of one session family."""
    single_turn_p: float
    turns: tuple            # ("geom", p) | ("zipf", s, cap) | ("pareto", alpha, cap)
    first_len: tuple        # (mu, sigma) of log first-prompt length
    append_len: tuple       # (mu, sigma) of log per-turn append length
    ctx_cap: int            # tokens
    gap: tuple              # ("exp", mean_s) | ("gamma", k, mean_s)
    sys_prompt_p: float = 0.0


TINY = SessionShape(0.30, ("geom", 0.2), (7.0, 1.0), (5.0, 1.0), 32768,
                    ("exp", 30.0))
CHAT = SessionShape(0.40, ("zipf", 1.5, 200), (7.5, 1.2), (6.0, 1.0), 262144,
                    ("exp", 30.0), sys_prompt_p=0.05)
AGENT = SessionShape(0.0, ("pareto", 1.1, 2000), (7.0, 1.5), (7.0, 1.5), 131072,
                     ("gamma", 4.0, 10.0))


@dataclasses.dataclass(frozen=True)
class TraceConfig:
    name: str
    mix: tuple                      # ((weight, SessionShape), ...)
    n_sessions: Optional[int]       # fixed session count, or None
    target_tokens: Optional[int]    # stop at first prefix with sum(final ctx) >= this
    concurrency: float
    block_size: int = 16
    caps: str = "wide"              # capacity list recipe
    seed: int = 1


def _log_caps(lo_exp: float, hi_exp: float, n: int) -> list:
    return [int(round(10.0 ** (lo_exp + (hi_exp - lo_exp) * k / (n - 1)))) for k in range(n)]


def capacities(recipe: str, block_size: int = 16) -> np.ndarray:
    """Capacity edges in blocks, non-decreasing, as uint64.

    * ``wide``: 65 log-spaced points over 1e2..1e8 blocks plus the four
      Table "Cache sizes" points (24/48/96 GiB, 1 TiB);
    * ``chat``: 65 log-spaced points over 1e3..1e7 blocks plus Table points;
    * ``tokens64``: 64 log-spaced points over 1e2..1e8 *tokens*, converted to
      blocks with floor division by the block size.
    """
    if recipe == "wide":
        c = _log_caps(2, 8, 65) + list(GIB_BLOCKS.values())
    elif recipe == "chat":
        c = _log_caps(3, 7, 65) + list(GIB_BLOCKS.values())
    elif recipe == "tokens64":
        c = [t // block_size for t in _log_caps(2, 8, 64)]
    else:
        raise ValueError(recipe)
    return np.array(sorted(set(c)) if recipe != "tokens64" else sorted(c), dtype=np.uint64)


CONFIGS = {
    # 64 sessions, ~4.5e4 block accesses: the seconds-on-CPU case
    "tiny": TraceConfig("tiny", ((1.0, TINY),), 64, None, 12.0, caps="wide"),
    # 20k chat sessions with shared system prompts
    "chat": TraceConfig("chat", ((1.0, CHAT),), 20000, None, 256.0, caps="chat"),
    # 5k agent sessions with extreme footprint skew
    "agent": TraceConfig("agent", ((1.0, AGENT),), 5000, None, 16.0, caps="wide"),
    # full-scale mixed trace: 70% chat / 30% agent up to 2e9 context tokens
    "full": TraceConfig("full", ((0.7, CHAT), (0.3, AGENT)), None, 2_000_000_000, 256.0,
                        caps="wide"),
}


def _lognormal_len(rng_normal: np.ndarray, mu: float, sigma: float) -> np.ndarray:
    return np.maximum(1, np.rint(np.exp(mu + sigma * rng_normal))).astype(np.int64)


def _turn_counts(rng: np.random.Generator, shape: SessionShape, n: int) -> np.ndarray:
    kind = shape.turns[0]
    if kind == "geom":
        t = 1 + rng.geometric(shape.turns[1], size=n).astype(np.int64)
    elif kind == "zipf":
        s, cap = shape.turns[1], shape.turns[2]
        z = rng.zipf(s, size=n).astype(np.int64)
        bad = np.nonzero(z > cap - 1)[0]
        while bad.size:
            z[bad] = rng.zipf(s, size=bad.size)
            bad = bad[z[bad] > cap - 1]
        t = 1 + z
    elif kind == "pareto":
        alpha, cap = shape.turns[1], shape.turns[2]
        t = np.minimum(np.floor(1.0 + rng.pareto(alpha, size=n)), cap).astype(np.int64)
    else:
        raise ValueError(kind)
    single = rng.random(n) < shape.single_turn_p
    return np.where(single, 1, t)


def _gaps(rng: np.random.Generator, shape: SessionShape, n: int) -> np.ndarray:
    if shape.gap[0] == "exp":
        return rng.exponential(shape.gap[1], size=n)
    k, mean = shape.gap[1], shape.gap[2]
    return rng.gamma(k, mean / k, size=n)


def _draw_batch(rng: np.random.Generator, mix: tuple, n: int) -> dict:
    """Draw n sessions; every family is drawn for every session (fixed draw
    order, independent of the mix outcome) and the family is then selected."""
    weights = np.array([w for w, _ in mix], dtype=np.float64)
    u = rng.random(n)
    fam = np.searchsorted(np.cumsum(weights) / weights.sum(), u, side="right")
    fam = np.minimum(fam, len(mix) - 1)
    turns = np.zeros(n, np.int64)
    first = np.zeros(n, np.int64)
    sysid = np.full(n, -1, np.int64)
    per_fam = []
    for f, (_, shape) in enumerate(mix):
        t = _turn_counts(rng, shape, n)
        fl = _lognormal_len(rng.standard_normal(n), *shape.first_len)
        has_sys = rng.random(n) < shape.sys_prompt_p
        sid = rng.integers(0, N_SYS_PROMPTS, size=n)
        sel = fam == f
        turns[sel] = t[sel]
        first[sel] = fl[sel]
        sysid[sel & has_sys] = sid[sel & has_sys]
        per_fam.append(shape)
    m = int((turns - 1).sum())
    seg = np.repeat(np.arange(n), turns - 1)
    appends = np.zeros(m, np.int64)
    gaps = np.zeros(m, np.float64)
    zn = rng.standard_normal(m)
    for f, shape in enumerate(per_fam):
        g = _gaps(rng, shape, m)
        sel = fam[seg] == f
        appends[sel] = _lognormal_len(zn[sel], *shape.append_len)
        gaps[sel] = g[sel]
    caps = np.array([s.ctx_cap for s in per_fam], dtype=np.int64)[fam]
    return dict(fam=fam, turns=turns, first=first, sysid=sysid, appends=appends,
                gaps=gaps, caps=caps)


@dataclasses.dataclass
class Trace:
    """A request stream: R requests over S sessions, one flat token buffer.

    Request r (time order) re-sends ``tokens[tok_start[r] : tok_start[r] +
    tok_len[r]]``.  ``blk_off`` is the exclusive prefix of ``tok_len // B``
    (the layout of per-block outputs, request-major)."""
    config: TraceConfig
    tokens: np.ndarray        # int32 [T]
    tok_start: np.ndarray     # uint64 [R]
    tok_len: np.ndarray       # uint32 [R]
    session: np.ndarray       # int64 [R]
    turn: np.ndarray          # int64 [R]
    ts_us: np.ndarray         # int64 [R]
    sess_len: np.ndarray      # int64 [S] final context tokens
    sess_fam: np.ndarray      # int64 [S]
    block_size: int

    @property
    def n_requests(self) -> int:
        return int(self.tok_len.size)

    def blk_off(self, block_size: Optional[int] = None) -> np.ndarray:
        b = block_size or self.block_size
        nb = (self.tok_len.astype(np.uint64) // np.uint64(b))
        off = np.zeros(nb.size + 1, dtype=np.uint64)
        np.cumsum(nb, out=off[1:])
        return off

    def n_blocks(self, block_size: Optional[int] = None) -> int:
        return int(self.blk_off(block_size)[-1])

    def caps(self, block_size: Optional[int] = None) -> np.ndarray:
        return capacities(self.config.caps, block_size or self.block_size)

    def processed_tokens(self) -> int:
        return int(self.tok_len.astype(np.uint64).sum())


def _fill_tokens(buf: np.ndarray, seed: int, threads: int = 8) -> None:
    """Uniform tokens in [0, VOCAB); chunk i of TOKEN_CHUNK positions uses its
    own PCG64 stream seeded by (seed, 2, i), so the content does not depend on
    the thread count."""
    n = buf.size
    nchunks = (n + TOKEN_CHUNK - 1) // TOKEN_CHUNK

    def work(i):
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 2, i])))
        lo, hi = i * TOKEN_CHUNK, min(n, (i + 1) * TOKEN_CHUNK)
        buf[lo:hi] = g.integers(0, VOCAB, size=hi - lo, dtype=np.int32)

    if nchunks <= 1 or threads <= 1:
        for i in range(nchunks):
            work(i)
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(work, range(nchunks)))


def _sessions(b: dict) -> dict:
    """Per-turn contexts for one batch; cut each session at its first over-cap
    turn.  Returns flattened kept turns (session-major) and per-session data."""
    turns, first, sysid = b["turns"], b["first"], b["sysid"]
    S = turns.size
    sys_len = np.where(sysid >= 0, SYS_PROMPT_LEN, 0)
    tstart = np.zeros(S + 1, np.int64)
    np.cumsum(turns, out=tstart[1:])
    nt = int(tstart[-1])
    tsess = np.repeat(np.arange(S), turns)
    tidx = np.arange(nt) - tstart[tsess]
    add = np.zeros(nt, np.int64)
    gap = np.zeros(nt, np.float64)
    add[tstart[:-1]] = sys_len + first
    later = tidx > 0
    add[later] = b["appends"]          # session-major, turns 1..T-1
    gap[later] = b["gaps"]
    ctx = _seg_cumsum(add, tstart)
    bad = _seg_cumsum((ctx > b["caps"][tsess]).astype(np.int64), tstart)
    keep = bad == 0
    toff = _seg_cumsum(np.where(keep, gap, 0.0), tstart)
    kept = np.bincount(tsess[keep], minlength=S)
    sess_len = np.zeros(S, np.int64)
    last = np.nonzero(keep & (tidx == kept[tsess] - 1))[0]
    sess_len[tsess[last]] = ctx[last]
    dur = np.zeros(S, np.float64)
    dur[tsess[last]] = toff[last]
    return dict(tsess=tsess[keep], tidx=tidx[keep], ctx=ctx[keep], toff=toff[keep],
                sess_len=sess_len, dur=dur, sysid=sysid, fam=b["fam"])


def _seg_cumsum(x: np.ndarray, start: np.ndarray) -> np.ndarray:
    """Inclusive cumulative sum restarting at each segment start."""
    c = np.cumsum(x)
    base = np.zeros(start.size - 1, dtype=c.dtype)
    nz = start[1:-1]
    base[1:] = c[nz - 1]
    seg = np.repeat(np.arange(start.size - 1), np.diff(start))
    return c - base[seg]


def make_trace(config, *, seed: Optional[int] = None, n_sessions: Optional[int] = None,
               target_tokens: Optional[int] = None, block_size: Optional[int] = None,
               threads: int = 8) -> Trace:
    """Build a trace from a named config (or TraceConfig).

    ``n_sessions`` / ``target_tokens`` override the config's size (used to
    make reduced-size variants with the same distributions)."""
    cfg = CONFIGS[config] if isinstance(config, str) else config
    seed = cfg.seed if seed is None else seed
    if n_sessions is None and target_tokens is None:
        n_sessions, target_tokens = cfg.n_sessions, cfg.target_tokens
    bsz = block_size or cfg.block_size
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 1])))

    parts = []
    got = 0
    while True:
        n = n_sessions if n_sessions is not None else 65536
        p = _sessions(_draw_batch(rng, cfg.mix, n))
        parts.append(p)
        got += int(p["sess_len"].sum())
        if n_sessions is not None or got >= target_tokens:
            break
    soff = np.cumsum([0] + [p["sess_len"].size for p in parts])
    tsess = np.concatenate([p["tsess"] + o for p, o in zip(parts, soff)])
    tidx = np.concatenate([p["tidx"] for p in parts])
    ctx = np.concatenate([p["ctx"] for p in parts])
    toff = np.concatenate([p["toff"] for p in parts])
    sess_len = np.concatenate([p["sess_len"] for p in parts])
    dur = np.concatenate([p["dur"] for p in parts])
    sysid = np.concatenate([p["sysid"] for p in parts])
    fam = np.concatenate([p["fam"] for p in parts])

    cut = sess_len.size
    if n_sessions is None:
        cut = min(cut, int(np.searchsorted(np.cumsum(sess_len), target_tokens, side="left")) + 1)
    sel = tsess < cut
    tsess, tidx, ctx, toff = tsess[sel], tidx[sel], ctx[sel], toff[sel]
    sess_len, dur, sysid, fam = sess_len[:cut], dur[:cut], sysid[:cut], fam[:cut]

    # Poisson session starts at the target concurrency
    arng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 3])))
    mean_dur = float(dur.mean()) if cut else 0.0
    rate = cfg.concurrency / mean_dur if mean_dur > 0 else 1.0
    starts = np.cumsum(arng.exponential(1.0 / rate, size=cut))
    ts = np.rint((starts[tsess] + toff) * 1e6).astype(np.int64)
    order = np.lexsort((tidx, tsess, ts))
    rs, rt, ts, rctx = tsess[order], tidx[order], ts[order], ctx[order]

    # token buffer: one stream per session, 16-byte aligned
    alen = (sess_len + ALIGN_TOKENS - 1) // ALIGN_TOKENS * ALIGN_TOKENS
    sbase = np.zeros(cut + 1, np.int64)
    np.cumsum(alen, out=sbase[1:])
    tokens = np.empty(int(sbase[-1]), dtype=np.int32)
    _fill_tokens(tokens, seed, threads)
    srng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 4])))
    sys_tokens = srng.integers(0, VOCAB, size=(N_SYS_PROMPTS, SYS_PROMPT_LEN), dtype=np.int32)
    for s in np.nonzero(sysid >= 0)[0]:
        n = min(SYS_PROMPT_LEN, int(sess_len[s]))
        tokens[sbase[s]:sbase[s] + n] = sys_tokens[sysid[s], :n]

    return Trace(config=cfg, tokens=tokens,
                 tok_start=sbase[rs].astype(np.uint64),
                 tok_len=rctx.astype(np.uint32),
                 session=rs, turn=rt, ts_us=ts,
                 sess_len=sess_len, sess_fam=fam, block_size=bsz)


def subtrace(tr: Trace, r0: int, r1: int) -> Trace:
    """Requests r0..r1-1 of a trace (same token buffer)."""
    return dataclasses.replace(tr, tok_start=tr.tok_start[r0:r1], tok_len=tr.tok_len[r0:r1],
                               session=tr.session[r0:r1], turn=tr.turn[r0:r1],
                               ts_us=tr.ts_us[r0:r1])


def random_keys(n: int, distinct: int, seed: int = 0, hot: float = 0.0) -> np.ndarray:
    """A raw key stream (uint64) for edge-case tests: ``distinct`` keys drawn
    uniformly, optionally with a fraction ``hot`` of accesses to one key."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 5])))
    vocab = g.integers(0, 2 ** 63, size=max(distinct, 1), dtype=np.int64).astype(np.uint64)
    vocab |= np.uint64(1) << np.uint64(63)
    idx = g.integers(0, max(distinct, 1), size=n)
    if hot > 0:
        idx[g.random(n) < hot] = 0
    return vocab[idx]
