"""Throughput of the prefix-cache hot path on one MI355X.

One step = the whole path over the resident trace: chained block hashing ->
prev/next-use indexing -> exact LRU stack distance -> hit-ratio /
compute-savings bins over every capacity.  Inputs (token streams and the
request table) are generated on the host, copied to HBM before timing, and
stay resident; the timed region contains only the four library calls.

Prints one JSON line (rank 0): block accesses per second, per-kernel times
from HIP events recorded by the library on its launch stream, the roofline
of the dominant kernel and the CPU oracle timed on a bounded sample.
"""
import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
AGENT_3E8_SESSIONS = 55000     # agent sessions for a trace of at least 3e8 block accesses (3.19e8)
P_LIN = 3_000_000_000          # FLOPs per token, linear part (agent cost model)

# algorithmic bytes per element for each kernel (inputs it must read and
# outputs it must write, once each)
ALGO_BYTES = {
    # tokens in, key out (the per-access hashing bytes of the measurement
    # plan; the 4-byte depth the kernel also writes is not counted)
    "hash_blocks": lambda B: 4 * B + 8,
    "sort_onesweep_pass": lambda B: 12 + 12,      # (key, t) in and out
    "link_partition": lambda B: 12 + 12,          # sorted (key, t) in, (t, prev, next) out
    "perm_partition": lambda B: 12 + 12,          # (t, prev, next) in and out
    "perm_local": lambda B: 12 + 8,               # (t, prev, next) in, prev + next out
    "sd_dominance_pass": lambda B: 8 + 8,         # (t, acc) in and out
    "sd_local_finish": lambda B: 8 + 4 + 4,       # (t, acc), prev in; dist out
    # dist, depth, next in (the per-access pipeline takes depth from the
    # request layout, so there only dist and next count; see mrc_bytes)
    "mrc_hist": lambda B: 12,
    "request_distance": lambda B: 4 + 4 + 4,      # prev, per-access dist in; dist_req out
    "session_distance": lambda B: 4 + 4,          # prev in; dist_sess out
    "reuse_profile_pack": lambda B: 4 + 8,        # next in; (next, request) out
    "reuse_profile_walk": lambda B: 4 + 8,        # prev (chain starts) and one (next, request) per step in
    # chained prev/next: its own key and the linked request's key at the same
    # depth in, the prev link and its mirrored next link out
    "chain_stair": lambda B: 8 + 8 + 4 + 4,
    # stack distance over runs: prev read once by the count (which keeps
    # three bits per position for the compaction), dist written by the fill
    # from the run list
    "runs_count": lambda B: 4,
    "runs_compact": lambda B: 0.5,
    "runs_fill": lambda B: 4,
}
# generic prev/next kernels: per element of the key streams they sort
GENERIC_PN = ("sort_digit_hist", "sort_digit_scan", "sort_onesweep_pass", "link_partition", "perm_partition",
              "perm_local")


def chain_bytes(name, n, n_slots, m, n_req):
    """Algorithmic bytes per launch of the chained prev/next's own kernels
    (n accesses, n_slots anchor slots, m unresolved accesses, n_req requests)."""
    return {# two launches: the layout check (offsets in), the anchors (key in; slot key + record out)
            "chain_anchor": (n_req * 16 + n_slots * (8 + 8 + 16)) // 2,
            "chain_scan": n_slots * (4 + 4 + 4) // 3,     # three launches over the slot counts
            # slot record, masks, offset in; key in, (key, pos, flag) out
            "chain_compact": n_slots * (16 + 16 + 4) + m * (8 + 8 + 4 + 1),
            "chain_merge": m * (1 + 4 + 4 + 4 + 8),       # (flag, pos, prev, next) in; prev / next out
            }.get(name)


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


# HIP kernel behind each timed kernel id (for the committed counter summary)
HIP_KERNEL = {"sort_onesweep_pass": "pc::sort_pass_kernel", "link_partition": "pc::link_partition_kernel",
              "perm_partition": "pc::perm_partition_kernel", "hash_blocks": "pc::hash_fused_kernel",
              "sd_local_finish": "pc::sd_local_kernel",
              "perm_local": "pc::perm_local_kernel", "mrc_hist": "pc::mrc_hist_kernel",
              "request_distance": "pc::req_dist_kernel",
              "session_distance": "pc::sess_dist_kernel", "reuse_profile_walk": "pc::prof_walk_kernel",
              "reuse_profile_pack": "pc::prof_pack_kernel", "chain_stair": "pc::chain_stair_kernel",
              "chain_compact": "pc::chain_compact_kernel", "chain_anchor": "pc::chain_anchor_kernel",
              "chain_merge": "pc::chain_merge_kernel", "runs_count": "pc::runs_count_kernel",
              "runs_compact": "pc::runs_compact_kernel", "runs_fill": "pc::runs_fill_kernel"}
# committed counter summaries, by (mode, prev/next path, workload, block
# size, session count); a run with none reports no counter traffic
PROFILES = {
    ("access", "chained", "full", 16, None): "all_kernels_full_mixed_2e9.md",
    ("request", "chained", "full", 16, None): "all_kernels_full_mixed_2e9_request.md",
    ("session", "chained", "full", 16, None): "all_kernels_full_mixed_2e9_session.md",
    ("profile", "chained", "full", 16, None): "all_kernels_full_mixed_2e9_profile.md",
    ("access", "generic", "full", 16, None): "all_kernels_full_mixed_2e9_generic.md",
    ("access", "chained", "chat", 16, None): "all_kernels_chat_2e8.md",
    ("access", "chained", "agent", 16, AGENT_3E8_SESSIONS): "all_kernels_agent_3e8.md",
    ("access", "chained", "agent", 16, None): "all_kernels_agent_B16.md",
    ("access", "chained", "agent", 64, None): "all_kernels_agent_B64.md",
    ("access", "chained", "agent", 256, None): "all_kernels_agent_B256.md",
}
PROFILE = os.path.join(ROOT, "profiles", PROFILES[("access", "chained", "full", 16, None)])


def profile_for(mode, prev_next, workload="full", block_size=16, sessions=None):
    """Path of the committed summary for this run's kernels, or None."""
    name = PROFILES.get((mode, prev_next, workload, block_size, sessions))
    return os.path.join(ROOT, "profiles", name) if name else None


def source_sha256():
    """Hash of the library sources and header, as recorded with the counters."""
    import hashlib
    h = hashlib.sha256()
    src = os.path.join(ROOT, "paper_2609_28870_amd", "csrc")
    for f in sorted(os.listdir(src)):
        with open(os.path.join(src, f), "rb") as fh:
            h.update(fh.read())
    with open(os.path.join(ROOT, "include", "pc.h"), "rb") as fh:
        h.update(fh.read())
    return h.hexdigest()


def _profile_blob():
    if PROFILE is None:
        return None
    try:
        text = open(PROFILE).read()
        blob = json.loads(text[text.index("```json") + 7:text.rindex("```")])
    except (OSError, ValueError):
        return None
    return blob if blob.get("source_sha256") == source_sha256() else None


def measured_stage_bytes(stage_of):
    """Measured HBM bytes per pipeline run of each stage (sum over its
    kernels' working launches) from the committed counter summary, or None
    when the library has changed since."""
    blob = _profile_blob()
    if blob is None:
        return None
    out = {}
    for e in blob["kernels"].values():
        st = stage_of(e["id"])
        out[st] = out.get(st, 0.0) + (e["read_bytes"] + e["write_bytes"]) * e["launches_per_run"]
    return out


def measured_traffic(kernel_id):
    """HBM bytes per working launch of a kernel from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary (calibrated on a plain copy), or None when
    the library has changed since those counters were taken."""
    blob = _profile_blob()
    want = HIP_KERNEL.get(kernel_id)
    # a kernel template appears under its instance's name, e.g. "k<2>"
    entry = next((e for name, e in blob["kernels"].items() if name.split("<")[0] == want), None) if blob else None
    if entry is None:
        return None
    return {"read_bytes": entry["read_bytes"], "write_bytes": entry["write_bytes"],
            "profiled_avg_ms": entry["avg_ms"], "source": os.path.relpath(PROFILE, ROOT)}


# time edges of the characterisation histograms (microseconds): 1-2-5 steps
# from 1 us to 1e11 us (~28 hours)
PROFILE_EDGES_US = sorted(m * 10 ** e for e in range(0, 11) for m in (1, 2, 5)) + [10 ** 11]


def _quantile(hist, edges, q):
    """Upper edge of the bin holding the q-quantile of a histogram."""
    total = sum(hist)
    if total == 0:
        return None
    run = 0
    for k, c in enumerate(hist):
        run += c
        if run >= q * total:
            return edges[k] if k < len(edges) else float("inf")
    return float("inf")


def profile_summary(rp, sp):
    """A few headline figures from the characterisation histograms (host
    arithmetic on exact integer bins)."""
    e = PROFILE_EDGES_US
    f = rp["freq"]
    at_least = [sum(f[k:]) for k in range(len(f))]
    fp = sp["footprint"]
    n_sess = sum(fp)
    blocks = sum(v * c for v, c in enumerate(fp))

    def top_share(frac):
        want = math.ceil(frac * n_sess - 1e-9)   # the largest ceil(frac * sessions) sessions
        got_s = got_b = 0
        for v in range(len(fp) - 1, -1, -1):
            take = min(fp[v], want - got_s)
            got_s += take
            got_b += take * v
            if got_s >= want:
                break
        return round(got_b / blocks, 4) if blocks else None

    return {"reuse_interval_us_p50_upper": _quantile(rp["interval"], e, 0.5),
            "reuse_interval_us_p99_upper": _quantile(rp["interval"], e, 0.99),
            "lifetime_us_p50_upper": _quantile(rp["lifetime"], e, 0.5),
            "one_access_blocks": round(f[1] / at_least[1], 4) if at_least[1] else None,
            "p_reuse_after_1": round(at_least[2] / at_least[1], 4) if at_least[1] else None,
            "p_reuse_after_2": round(at_least[3] / at_least[2], 4) if at_least[2] else None,
            "sessions": n_sess,
            "footprint_top10pct_share": top_share(0.1),
            "footprint_top1pct_share": top_share(0.01),
            "session_duration_us_p50_upper": _quantile(sp["duration"], e, 0.5),
            "intra_session_gap_us_p50_upper": _quantile(sp["gap"], e, 0.5)}


def cpu_model():
    """The host CPU's model name (Linux /proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def baseline_threads(n_caps):
    """One capacity simulation per thread, as many threads as capacities but
    no more than the host's cores and a one-GPU share of them (16)."""
    return max(1, min(n_caps, os.cpu_count() or 1, 16))


def cpu_baseline(trace, caps, alpha, beta, budget_accesses, request=False):
    """The oracle (plain C) over the first requests of the same trace: hash,
    prev/next, next-use histogram and one LRU simulation per capacity edge --
    the same outputs as one GPU step.  Requests are hashed by ranges on a
    thread pool and the per-capacity simulations run one per thread.  In
    request mode: hash and the request-level bins (one pinned-request
    simulation per feasible edge, the recency-list walk for the others); in
    Belady mode the per-access outputs plus one MIN simulation per edge."""
    import oracle
    import pcgen
    threads = baseline_threads(len(caps))
    nb = (trace.tok_len // np.uint32(trace.block_size)).astype(np.int64)
    r = int(np.searchsorted(np.cumsum(nb), budget_accesses)) + 1
    r = min(r, trace.n_requests)
    sub = pcgen.subtrace(trace, 0, r)
    t0 = time.perf_counter()
    keys, depth = oracle.hash_trace(sub, threads=threads)
    ids = oracle.key_ids(keys)
    if request == "profile":
        bo = sub.blk_off()
        ts = sub.ts_us.astype(np.uint64)
        oracle.reuse_profile(keys, bo, ts, PROFILE_EDGES_US, 2048)
        oracle.session_profile(bo, sub.session, ts, PROFILE_EDGES_US, 1 << 16, 2048)
        what = "reuse and session profiles"
    elif request == "session":
        oracle.mrc_bins_session(keys, sub.blk_off(), sub.session.astype(np.uint32), caps, depth, alpha, beta, ids,
                                threads=threads)
        what = "prev/next + session-level bins (%d per-capacity session LRU simulations)" % len(caps)
    elif request and request != "belady":
        oracle.mrc_bins_req(keys, sub.blk_off(), caps, depth, alpha, beta, ids, threads=threads)
        what = "request-level bins"
    else:
        _, nxt = oracle.prev_next(keys, ids)
        oracle.nextuse_hist(nxt, caps)
        oracle.mrc_bins(keys, caps, depth, alpha, beta, ids, threads=threads)
        what = "prev/next + %d per-capacity LRU simulations" % len(caps)
        if request == "belady":
            oracle.belady(keys, caps, ids, nxt, threads=threads)
            what += " + %d per-capacity Belady MIN simulations" % len(caps)
    dt = time.perf_counter() - t0
    return {"value": keys.size / dt, "unit": "block-accesses/s", "cores": threads, "kind": "oracle",
            "nproc": os.cpu_count(), "cpu_model": cpu_model(),
            "sample": "first %d requests (%d block accesses) of the same trace; hash + %s; %.1f s on %d threads "
                      "(hashing by request ranges, one capacity simulation per thread)" % (
                          r, keys.size, what, dt, threads)}


GOLDEN_FULL = os.path.join(ROOT, "tests", "golden", "fullsize_full.txt")
# the oracle's full-size references, by (workload, block size, session count)
GOLDEN = {("full", 16, None): GOLDEN_FULL,
          ("chat", 16, None): os.path.join(ROOT, "tests", "golden", "fullsize_chat.txt")}


def read_fullsize_golden(path):
    """The oracle's full-size reference: n, per-capacity (cap, hits,
    depth sum over hits) and the next-use histogram."""
    g = {"caps": []}
    with open(path) as f:
        for line in f:
            w = line.split("#", 1)[0].split()
            if not w:
                continue
            if w[0] == "cap":
                g["caps"].append((int(w[1]), int(w[2]), int(w[3]), int(w[4], 16)))
            elif w[0] == "nextuse":
                g["nextuse"] = [int(x) for x in w[1:]]
            elif w[0] in ("n", "requests", "distinct", "depth_total"):
                g[w[0]] = int(w[1])
            elif w[0].startswith("fp_"):
                g[w[0]] = int(w[1], 16)
    return g


def check_against_golden(bins, caps, n, path):
    """Compare this run's bins with the oracle's full-size reference (hits and
    depth sums at every capacity, next-use histogram); raises on a mismatch."""
    g = read_fullsize_golden(path)
    if g["n"] != n or [c for c, _, _, _ in g["caps"]] != [int(c) for c in caps]:
        raise SystemExit("reference %s is for another trace or capacity list" % path)
    h = d = 0
    for k, (c, hits, dsum, _) in enumerate(g["caps"]):
        h += bins["count"][k]
        d += bins["depthsum"][k]
        if h != hits or d != dsum:
            raise SystemExit("bins differ from the oracle's reference at capacity %d: hits %d vs %d, "
                             "depth sum %d vs %d" % (c, h, hits, d, dsum))
    if sum(bins["count"]) != n or bins["depthsum"] and sum(bins["depthsum"]) != g["depth_total"]:
        raise SystemExit("bin totals differ from the oracle's reference")
    if bins["nextuse"] != g["nextuse"]:
        raise SystemExit("next-use histogram differs from the oracle's reference")
    return {"reference": os.path.relpath(path, ROOT), "capacities": len(g["caps"]), "bins_match": True}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="full", choices=["tiny", "chat", "agent", "full"])
    ap.add_argument("--sessions", type=int, default=None, help="override the session count")
    ap.add_argument("--block-size", type=int, default=16)
    ap.add_argument("--residency", default="access", choices=["access", "request", "session"],
                    help="per-access LRU (default), request-level residency (whole request pinned) "
                         "or session-level eviction (whole sessions evicted)")
    ap.add_argument("--profile", action="store_true",
                    help="time the workload characterisation instead (hash, prev/next, reuse and session "
                         "profiles)")
    ap.add_argument("--cpu-sample", type=int, default=None,
                    help="block accesses in the oracle's timed sample (0 = skip; default 4e8, "
                         "1e6 with --residency request)")
    ap.add_argument("--belady", action="store_true",
                    help="also run Belady's MIN at every capacity in each step (pc_belady on the step's "
                         "next-use index) and report the LRU-Belady gap at the paper's cache sizes; MIN is "
                         "sequential per capacity (about 6 s per step on the agent trace), so traces above "
                         "--belady-max accesses are refused")
    ap.add_argument("--belady-max", type=float, default=1e8,
                    help="largest trace (block accesses) --belady runs on")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 4 GiB device copy (for rocprof counter calibration)")
    ap.add_argument("--prev-next", default="chained", choices=["chained", "generic"],
                    help="prev/next from the chain structure of the keys and the stack distance over runs "
                         "(default), or the generic sort and the dominance count over accesses")
    ap.add_argument("--settle", type=float, default=0.0,
                    help="seconds to wait before touching the device (0 by default: a process started "
                         "right after another one that held most of HBM runs at the same speed)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the hot path here is single-GPU "
              "(multi-GPU sharding is a design note, not built); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    if args.settle > 0:
        log("waiting %.0f s before touching the device" % args.settle)
        time.sleep(args.settle)
    import torch
    import pcgen
    from paper_2609_28870_amd import pc

    B = args.block_size
    t0 = time.perf_counter()
    trace = pcgen.make_trace(args.workload, n_sessions=args.sessions, block_size=B)
    caps_np = trace.caps(B)
    n_blocks = trace.n_blocks(B)
    if args.belady and n_blocks > args.belady_max:
        raise SystemExit("--belady on %d block accesses: Belady's MIN runs one sequential simulation per "
                         "capacity (minutes per step at this size); use --workload agent, or raise "
                         "--belady-max" % n_blocks)
    log("trace %s: %d requests, %d block accesses, %d processed tokens, generated in %.1f s" % (
        args.workload, trace.n_requests, n_blocks, trace.processed_tokens(), time.perf_counter() - t0))

    torch.cuda.set_device(0)
    alpha, beta = 2 * B * P_LIN, 2 * B * B
    up = pc.upload_trace(trace, B)
    caps = pc.to_dev_u64(caps_np)
    request = args.residency == "request"
    session_mode = args.residency == "session"
    global PROFILE
    PROFILE = profile_for("profile" if args.profile else args.residency, args.prev_next, args.workload, B,
                          args.sessions)
    if args.profile:
        prof_edges = pc.to_dev_u64(np.array(PROFILE_EDGES_US, np.uint64))
        pipe = pc.Profiler(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"],
                           up["session"], up["ts_us"], prof_edges, B, chained=args.prev_next == "chained")
    else:
        pipe = pc.Pipeline(up["tokens"], up["tok_start"], up["tok_len"], up["blk_off"], up["n_blocks"],
                           caps, B, alpha, beta, residency=args.residency, session=up["session"],
                           chained=args.prev_next == "chained", with_belady=args.belady)
    torch.cuda.synchronize()
    log("inputs resident in HBM; device memory in use %.1f GB" % (torch.cuda.memory_allocated() / 1e9))

    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log("copy calibration: 4 GiB read + 4 GiB written")

    for i in range(args.warmup):
        pipe.run()
    torch.cuda.synchronize()
    st = pipe.status()
    if any(st.values()):
        raise SystemExit("device status after warm-up: %s" % st)
    log("warm-up done")

    pc.prof_enable(True)
    pc.prof_read()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for i in range(args.steps):
        pipe.run()
        if args.belady:   # seconds per step: say where the run is
            torch.cuda.synchronize()
            log("step %d done" % (i + 1))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t1
    pc.prof_enable(False)
    prof = pc.prof_read()
    st = pipe.status()
    if any(st.values()):
        raise SystemExit("device status after timing: %s" % st)
    log("timed %d steps in %.3f s" % (args.steps, wall))

    ms_step = wall * 1e3 / args.steps
    value = n_blocks / (ms_step / 1e3)
    # the four high-key sort passes of each inner prev/next exit at once
    # unless its first link asked for them; count only passes that moved data
    chain = pc.chained_info(pipe.ws_pn) if pipe.chained else None
    if chain:
        log("chained prev/next:", chain)
        if chain["generic"]:
            raise SystemExit("the chained prev/next fell back to the generic path on this trace: %s" % chain)
        calls = 2
        highs = int(chain["high_anchor"]) + int(chain["high_unresolved"])
        n_slots = n_blocks // 64 + trace.n_requests + 1
        pn_elems = n_slots + chain["unresolved"]
    else:
        calls = 1
        highs = int(pc.high_key_passes_ran(pipe.ws_pn))
        n_slots = pn_elems = n_blocks
    work_launches = {"sort_onesweep_pass": 4 * calls + 4 * highs, "link_partition": calls + highs,
                     "sort_digit_hist": calls + highs}
    # bins: dist in, depth in unless it comes from the request layout, next in
    # when the next-use histogram is taken
    layout_depth = getattr(pipe, "layout_depth", False)
    mrc_bytes = 4 + (0 if layout_depth else 4) + (4 if getattr(pipe, "with_nextuse", False) else 0)
    kernels = {}
    for name, (launches, ms) in prof.items():
        if launches == 0:
            continue
        per_step = ms / args.steps
        wl = work_launches.get(name, launches // args.steps)
        entry = {"launches_per_step": launches // args.steps, "working_launches_per_step": wl,
                 "ms_per_step": round(per_step, 4)}
        cb_bytes = chain_bytes(name, n_blocks, n_slots, chain["unresolved"], trace.n_requests) if chain else None
        if name in ALGO_BYTES or cb_bytes is not None:
            if cb_bytes is not None:
                per_launch = cb_bytes
            elif name in GENERIC_PN:
                # elements sorted per inner call, averaged over the calls
                per_launch = ALGO_BYTES[name](B) * pn_elems // calls
            else:
                per_launch = (mrc_bytes if name == "mrc_hist" else ALGO_BYTES[name](B)) * n_blocks
            entry["algo_bytes_per_launch"] = per_launch
            entry["avg_working_launch_ms"] = round(per_step / wl, 4)
            entry["algo_GBps"] = round(per_launch * wl / per_step / 1e6, 1)
        kernels[name] = entry
    # the roofline is the memory path's: Belady's MIN is a per-capacity
    # sequential simulation (one wave per capacity), reported on its own
    dom = max((k for k in kernels if k != "belady"), key=lambda k: kernels[k]["ms_per_step"])
    d = kernels[dom]
    achieved = d.get("algo_GBps")
    roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4) if achieved else None}
    roof["kernel"] = dom
    mt = measured_traffic(dom)
    roof["traffic"] = mt["read_bytes"] + mt["write_bytes"] if mt else None
    if mt:
        mt["GBps_at_this_run"] = round(roof["traffic"] / (d["avg_working_launch_ms"] / 1e3) / 1e9, 1)
    roof["traffic_detail"] = mt
    stage_of = {"hash_blocks": "hash", "sort_digit_hist": "prev_next",
                "sort_digit_scan": "prev_next", "sort_onesweep_pass": "prev_next",
                "link_partition": "prev_next",
                "perm_partition": "prev_next", "perm_local": "prev_next", "chain_anchor": "prev_next",
                "chain_stair": "prev_next", "chain_scan": "prev_next", "chain_compact": "prev_next",
                "chain_merge": "prev_next", "mrc_hist": "mrc", "mrc_map": "mrc",
                "mrc_cost": "mrc", "request_distance": "request_distance",
                "session_requests": "session_profile" if args.profile else "session_distance",
                "session_distance": "session_distance",
                "reuse_profile_pack": "reuse_profile", "reuse_profile_walk": "reuse_profile",
                "session_profile": "session_profile", "belady": "belady"}
    stage_bytes = {"hash": 4 * B + 8, "prev_next": 16, "stack_distance": 8,
                   "mrc": mrc_bytes, "request_distance": 12,
                   "session_distance": 8, "reuse_profile": 24}

    def stage_name(kid):
        return stage_of.get(kid, "stack_distance" if kid.startswith(("sd_", "runs_")) else "other")

    stages = {}
    for name, e in kernels.items():
        st_name = stage_name(name)
        stages[st_name] = stages.get(st_name, 0.0) + e["ms_per_step"]
    measured = measured_stage_bytes(stage_name)
    stages = {k: {"ms_per_step": round(v, 3),
                  "algo_GBps": round(stage_bytes[k] * n_blocks / v / 1e6, 1) if k in stage_bytes else None,
                  # counter-measured bytes (committed summary) over this run's time
                  "measured_GBps": (round(measured[k] / v / 1e6, 1) if measured and k in measured
                                    and k in stage_bytes else None)}
              for k, v in stages.items()}

    # request-level bins hold only at capacities that fit the largest request
    min_cap = int((trace.tok_len // np.uint32(B)).max()) if request else 0
    summary = None
    if args.profile:
        summary = profile_summary(pc.hists_to_host(pipe.reuse), pc.hists_to_host(pipe.sessions))
    else:
        # the curves themselves (exact integers -> float64 ratios)
        bins = pc.bins_to_host(pipe.bins)
        hr, csr = pc.curves(bins["count"], bins["cost"])
    # the last timed step's bins against the oracle's full-size reference
    oracle_check = None
    golden = GOLDEN.get((args.workload, B, args.sessions))
    if not args.profile and args.residency == "access" and golden and os.path.exists(golden):
        oracle_check = check_against_golden(bins, caps_np, n_blocks, golden)
        log("bins match the oracle's full-size reference at all %d capacities" % oracle_check["capacities"])
    cb = None
    sample = args.cpu_sample if args.cpu_sample is not None else (
        1_000_000 if request else 20_000_000 if args.belady else 400_000_000)
    if sample > 0:
        log("timing the CPU oracle on a %d-access sample" % sample)
        kind = "profile" if args.profile else "session" if session_mode else "belady" if args.belady else request
        cb = cpu_baseline(trace, caps_np, alpha, beta, sample, kind)

    out = {
        "metric": "KV-block accesses/sec for hash+stack-distance+MRC; achieved HBM GB/s",
        "residency": args.residency,
        "value": value,
        "unit": "block-accesses/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "strong",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic",
        "config": {
            "workload": "%s trace (%s), block size %d" % (
                args.workload, "70% chat / 30% agent sessions up to 2e9 context tokens"
                if args.workload == "full" else "%s sessions" % (args.sessions or "default"), B),
            "n_block_accesses": n_blocks,
            "n_requests": trace.n_requests,
            "processed_tokens": trace.processed_tokens(),
            "capacities": int(caps_np.size),
            "cost_model": "2*B*(P_lin + B*depth), P_lin=3e9",
            "residency": ("request-level (whole request resident; bins valid from %d blocks)" % min_cap
                          if request else "session-level (whole sessions evicted)" if session_mode
                          else "per-access LRU"),
            "parallelism": "single GPU",
        },
        "roofline": roof,
        "cpu_baseline": cb,
        "oracle_check": oracle_check,
        "kernels": kernels,
        "stages": stages,
        "high_key_sort_passes": highs,
        "chained_prev_next": chain,
        "stack_distance_runs": (pc.runs_info(pipe.ws_sd) if pipe.chained and not args.profile
                                and not session_mode else None),
    }
    if args.profile:
        out["metric"] = "KV-block accesses/sec for hash+prev/next+workload characterisation; achieved HBM GB/s"
        out["residency"] = None
        out["config"]["residency"] = None
        out["config"]["analysis"] = "reuse intervals, lifetimes, frequencies, session footprints (Sec. 4)"
        out["characterisation"] = summary
    else:
        out["curves_at"] = {str(int(c)): [round(h, 6), round(s, 6)] if int(c) >= min_cap else None
                            for c, h, s in zip(caps_np, hr, csr) if int(c) in pcgen.GIB_BLOCKS.values()}
    if args.belady and not args.profile:
        bh = [int(x) for x in pc.as_u64(pipe.belady_out["hits"])]
        bms = kernels.get("belady", {}).get("ms_per_step")
        out["belady"] = {
            "ms_per_step": bms,
            "capacity_accesses_per_s": (n_blocks * len(bh) / (bms / 1e3)) if bms else None,
            "capacities": len(bh),
            # hit ratios at the paper's cache sizes: [LRU, Belady, Belady - LRU]
            "hit_ratio_at": {str(int(c)): [round(h, 6), round(b / n_blocks, 6), round(b / n_blocks - h, 6)]
                             for c, h, b in zip(caps_np, hr, bh) if int(c) in pcgen.GIB_BLOCKS.values()},
            "lru_never_above": all(sum(bins["count"][:k + 1]) <= b for k, b in enumerate(bh)),
        }
        out["metric"] = "KV-block accesses/sec for hash+stack-distance+MRC+Belady MIN; achieved HBM GB/s"
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
