"""rocprofv3 CSV output -> the short markdown summaries under profiles/.

Reads one kernel trace (``--kernel-trace --stats --output-format csv``) and
two counter runs (``--pmc FETCH_SIZE`` and ``--pmc WRITE_SIZE``), each of a
bench.py command that also runs a plain 4 GiB device copy
(``--copy-calibration``): the copy's counter values give the factors that turn
FETCH_SIZE and WRITE_SIZE (KiB per dispatch) into bytes.  Writes a table of
per-kernel launches, times and HBM bytes, and a machine-readable block that
bench.py reads (per working launch, tied to a hash of the library sources).

    python -m paper_2609_28870_amd.profile_summary --trace KT.csv --fetch F.csv --write W.csv \\
        --runs R --title T --out profiles/NAME.md --cmd "..." [--cmd "..."]

Launches gated off on the device (or past a device-side count) return at
once and are left out of the averages: a launch is "working" when its
counters are at least 1% of the kernel's largest in the counter runs (one
pipeline run each), and the kernel trace's working launches are its longest
ones, as many per pipeline run as the counter runs found.  A kernel without
counters counts launches of at least 5% of its longest duration.
"""
import argparse
import collections
import csv
import hashlib
import json
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
COPY_GRID = 131072            # the calibration copy's grid (4 GiB of int32)
COPY_KIB = 4 * 1024 * 1024    # KiB it reads and writes

# library kernel -> the kernel id the bench and the library's timers use
IDS = {"pc::hash_fused_kernel": "hash_blocks",
       "pc::sort_hist_kernel": "sort_digit_hist", "pc::sort_scan_kernel": "sort_digit_scan",
       "pc::sort_pass_kernel": "sort_onesweep_pass", "pc::link_partition_kernel": "link_partition",
       "pc::perm_partition_kernel": "perm_partition", "pc::perm_local_kernel": "perm_local",
       "pc::perm_cursor_kernel": "fill_u32", "pc::fill_u32_kernel": "fill_u32",
       "pc::fill_u32_gated_kernel": "fill_u32",
       "pc::sd_cold_count_kernel": "sd_cold_count", "pc::sd_scan_kernel": "sd_scan",
       "pc::sd_scan_reduce_kernel": "sd_scan", "pc::sd_scan_apply_kernel": "sd_scan",
       "pc::sd_tile_count_kernel": "sd_tile_map", "pc::sd_tile_bucket_kernel": "sd_tile_map",
       "pc::sd_count_kernel<true>": "sd_count", "pc::sd_count_kernel<false>": "sd_count",
       "pc::sd_seg_reduce_kernel": "sd_seg_scan", "pc::sd_seg_carry_kernel": "sd_seg_scan",
       "pc::sd_seg_scan_kernel": "sd_seg_scan",
       "pc::sd_dominance_kernel<true>": "sd_dominance_pass", "pc::sd_dominance_kernel<false>": "sd_dominance_pass",
       "pc::sd_local_kernel": "sd_local_finish", "pc::mrc_hist_kernel": "mrc_hist", "pc::mrc_cost_kernel": "mrc_cost",
       "pc::mrc_map_kernel": "mrc_map",
       "pc::req_order_kernel": "request_order", "pc::req_dist_kernel": "request_distance",
       "pc::sess_dist_kernel": "session_distance", "pc::sess_profile_kernel": "session_profile",
       "pc::prof_pack_kernel": "reuse_profile_pack", "pc::prof_walk_kernel": "reuse_profile_walk",
       "pc::sess_page_kernel": "session_requests", "pc::sess_keys_kernel": "session_requests",
       "pc::sess_status_kernel": "session_requests", "pc::sess_footprint_kernel": "session_requests",
       "pc::chain_layout_kernel": "chain_anchor", "pc::chain_open_kernel": "chain_anchor",
       "pc::chain_anchor_kernel": "chain_anchor", "pc::chain_stair_kernel": "chain_stair",
       "pc::chain_count_kernel": "chain_scan", "pc::chain_scan_tiles_kernel": "chain_scan",
       "pc::chain_scan_top_kernel": "chain_scan", "pc::chain_scan_apply_kernel": "chain_scan",
       "pc::chain_decide_kernel": "chain_scan", "pc::chain_compact_kernel": "chain_compact",
       "pc::chain_merge_kernel": "chain_merge", "pc::chain_verdict_kernel": "chain_merge",
       "pc::chain_status_kernel": "fill_u32", "pc::runs_count_kernel": "runs_count",
       "pc::runs_scan_tiles_kernel": "runs_scan", "pc::runs_scan_top_kernel": "runs_scan",
       "pc::runs_scan_apply_kernel": "runs_scan", "pc::runs_decide_kernel": "runs_scan",
       "pc::runs_compact_kernel": "runs_compact", "pc::runs_init_kernel": "runs_merge",
       "pc::runs_merge_kernel": "runs_merge", "pc::runs_dist_kernel": "runs_merge",
       "pc::runs_fill_kernel": "runs_fill", "pc::runs_status_kernel": "fill_u32",
       "pc::belady_kernel": "belady"}


def kernel_name(s):
    return s.split("(")[0].replace("void ", "").strip()


def source_sha256():
    """Hash of the library sources and header (the one bench.py checks)."""
    h = hashlib.sha256()
    src = os.path.join(ROOT, "paper_2609_28870_amd", "csrc")
    for f in sorted(os.listdir(src)):
        with open(os.path.join(src, f), "rb") as fh:
            h.update(fh.read())
    with open(os.path.join(ROOT, "include", "pc.h"), "rb") as fh:
        h.update(fh.read())
    return h.hexdigest()


def durations(path):
    dur = collections.defaultdict(list)
    with open(path) as f:
        for r in csv.DictReader(f):
            dur[kernel_name(r["Kernel_Name"])].append(
                (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e6)
    return dur


def counters(path):
    """Counter values per kernel, the calibration copy's value and its time."""
    d = collections.defaultdict(list)
    cal = copy_ms = None
    with open(path) as f:
        for r in csv.DictReader(f):
            name = kernel_name(r["Kernel_Name"])
            v = float(r["Counter_Value"])
            if "copyBuffer" in name and int(r["Grid_Size"]) == COPY_GRID:
                cal = v
                copy_ms = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e6
            d[name].append(v)
    if cal is None:
        raise SystemExit("%s: no calibration copy (run bench.py with --copy-calibration)" % path)
    return d, cal, copy_ms


def working(vals, frac):
    m = max(vals)
    return [v for v in vals if v >= frac * m] if m > 0 else vals


def summarize(trace, fetch, write, runs, title, cmds):
    dur = durations(trace)
    F, fcal, c1 = counters(fetch)
    W, wcal, c2 = counters(write)
    ff, wf = COPY_KIB / fcal, COPY_KIB / wcal
    copy_ms = min(c1, c2)
    rows, machine = [], {}
    for name, ds in sorted(dur.items(), key=lambda kv: -sum(kv[1])):
        if name.startswith("__amd"):
            continue
        rd = wr = None
        if name in F and name in W:
            fw, ww = working(F[name], 0.01), working(W[name], 0.01)
            rd = sum(fw) / len(fw) * ff * 1024
            wr = sum(ww) / len(ww) * wf * 1024
            n_work = max(len(fw), len(ww))
            wd = sorted(ds, reverse=True)[:n_work * runs]
        else:
            wd = working(ds, 0.05)
        avg = sum(wd) / len(wd)
        rate = (rd + wr) / (avg / 1e3) / 1e9 if rd is not None and avg > 0 else None
        rows.append((name, len(ds) / runs, len(wd) / runs, sum(ds) / runs, avg, rd, wr, rate))
        if rd is not None:
            machine[name] = {"id": IDS.get(name, IDS.get(name.split("<")[0], name)), "avg_ms": round(avg, 4),
                             "launches_per_run": round(len(wd) / runs, 2),
                             "read_bytes": int(rd), "write_bytes": int(wr)}
    L = ["# %s" % title, "",
         "Commands (from the repository root on the MI355X host; the profiler runs from /tmp with TMPDIR=/tmp), "
         "then `python -m paper_2609_28870_amd.profile_summary` over their CSV output:", ""]
    L += ["    " + c for c in cmds]
    L += ["",
          "Counter calibration: a plain 4 GiB device-to-device copy (`--copy-calibration`) reads "
          "FETCH_SIZE = %.0f KiB and WRITE_SIZE = %.0f KiB for 4194304 KiB moved each way, so FETCH_SIZE is "
          "scaled by %.3f and WRITE_SIZE by %.3f below.  That copy moves 8 GiB in %.2f ms "
          "(%.0f GB/s, read + write), the practical streaming rate on this device.  FETCH_SIZE counts L2 "
          "misses, some of which the 256 MB Infinity Cache serves, so a kernel that re-reads data (the "
          "hash kernel: every turn re-sends its session's context) can show more than the HBM rate." % (
              fcal, wcal, ff, wf, copy_ms, 2 * 4 * 2 ** 30 / (copy_ms / 1e3) / 1e9), "",
          "Working launches: launches gated off on the device (the generic prev/next behind the chained one, "
          "the dominance count behind the runs path, the sort passes over the high key bits) return at once; "
          "averages are over launches that did work: counters at least 1% of the kernel's largest in the "
          "counter runs, and in the kernel trace the kernel's longest launches, as many per pipeline run as "
          "the counter runs found (kernels without counters: duration at least 5% of the longest).", "",
          "| kernel | launches / run | working / run | ms / run | avg working ms | HBM read GB | HBM write GB | "
          "measured GB/s |",
          "|---|---|---|---|---|---|---|---|"]
    for name, cl, cw, tot, avg, rd, wr, rate in rows:
        L.append("| %s | %.3g | %.3g | %.3f | %.3f | %s | %s | %s |" % (
            name, cl, cw, tot, avg, "%.2f" % (rd / 1e9) if rd is not None else "-",
            "%.2f" % (wr / 1e9) if wr is not None else "-", "%.0f" % rate if rate else "-"))
    L += ["", "Machine-readable (per working launch; `source_sha256` covers the library sources and header "
          "the counters were taken with):", "", "```json",
          json.dumps({"source_sha256": source_sha256(), "fetch_scale": round(ff, 4), "write_scale": round(wf, 4),
                      "kernels": machine}, indent=1), "```"]
    return "\n".join(L) + "\n"


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--trace", required=True, help="kernel_trace.csv of the kernel-trace run")
    ap.add_argument("--fetch", required=True, help="counter_collection.csv of the FETCH_SIZE run")
    ap.add_argument("--write", required=True, help="counter_collection.csv of the WRITE_SIZE run")
    ap.add_argument("--runs", type=int, required=True, help="pipeline runs in the kernel-trace command")
    ap.add_argument("--title", required=True)
    ap.add_argument("--out", required=True)
    ap.add_argument("--cmd", action="append", default=[], help="a command that made the input (repeat)")
    a = ap.parse_args()
    text = summarize(a.trace, a.fetch, a.write, a.runs, a.title, a.cmd)
    with open(a.out, "w") as f:
        f.write(text)
    print(text)


if __name__ == "__main__":
    main()
