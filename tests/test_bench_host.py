"""Host logic of bench.py (CPU only): the one-GPU guard, the kernel tables,
the committed counter summaries it reads and the characterisation summary
arithmetic."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2", "--settle", "0"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_every_timed_kernel_has_algorithmic_bytes():
    chain = {k for k in bench.HIP_KERNEL if bench.chain_bytes(k, 1 << 20, 1 << 14, 1 << 17, 1000) is not None}
    assert set(bench.HIP_KERNEL) <= set(bench.ALGO_BYTES) | chain
    for name, f in bench.ALGO_BYTES.items():
        assert f(16) > 0, name
    for name in chain:
        assert bench.chain_bytes(name, 1 << 20, 1 << 14, 1 << 17, 1000) > 0, name


@pytest.mark.parametrize("key", sorted(bench.PROFILES, key=str))
def test_committed_profiles_parse(key):
    path = bench.profile_for(*key)
    text = open(path).read()
    blob = json.loads(text[text.index("```json") + 7:text.rindex("```")])
    assert len(blob["source_sha256"]) == 64
    # the copy calibration: FETCH_SIZE counts half of what a copy reads
    assert 1.9 < blob["fetch_scale"] < 2.1 and 0.9 < blob["write_scale"] < 1.1
    ids = {e["id"] for e in blob["kernels"].values()}
    assert "hash_blocks" in ids and ("chain_stair" in ids or "sort_onesweep_pass" in ids)
    for e in blob["kernels"].values():
        assert e["avg_ms"] > 0 and e["launches_per_run"] > 0
        assert e["read_bytes"] >= 0 and e["write_bytes"] >= 0
    # each summary names the commands that made it, from committed files only
    assert "rocprofv3 --kernel-trace --stats" in text and "--pmc FETCH_SIZE" in text
    assert "_work" not in text
    # the bench arguments of the configuration, in every command
    for arg in {"generic": ["--prev-next generic"], "chained": []}[key[1]] + \
            {"request": ["--residency request"], "session": ["--residency session"], "profile": ["--profile"],
             "access": []}[key[0]] + (["--workload %s" % key[2]] if key[2] != "full" else []) + \
            (["--block-size %d" % key[3]] if key[3] != 16 else []) + \
            (["--sessions %d" % key[4]] if key[4] else []):
        assert text.count(arg) == 3, (key, arg)


def test_traffic_only_for_the_sources_it_was_taken_with(monkeypatch, tmp_path):
    text = open(bench.profile_for("access", "chained")).read()
    blob = json.loads(text[text.index("```json") + 7:text.rindex("```")])
    for sha, want in ((bench.source_sha256(), True), ("0" * 64, False)):
        blob["source_sha256"] = sha
        p = tmp_path / ("p_%s.md" % want)
        p.write_text("x\n```json\n" + json.dumps(blob) + "\n```\n")
        monkeypatch.setattr(bench, "PROFILE", str(p))
        got = bench.measured_traffic("sort_onesweep_pass")
        assert (got is not None) == want
        if want:
            e = blob["kernels"]["pc::sort_pass_kernel"]
            assert got["read_bytes"] == e["read_bytes"] and got["write_bytes"] == e["write_bytes"]


def test_quantile_and_profile_summary():
    e = [10, 20, 30]
    assert bench._quantile([0, 0, 0, 0], e, 0.5) is None
    assert bench._quantile([1, 1, 1, 1], e, 0.5) == 20       # two of four at or below the second bin
    assert bench._quantile([0, 0, 0, 4], e, 0.5) == float("inf")
    # 4 blocks used once, 2 used twice, 1 used three times; sessions of
    # footprint 1 (x3) and 7 (x1)
    freq = [0, 4, 2, 1]
    rp = {"interval": [1, 0, 0, 0], "lifetime": [5, 1, 1, 0], "freq": freq}
    fp = [0, 3, 0, 0, 0, 0, 0, 1]
    sp = {"footprint": fp, "duration": [4, 0], "gap": [0, 0]}
    bench.PROFILE_EDGES_US, saved = [10, 20, 30], bench.PROFILE_EDGES_US
    try:
        s = bench.profile_summary(rp, sp)
    finally:
        bench.PROFILE_EDGES_US = saved
    assert s["one_access_blocks"] == round(4 / 7, 4)
    assert s["p_reuse_after_1"] == round(3 / 7, 4)
    assert s["p_reuse_after_2"] == round(1 / 3, 4)
    assert s["sessions"] == 4
    # the top 10% of 4 sessions is the largest one: 7 of 10 blocks
    assert s["footprint_top10pct_share"] == 0.7


def test_profile_is_chosen_by_mode_path_and_workload(monkeypatch):
    assert bench.profile_for("access", "chained") == bench.PROFILE
    assert bench.profile_for("access", "chained", "chat").endswith("all_kernels_chat_2e8.md")
    assert bench.profile_for("access", "chained", "agent", 64).endswith("all_kernels_agent_B64.md")
    assert bench.profile_for("access", "chained", "agent", 16, bench.AGENT_3E8_SESSIONS).endswith(
        "all_kernels_agent_3e8.md")
    assert bench.profile_for("access", "chained", "full", 64) is None
    assert bench.profile_for("access", "chained", "agent", 16, 1234) is None
    # a path without a committed summary reports no counter traffic
    monkeypatch.setattr(bench, "PROFILE", bench.profile_for("request", "generic"))
    assert bench.PROFILE is None
    assert bench.measured_traffic("hash_blocks") is None and bench.measured_stage_bytes(lambda k: k) is None


def test_cpu_baseline_reports_threads_nproc_and_model():
    import numpy as np
    import pcgen
    tr = pcgen.make_trace("tiny")
    cb = bench.cpu_baseline(tr, tr.caps(), 1, 0, 20_000)
    assert cb["cores"] == bench.baseline_threads(tr.caps().size) >= 1
    assert cb["nproc"] == os.cpu_count()
    assert cb["kind"] == "oracle" and cb["value"] > 0 and "threads" in cb["sample"]
    assert "cpu_model" in cb


def test_golden_check_accepts_the_oracle_and_rejects_a_change(tmp_path):
    # a reference written the way tests/golden/make_fullsize.py writes it,
    # for the tiny trace, checked against the oracle's own bins
    import numpy as np
    import oracle
    import pcgen
    tr = pcgen.make_trace("tiny")
    caps = tr.caps()
    keys, depth = oracle.hash_trace(tr)
    prev, nxt = oracle.prev_next(keys)
    sims = oracle.lru(keys, [int(c) for c in caps], depth, fingerprints=True)
    nu = oracle.nextuse_hist(nxt, caps)
    p = tmp_path / "ref.txt"
    with open(p, "w") as f:
        f.write("n %d\ndepth_total %d\nnextuse %s\n" % (keys.size, int(depth.sum()), " ".join(map(str, nu))))
        for c, (h, dh, fp) in zip(caps, sims):
            f.write("cap %d %d %d 0x%016x\n" % (int(c), h, dh, fp))
    count, dsum, cost = oracle.mrc_bins(keys, caps, depth)
    bins = {"count": count, "depthsum": dsum, "nextuse": nu}
    assert bench.check_against_golden(bins, caps, keys.size, str(p))["bins_match"]
    bad = dict(bins, count=list(count))
    bad["count"][3] += 1
    bad["count"][4] -= 1
    with pytest.raises(SystemExit):
        bench.check_against_golden(bad, caps, keys.size, str(p))
