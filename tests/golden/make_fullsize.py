"""Write the full-size oracle references ``fullsize_<workload>.txt``.

Run as ``python tests/golden/make_fullsize.py <workload> [threads]`` with
workload one of ``chat`` (the chat-shaped trace, 20,000 sessions), ``full``
(the mixed 2e9-context-token trace) or ``full_2g2`` (the same mix up to
2.2e9 context tokens, so that access positions pass 2^31).  It calls only
``pcgen`` (the seeded inputs) and ``oracle/`` (the plain CPU definitions):

* keys and depths of every block, hashed request by request;
* prev / next from a last-seen scan over dense key ids;
* the exact stack distance of every access (Fenwick tree over
  last-occurrence marks, Bennett & Kruskal 1975);
* one LRU list simulation per capacity edge (Sec. 5 "LRU as a bedrock";
  Appendix A sweeps capacities), run on a thread pool, each giving the hit
  count, the depth sum over the hits and the hit-set fingerprint
  (sum of mix64(t + 1) over the hits t).

The two ways of scoring LRU (per-capacity simulation, distances binned on
the edges) must agree on every capacity's hit count and hit-set
fingerprint before anything is written.  Whole arrays are recorded as
fingerprints: sum over t of mix64(mix64(t + 1) + a[t]) mod 2^64.
"""
import dataclasses
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import pcgen  # noqa: E402

WORKLOADS = {
    "chat": dict(config="chat"),
    "full": dict(config="full"),
    "full_2g2": dict(config="full", target_tokens=2_200_000_000),
}
CHUNK = 1 << 26


def plain_pages():
    """Ask numpy not to request transparent huge pages for its large arrays:
    on hosts that compact memory to serve them, first touching tens of GB
    otherwise takes minutes of kernel time."""
    for mod in ("_core", "core"):
        try:
            getattr(np, mod).multiarray._set_madvise_hugepage(False)
            return
        except AttributeError:
            continue


def make(name):
    w = WORKLOADS[name]
    return pcgen.make_trace(w["config"], target_tokens=w.get("target_tokens"))


def log(*a):
    print("[make_fullsize]", *a, file=sys.stderr, flush=True)


def main():
    name = sys.argv[1]
    plain_pages()
    threads = int(sys.argv[2]) if len(sys.argv) > 2 else (os.cpu_count() or 1)
    secs = {}
    t0 = time.time()
    tr = make(name)
    caps = tr.caps()
    k = caps.size
    n = tr.n_blocks()
    log(name, "trace:", tr.n_requests, "requests", n, "accesses")
    secs["generate"] = time.time() - t0

    t0 = time.time()
    keys, depth = oracle.hash_trace(tr, threads=threads)
    secs["hash"] = time.time() - t0
    tr = dataclasses.replace(tr, tokens=np.empty(0, np.int32))   # tokens no longer needed
    fp_keys = oracle.fingerprint(keys)
    fp_depth = oracle.fingerprint(depth)
    depth_total = int(sum(int(depth[i:i + CHUNK].sum(dtype=np.uint64)) for i in range(0, n, CHUNK)))
    log("hashed in %.0f s" % secs["hash"])

    t0 = time.time()
    ids = oracle.key_ids(keys)
    del keys
    secs["key_ids"] = time.time() - t0
    log("%d distinct keys in %.0f s" % (ids[1], secs["key_ids"]))

    t0 = time.time()
    prev, nxt = oracle.prev_next(None, ids)
    secs["prev_next"] = time.time() - t0
    fp_prev = oracle.fingerprint(prev)
    fp_next = oracle.fingerprint(nxt)
    nextuse = np.zeros(k + 1, np.int64)
    for i in range(0, n, CHUNK):
        nextuse += np.array(oracle.nextuse_hist(nxt[i:i + CHUNK], caps, t0=i), np.int64)
    del nxt
    log("prev/next in %.0f s" % secs["prev_next"])

    t0 = time.time()
    dist = oracle.stack_distance_bit(prev)
    secs["stack_distance"] = time.time() - t0
    del prev
    fp_dist = oracle.fingerprint(dist)
    dcount = np.zeros(k + 1, np.uint64)
    dfp = np.zeros(k + 1, np.uint64)
    for i in range(0, n, CHUNK):
        oracle.dist_bins(dist[i:i + CHUNK], caps, t0=i, count=dcount, fp=dfp)
    del dist
    log("stack distances in %.0f s" % secs["stack_distance"])

    t0 = time.time()
    sims = oracle.lru(None, [int(c) for c in caps], depth, ids, threads=threads, fingerprints=True)
    secs["lru_per_capacity"] = time.time() - t0
    log("%d LRU simulations on %d threads in %.0f s" % (k, threads, secs["lru_per_capacity"]))

    # the per-capacity simulations and the binned distances must agree
    hits_d = np.cumsum(dcount[:k].astype(np.uint64))
    fp_d = np.cumsum(dfp[:k], dtype=np.uint64)
    for j, (h, dh, fp) in enumerate(sims):
        assert h == int(hits_d[j]) and fp == int(fp_d[j]), (j, int(caps[j]), h, int(hits_d[j]))
    assert int(dcount.sum()) == n

    out = os.path.join(HERE, "fullsize_%s.txt" % name)
    with open(out, "w") as f:
        f.write("# Full-size oracle reference for the '%s' trace (pcgen, seed %d).\n" % (name, tr.config.seed))
        f.write("# Written by: python tests/golden/make_fullsize.py %s  (calls pcgen and oracle/ only).\n" % name)
        f.write("# Array fingerprints: sum_t mix64(mix64(t+1) + a[t]) mod 2^64 (u32 arrays zero-extended).\n")
        f.write("# Per capacity: LRU hits, depth sum over the hits, hit-set fingerprint sum mix64(t+1);\n")
        f.write("# per-capacity list simulations and the Fenwick stack distances agreed on every one.\n")
        f.write("# Oracle seconds (%d threads for hashing and the simulations): %s\n" % (
            threads, " ".join("%s=%.0f" % kv for kv in secs.items())))
        f.write("workload %s\n" % name)
        f.write("n %d\n" % n)
        f.write("requests %d\n" % tr.n_requests)
        f.write("distinct %d\n" % ids[1])
        f.write("depth_total %d\n" % depth_total)
        for nm, v in (("keys", fp_keys), ("depth", fp_depth), ("prev", fp_prev), ("next", fp_next),
                      ("dist", fp_dist)):
            f.write("fp_%s 0x%016x\n" % (nm, v))
        f.write("nextuse %s\n" % " ".join(str(int(x)) for x in nextuse))
        f.write("# cap hits depthsum_hits hitset_fp\n")
        for c, (h, dh, fp) in zip(caps, sims):
            f.write("cap %d %d %d 0x%016x\n" % (int(c), h, dh, fp))
    log("wrote", out)


if __name__ == "__main__":
    main()
