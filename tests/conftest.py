import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def read_golden(name):
    """Non-comment, non-empty lines of a golden fixture, split on whitespace."""
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append(line.split())
    return rows


NONE = 0xFFFFFFFF


def request_golden():
    """(name, keys, blk_off, D_req per access, {capacity: hits}) per row of the
    hand-worked request-level fixture; blocks named in a row get small ids."""
    for row in read_golden("request_residency_examples.txt"):
        bars = [i for i, x in enumerate(row) if x == "|"]
        names, reqs, cur = {}, [], []
        for x in row[1:bars[0]]:
            if x == "/":
                reqs.append(cur)
                cur = []
            else:
                cur.append(names.setdefault(x, len(names) + 7))
        reqs.append(cur)
        keys = np.array([k for r in reqs for k in r], np.uint64)
        blk_off = np.concatenate([[0], np.cumsum([len(r) for r in reqs])]).astype(np.uint64)
        want = [NONE if v == "-" else int(v) for v in row[bars[0] + 1:bars[1]]]
        hits = {int(c): int(h) for c, h in (x.split(":") for x in row[bars[1] + 1:])}
        yield row[0], keys, blk_off, want, hits


def session_golden():
    """(name, keys, blk_off, session per request, D per access, {capacity:
    hits}) per row of the hand-worked session-level fixture."""
    for row in read_golden("session_level_examples.txt"):
        bars = [i for i, x in enumerate(row) if x == "|"]
        names, snames, reqs, sess = {}, {}, [], []
        for x in row[1:bars[0]]:
            if x.endswith(":"):
                reqs.append([])
                sess.append(snames.setdefault(x[:-1], len(snames)))
            elif x != "/":
                reqs[-1].append(names.setdefault(x, len(names) + 7))
        keys = np.array([k for r in reqs for k in r], np.uint64)
        blk_off = np.concatenate([[0], np.cumsum([len(r) for r in reqs])]).astype(np.uint64)
        want = [NONE if v == "-" else int(v) for v in row[bars[0] + 1:bars[1]]]
        hits = {int(c): int(h) for c, h in (x.split(":") for x in row[bars[1] + 1:])}
        yield row[0], keys, blk_off, np.array(sess, np.uint32), want, hits


def characterization_golden():
    """The hand-worked characterisation fixture: the trace (keys, blk_off,
    session, ts_us) and a dict of expected rows."""
    rows = read_golden("characterization_example.txt")
    reqs = [r for r in rows if r[0] == "request"]
    want = {r[0]: [int(x) for x in r[1:]] for r in rows if r[0] != "request"}
    snames = {}
    sess = np.array([snames.setdefault(r[1], len(snames)) for r in reqs], np.uint32)
    ts = np.array([int(r[2]) for r in reqs], np.uint64)
    keys = np.array([int(x) for r in reqs for x in r[3:]], np.uint64)
    blk_off = np.concatenate([[0], np.cumsum([len(r) - 3 for r in reqs])]).astype(np.uint64)
    return keys, blk_off, sess, ts, want
