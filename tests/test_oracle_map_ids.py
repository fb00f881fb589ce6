"""Pins of the oracle's MapId preprocessing (CPU only): the paper's worked
example, numpy's searchsorted, and the properties that determine the output."""
import json
import os

import numpy as np

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "mapid_example.json")


def test_paper_worked_example(oracle_lib):
    ex = json.load(open(GOLDEN))
    np.testing.assert_array_equal(oracle.map_ids(ex["values"], ex["mapping"]), ex["expected"])


def random_case(rng, m, n, dup=False):
    M = np.sort(rng.integers(-50, 50, size=m) if dup else rng.choice(np.arange(-1000, 1000), size=m, replace=False))
    v = rng.integers(-60, 60, size=n) if dup else rng.integers(-1100, 1100, size=n)
    if m and n:
        hit = rng.random(n) < 0.5
        v[hit] = rng.choice(M, size=int(hit.sum()))
    return M.astype(np.int64), v.astype(np.int64)


def test_matches_searchsorted(oracle_lib):
    rng = np.random.default_rng(31)
    for _ in range(200):
        m, n = int(rng.integers(1, 40)), int(rng.integers(0, 60))
        M, v = random_case(rng, m, n, dup=bool(rng.integers(2)))
        p = np.minimum(np.searchsorted(M, v, side="left"), m - 1)
        want = np.where(M[p] == v, p + 1, 0)
        np.testing.assert_array_equal(oracle.map_ids(v, M), want)


def test_output_properties(oracle_lib):
    """out = 0 exactly for values not in the mapping; otherwise out - 1 is the
    first position holding the value."""
    rng = np.random.default_rng(32)
    for _ in range(100):
        m, n = int(rng.integers(1, 30)), 50
        M, v = random_case(rng, m, n, dup=True)
        out = oracle.map_ids(v, M)
        for x, o in zip(v, out):
            if x in M:
                assert 1 <= o <= m and M[o - 1] == x and (o == 1 or M[o - 2] < x)
            else:
                assert o == 0


def test_edges(oracle_lib):
    assert oracle.map_ids([5, -3], []).tolist() == [0, 0]      # no known ids
    assert oracle.map_ids([7, 6, 8], [7]).tolist() == [1, 0, 0]
    big = np.array([np.iinfo(np.int64).min, -1, 0, np.iinfo(np.int64).max], np.int64)
    assert oracle.map_ids(big, big).tolist() == [1, 2, 3, 4]
    assert oracle.map_ids(np.zeros(0, np.int64), big).size == 0
