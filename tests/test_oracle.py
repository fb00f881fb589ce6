"""Pins for the CPU oracle: brute-force dense one-hot products, library special
cases, a hand-worked fixture and the invariants of the pooled-lookup definition.

None of these checks re-types the oracle's own loops: the dense checks build the
multi-hot matrix explicitly and multiply it with numpy; the library checks call
torch.nn.functional.embedding_bag and numpy's sort/unique routines; the fixture
was worked by hand; the invariants follow from linearity of the definition.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
from tests.tiny_cases import dense_backward, dense_forward, table_as_f64, tiny_case

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def fwd(case):
    return oracle.forward(case["rows"], case["dims"], case["dtype"], case["tables"], case["indices"],
                          case["offsets"], case["B"], case["weights"])


# ---------------------------------------------------------------- formats


def test_fp16_decode_matches_numpy_for_every_pattern(oracle_lib):
    words = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = oracle.decode(words, "f16")
    ref = words.view(np.float16).astype(np.float64)
    finite = np.isfinite(ref)
    np.testing.assert_array_equal(got[finite], ref[finite])
    assert np.all(np.isnan(got[np.isnan(ref)]))
    assert np.all(got[np.isinf(ref)] == ref[np.isinf(ref)])


def test_bf16_decode_matches_torch_for_every_pattern(oracle_lib):
    words = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = oracle.decode(words, "bf16")
    ref = torch.from_numpy(words.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    finite = np.isfinite(ref)
    np.testing.assert_array_equal(got[finite], ref[finite])


# ---------------------------------------------------------------- forward


def test_hand_worked_forward(oracle_lib):
    g = json.load(open(os.path.join(GOLDEN, "hand_worked.json")))
    tabs = [np.array(t, np.float32) for t in g["tables"]]
    out, _ = oracle.forward(g["rows"], g["dims"], "f32", tabs, g["indices"], g["offsets"], g["B"])
    np.testing.assert_array_equal(out, np.array(g["out"], np.float64))
    out, ab = oracle.forward(g["rows"], g["dims"], "f32", tabs, g["indices"], g["offsets"], g["B"],
                             np.array(g["weights"], np.float32))
    np.testing.assert_array_equal(out, np.array(g["out_weighted"], np.float64))
    np.testing.assert_array_equal(ab, np.array(g["abs_weighted"], np.float64))


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("weighted", [False, True])
def test_forward_matches_dense_one_hot(oracle_lib, dtype, weighted):
    rng = np.random.default_rng([7, len(dtype), weighted])
    for _ in range(40):
        case = tiny_case(rng, dtype=dtype, weighted=weighted)
        out, ab = fwd(case)
        ref = dense_forward(case)
        err = oracle.summation_error(out, ref, ab)
        assert err.max() <= 1e-13, err.max()


def test_forward_matches_torch_embedding_bag(oracle_lib):
    rng = np.random.default_rng(11)
    for _ in range(30):
        case = tiny_case(rng, dtype="f32", weighted=bool(rng.integers(2)))
        out, _ = fwd(case)
        cols = []
        for t in range(case["T"]):
            B = case["B"]
            o = case["offsets"][t * B:(t + 1) * B + 1]
            idx = torch.from_numpy(case["indices"][o[0]:o[-1]])
            w = None if case["weights"] is None else torch.from_numpy(case["weights"][o[0]:o[-1]]).double()
            W = torch.from_numpy(table_as_f64(case["tables"][t], "f32"))
            cols.append(torch.nn.functional.embedding_bag(idx, W, torch.from_numpy(o[:-1] - o[0]), mode="sum",
                                                          per_sample_weights=w).numpy())
        np.testing.assert_allclose(out, np.concatenate(cols, 1), rtol=1e-12, atol=1e-12)


def test_one_hot_bags_are_a_plain_gather(oracle_lib):
    rng = np.random.default_rng(5)
    rows = np.array([50, 7, 300]); dims = np.array([8, 16, 64], np.int32); B = 33
    tabs = [rng.standard_normal((r, d)).astype(np.float16) for r, d in zip(rows, dims)]
    idx = np.concatenate([rng.integers(0, r, B) for r in rows]).astype(np.int64)
    off = np.arange(3 * B + 1, dtype=np.int64)
    out, _ = oracle.forward(rows, dims, "f16", tabs, idx, off, B)
    ref = np.concatenate([np.take(tabs[t], idx[t * B:(t + 1) * B], axis=0).astype(np.float64)
                          for t in range(3)], 1)
    np.testing.assert_array_equal(out, ref)


def test_invariants(oracle_lib):
    rng = np.random.default_rng(3)
    for _ in range(25):
        case = tiny_case(rng, dtype="f32", weighted=True, integer_values=True, p_empty=0.3)
        case["weights"] = rng.integers(-4, 5, case["indices"].size).astype(np.float32)  # exact sums
        out, _ = fwd(case)
        T, B, off = case["T"], case["B"], case["offsets"]
        dim_off = np.concatenate([[0], np.cumsum(case["dims"])])
        # empty bag -> exactly +0.0
        for k in range(T * B):
            if off[k] == off[k + 1]:
                seg = out[k % B, dim_off[k // B]:dim_off[k // B + 1]]
                assert np.all(seg == 0) and not np.any(np.signbit(seg))
        # permuting the lookups inside each bag leaves the result unchanged
        p = case.copy()
        perm = np.arange(case["indices"].size)
        for k in range(T * B):
            perm[off[k]:off[k + 1]] = rng.permutation(perm[off[k]:off[k + 1]])
        p["indices"], p["weights"] = case["indices"][perm], case["weights"][perm]
        np.testing.assert_array_equal(fwd(p)[0], out)
        # a lookup listed twice equals the same lookup with twice the weight
        if case["indices"].size:
            j = int(rng.integers(case["indices"].size))
            k = int(np.searchsorted(off, j, side="right") - 1)
            d = case.copy()
            d["indices"] = np.insert(case["indices"], j, case["indices"][j])
            d["weights"] = np.insert(case["weights"], j, case["weights"][j])
            d["offsets"] = off + (np.arange(off.size) > k)
            w2 = case.copy()
            w2["weights"] = case["weights"].copy()
            w2["weights"][j] *= 2
            np.testing.assert_array_equal(fwd(d)[0], fwd(w2)[0])
        # scaling every table by 2^k scales the output by exactly 2^k
        s = case.copy()
        s["tables"] = [t * np.float32(2.0 ** -3) for t in case["tables"]]
        np.testing.assert_array_equal(fwd(s)[0], out * 2.0 ** -3)


def test_additivity_split_bag(oracle_lib):
    rng = np.random.default_rng(4)
    case = tiny_case(rng, dtype="f32", weighted=True, max_T=1, max_B=1, max_L=12, p_empty=0.0)
    case["offsets"] = np.array([0, case["indices"].size], np.int64)
    full, _ = fwd(case)
    n = case["indices"].size
    m = n // 2
    a = dict(case, offsets=np.array([0, m], np.int64), indices=case["indices"][:m], weights=case["weights"][:m])
    b = dict(case, offsets=np.array([0, n - m], np.int64), indices=case["indices"][m:], weights=case["weights"][m:])
    np.testing.assert_allclose(fwd(a)[0] + fwd(b)[0], full, rtol=1e-14, atol=1e-14)


def test_forward_rejects_bad_inputs(oracle_lib):
    tabs = [np.zeros((4, 8), np.float32)]
    with pytest.raises(oracle.OracleError):
        oracle.forward([4], [8], "f32", tabs, [0, 4], [0, 2], 1)  # index 4 of 4 rows
    with pytest.raises(oracle.OracleError):
        oracle.forward([4], [8], "f32", tabs, [0, 1], [0, 3, 2], 2)  # offsets not monotone
    with pytest.raises(oracle.OracleError):
        oracle.forward([4], [8], "f32", tabs, [0, 1], [0, 1], 1)  # last offset != N


# ---------------------------------------------------------------- backward


def test_hand_worked_backward(oracle_lib):
    g = json.load(open(os.path.join(GOLDEN, "hand_worked.json")))
    seg = oracle.backward_segments(g["rows"], g["dims"], g["indices"], g["offsets"], g["B"])
    for key in ("perm", "sorted_keys", "grad_idx", "seg_offsets", "grad_row_offsets"):
        np.testing.assert_array_equal(seg[key], g[key], err_msg=key)
    G = np.array(g["grad_out"], np.float32)
    rows, _, _ = oracle.backward_rows(g["rows"], g["dims"], g["offsets"], g["B"], G, seg)
    np.testing.assert_array_equal(rows, g["grad_rows"])
    rows, _, _ = oracle.backward_rows(g["rows"], g["dims"], g["offsets"], g["B"], G, seg,
                                      weights=np.array(g["weights"], np.float32))
    np.testing.assert_array_equal(rows, g["grad_rows_weighted"])


@pytest.mark.parametrize("weighted", [False, True])
def test_backward_matches_library_sort_and_dense(oracle_lib, weighted):
    rng = np.random.default_rng([21, weighted])
    for _ in range(40):
        case = tiny_case(rng, dtype="f16", weighted=weighted, max_R=16)
        T, B = case["T"], case["B"]
        row_base = np.concatenate([[0], np.cumsum(case["rows"])])
        off, idx = case["offsets"], case["indices"]
        tab_of_j = np.repeat(np.arange(T), [off[(t + 1) * B] - off[t * B] for t in range(T)])
        keys = row_base[tab_of_j] + idx
        seg = oracle.backward_segments(case["rows"], case["dims"], idx, off, B)
        uniq, counts = np.unique(keys, return_counts=True)
        np.testing.assert_array_equal(seg["grad_idx"], uniq)
        np.testing.assert_array_equal(seg["seg_offsets"], np.concatenate([[0], np.cumsum(counts)]))
        np.testing.assert_array_equal(seg["perm"], np.argsort(keys, kind="stable"))
        np.testing.assert_array_equal(seg["sorted_keys"], np.sort(keys))
        tab_of_u = np.searchsorted(row_base, uniq, side="right") - 1
        np.testing.assert_array_equal(seg["grad_row_offsets"],
                                      np.concatenate([[0], np.cumsum(case["dims"][tab_of_u])]))
        G = rng.standard_normal((B, int(case["dims"].sum()))).astype(np.float32)
        rows, ab, ro = oracle.backward_rows(case["rows"], case["dims"], off, B, G, seg, weights=case["weights"])
        dense = dense_backward(case, G)
        assert sorted(dense) == list(uniq)
        for u, key in enumerate(uniq):
            got = rows[ro[u]:ro[u + 1]]
            err = oracle.summation_error(got, dense[int(key)], ab[ro[u]:ro[u + 1]])
            assert err.max() <= 1e-13


def test_backward_identities(oracle_lib):
    """Column sums equal grad_out times the pooling factor; the adjoint identity
    <G, F(W)> = sum_u <g_u, W[row_u]> holds."""
    rng = np.random.default_rng(8)
    for _ in range(20):
        case = tiny_case(rng, dtype="f32", weighted=True, integer_values=True)
        case["weights"] = rng.integers(-3, 4, case["indices"].size).astype(np.float32)
        T, B, off = case["T"], case["B"], case["offsets"]
        dims = case["dims"].astype(np.int64)
        dim_off = np.concatenate([[0], np.cumsum(dims)])
        row_base = np.concatenate([[0], np.cumsum(case["rows"])])
        G = rng.integers(-5, 6, (B, int(dims.sum()))).astype(np.float32)
        seg = oracle.backward_segments(case["rows"], dims, case["indices"], off, B)
        rows, _, ro = oracle.backward_rows(case["rows"], dims, off, B, G, seg, weights=case["weights"])
        tab_of_u = np.searchsorted(row_base, seg["grad_idx"], side="right") - 1
        for t in range(T):
            colsum = np.zeros(dims[t])
            for u in np.nonzero(tab_of_u == t)[0]:
                colsum += rows[ro[u]:ro[u + 1]]
            factor = np.array([case["weights"][off[t * B + b]:off[t * B + b + 1]].astype(np.float64).sum()
                               for b in range(B)])
            expect = factor @ G[:, dim_off[t]:dim_off[t + 1]].astype(np.float64)
            np.testing.assert_array_equal(colsum, expect)
        out, _ = fwd(case)
        lhs = float((G.astype(np.float64) * out).sum())
        rhs = 0.0
        for u, key in enumerate(seg["grad_idx"]):
            t = int(tab_of_u[u])
            W = table_as_f64(case["tables"][t], "f32")
            rhs += float(rows[ro[u]:ro[u + 1]] @ W[key - row_base[t]])
        assert lhs == rhs


def test_backward_selected_rows_equal_full(oracle_lib):
    rng = np.random.default_rng(9)
    case = tiny_case(rng, dtype="f32", max_R=8, max_B=8, max_L=12)
    G = rng.standard_normal((case["B"], int(case["dims"].sum()))).astype(np.float32)
    seg = oracle.backward_segments(case["rows"], case["dims"], case["indices"], case["offsets"], case["B"])
    full, _, ro = oracle.backward_rows(case["rows"], case["dims"], case["offsets"], case["B"], G, seg)
    sel = np.array(sorted(rng.choice(seg["U"], size=min(3, seg["U"]), replace=False)), np.int64)
    part, _, pro = oracle.backward_rows(case["rows"], case["dims"], case["offsets"], case["B"], G, seg, sel=sel)
    for s, u in enumerate(sel):
        np.testing.assert_array_equal(part[pro[s]:pro[s + 1]], full[ro[u]:ro[u + 1]])
