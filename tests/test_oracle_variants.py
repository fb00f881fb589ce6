"""Pins for the oracle's variants: mean pooling (forward and gradient), 8-bit
row-wise quantised tables, and int32 indices / offsets.

Independent of the oracle's loops: a hand-worked fixture, torch's CPU
embedding_bag in "mean" mode, dense multi-hot products built explicitly with
numpy, the oracle's own (separately pinned) fp32 path on exactly representable
tables, and identities of the definitions (the mean of equal rows is that row,
column sums, the adjoint identity).
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
from tests.tiny_cases import dense_A, table_as_f64, tiny_case

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _hand():
    g = json.load(open(os.path.join(GOLDEN, "variants_hand_worked.json")))
    D = g["dims"][0]
    rows = []
    for c, s, b in zip(g["codes"], g["scale"], g["bias"]):
        rows.append(np.concatenate([np.array(c, np.uint8), np.array([s, b], np.float32).view(np.uint8),
                                    np.zeros(8, np.uint8)]))
    g["u8_table"] = np.stack(rows)
    assert g["u8_table"].shape == (g["rows"][0], D + 16)
    return g


def lengths_of(case):
    return np.diff(case["offsets"]).astype(np.float64)


def dense_mean_forward(case):
    """Brute force: (A_t / L_b) @ W_t, the multi-hot matrix with each bag's row
    divided by its lookup count (empty bags stay zero)."""
    T, B = case["T"], case["B"]
    L = lengths_of(case)
    cols = []
    for t in range(T):
        A = dense_A(case, t)
        Lt = L[t * B:(t + 1) * B]
        A = A / np.where(Lt > 0, Lt, 1.0)[:, None]
        cols.append(A @ table_as_f64(case["tables"][t], case["dtype"]))
    return np.concatenate(cols, 1)


# ------------------------------------------------------------ hand-worked


def test_u8_rows_decode_by_hand(oracle_lib):
    g = _hand()
    D = g["dims"][0]
    for r in range(g["rows"][0]):
        for d in range(D):
            assert oracle.decode_row(g["u8_table"], "u8", D, r, d) == g["values"][r][d]


@pytest.mark.parametrize("pooling", ["sum", "mean"])
def test_hand_worked_u8_forward(oracle_lib, pooling):
    g = _hand()
    out, _ = oracle.forward(g["rows"], g["dims"], "u8", [g["u8_table"]], g["indices"], g["offsets"], g["B"],
                            pooling=pooling)
    np.testing.assert_array_equal(out, np.array(g["out_" + pooling]))


@pytest.mark.parametrize("pooling", ["sum", "mean"])
def test_hand_worked_backward_pooling(oracle_lib, pooling):
    g = _hand()
    seg = oracle.backward_segments(g["rows"], g["dims"], g["indices"], g["offsets"], g["B"])
    np.testing.assert_array_equal(seg["grad_idx"], g["grad_idx"])
    rows, _, _ = oracle.backward_rows(g["rows"], g["dims"], g["offsets"], g["B"],
                                      np.array(g["grad_out"], np.float32), seg, pooling=pooling)
    np.testing.assert_array_equal(rows, np.array(g["grad_rows_" + pooling], np.float64).reshape(-1))


# ------------------------------------------------------------ mean pooling


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_mean_matches_dense_and_torch(oracle_lib, dtype):
    rng = np.random.default_rng([31, len(dtype)])
    for _ in range(30):
        case = tiny_case(rng, dtype=dtype)
        out, ab = oracle.forward(case["rows"], case["dims"], dtype, case["tables"], case["indices"],
                                 case["offsets"], case["B"], pooling="mean")
        err = oracle.summation_error(out, dense_mean_forward(case), ab)
        assert err.max() <= 1e-13
        cols = []
        B = case["B"]
        for t in range(case["T"]):
            o = case["offsets"][t * B:(t + 1) * B + 1]
            idx = torch.from_numpy(case["indices"][o[0]:o[-1]])
            W = torch.from_numpy(table_as_f64(case["tables"][t], dtype))
            cols.append(torch.nn.functional.embedding_bag(idx, W, torch.from_numpy(o[:-1] - o[0]),
                                                          mode="mean").numpy())
        np.testing.assert_allclose(out, np.concatenate(cols, 1), rtol=1e-12, atol=1e-14)


def test_mean_identities(oracle_lib):
    rng = np.random.default_rng(32)
    for _ in range(20):
        case = tiny_case(rng, dtype="f16", p_empty=0.3)
        T, B, off = case["T"], case["B"], case["offsets"]
        dim_off = np.concatenate([[0], np.cumsum(case["dims"])])
        # every lookup of a bag on one row: the mean is that row, exactly
        same = case.copy()
        same["indices"] = case["indices"].copy()
        for k in range(T * B):
            if off[k] < off[k + 1]:
                same["indices"][off[k]:off[k + 1]] = case["indices"][off[k]]
        out, _ = oracle.forward(case["rows"], case["dims"], "f16", case["tables"], same["indices"], off, B,
                                pooling="mean")
        for k in range(T * B):
            t, b = divmod(k, B)
            seg = out[b, dim_off[t]:dim_off[t + 1]]
            if off[k] == off[k + 1]:
                assert np.all(seg == 0) and not np.any(np.signbit(seg))
            else:
                np.testing.assert_array_equal(seg, case["tables"][t][case["indices"][off[k]]].astype(np.float64))


def test_mean_takes_no_weights(oracle_lib):
    tabs = [np.zeros((4, 8), np.float32)]
    with pytest.raises(oracle.OracleError):
        oracle.forward([4], [8], "f32", tabs, [0, 1], [0, 2], 1, weights=np.ones(2, np.float32), pooling="mean")
    seg = oracle.backward_segments([4], [8], [0, 1], [0, 2], 1)
    with pytest.raises(oracle.OracleError):
        oracle.backward_rows([4], [8], [0, 2], 1, np.zeros((1, 8), np.float32), seg,
                             weights=np.ones(2, np.float32), pooling="mean")


def test_mean_backward_matches_dense_and_identities(oracle_lib):
    rng = np.random.default_rng(33)
    for _ in range(25):
        case = tiny_case(rng, dtype="f32", max_R=16, p_empty=0.25)
        T, B, off = case["T"], case["B"], case["offsets"]
        dims = case["dims"].astype(np.int64)
        dim_off = np.concatenate([[0], np.cumsum(dims)])
        row_base = np.concatenate([[0], np.cumsum(case["rows"])])
        L = lengths_of(case)
        G = rng.standard_normal((B, int(dims.sum()))).astype(np.float32)
        seg = oracle.backward_segments(case["rows"], dims, case["indices"], off, B)
        rows, ab, ro = oracle.backward_rows(case["rows"], dims, off, B, G, seg, pooling="mean")
        tab_of_u = np.searchsorted(row_base, seg["grad_idx"], side="right") - 1
        for t in range(T):
            A = dense_A(case, t)
            Lt = L[t * B:(t + 1) * B]
            A = A / np.where(Lt > 0, Lt, 1.0)[:, None]
            full = A.T @ G[:, dim_off[t]:dim_off[t + 1]].astype(np.float64)
            colsum = np.zeros(dims[t])
            for u in np.nonzero(tab_of_u == t)[0]:
                r = int(seg["grad_idx"][u] - row_base[t])
                got = rows[ro[u]:ro[u + 1]]
                assert oracle.summation_error(got, full[r], ab[ro[u]:ro[u + 1]]).max() <= 1e-13
                colsum += got
            # column sums: each nonempty bag passes its grad_out row once in total
            expect = G[Lt > 0, dim_off[t]:dim_off[t + 1]].astype(np.float64).sum(0)
            np.testing.assert_allclose(colsum, expect, rtol=1e-12, atol=1e-12)
        # adjoint identity <G, F_mean(W)> = sum_u <g_u, W[row_u]>
        out, _ = oracle.forward(case["rows"], dims, "f32", case["tables"], case["indices"], off, B, pooling="mean")
        lhs = float((G.astype(np.float64) * out).sum())
        rhs = 0.0
        for u, key in enumerate(seg["grad_idx"]):
            t = int(tab_of_u[u])
            rhs += float(rows[ro[u]:ro[u + 1]] @ table_as_f64(case["tables"][t], "f32")[key - row_base[t]])
        assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))


# ------------------------------------------------------------ 8-bit row-wise tables


def _u8_case(rng, exact: bool):
    """A tiny case whose tables are 8-bit row-wise; with exact=True every
    scale is a power of two and every bias a multiple of 2^-10, so every
    dequantised value is exactly an fp32 (returned beside it as an f32 table
    built from codes and parameters with numpy)."""
    case = tiny_case(rng, dtype="f32", dims=(8, 16, 64))
    u8, f32 = [], []
    for t in range(case["T"]):
        R, D = int(case["rows"][t]), int(case["dims"][t])
        codes = rng.integers(0, 256, (R, D)).astype(np.uint8)
        if exact:
            scale = (2.0 ** -rng.integers(4, 12, R)).astype(np.float32)
            bias = (rng.integers(-64, 64, R) * 2.0 ** -10).astype(np.float32)
        else:
            scale = rng.uniform(1e-4, 1e-2, R).astype(np.float32)
            bias = rng.uniform(-0.1, 0.1, R).astype(np.float32)
        pad = rng.integers(0, 256, (R, 8)).astype(np.uint8)  # padding bytes carry no meaning
        u8.append(np.concatenate([codes, np.stack([scale, bias], 1).view(np.uint8), pad], 1))
        f32.append((codes.astype(np.float64) * scale[:, None].astype(np.float64)
                    + bias[:, None].astype(np.float64)))
    return case, u8, f32


@pytest.mark.parametrize("pooling", ["sum", "mean"])
def test_u8_equals_f32_path_on_exact_tables(oracle_lib, pooling):
    rng = np.random.default_rng(34)
    for _ in range(20):
        case, u8, f32 = _u8_case(rng, exact=True)
        assert all(np.array_equal(t.astype(np.float32).astype(np.float64), t) for t in f32)
        w = rng.standard_normal(case["indices"].size).astype(np.float32) if pooling == "sum" else None
        a, aa = oracle.forward(case["rows"], case["dims"], "u8", u8, case["indices"], case["offsets"], case["B"],
                               weights=w, pooling=pooling)
        b, bb = oracle.forward(case["rows"], case["dims"], "f32", [t.astype(np.float32) for t in f32],
                               case["indices"], case["offsets"], case["B"], weights=w, pooling=pooling)
        np.testing.assert_array_equal(a, b)
        np.testing.assert_array_equal(aa, bb)


def test_u8_matches_torch_on_dequantised_tables(oracle_lib):
    rng = np.random.default_rng(35)
    for _ in range(20):
        case, u8, f64 = _u8_case(rng, exact=False)
        for pooling in ("sum", "mean"):
            out, _ = oracle.forward(case["rows"], case["dims"], "u8", u8, case["indices"], case["offsets"],
                                    case["B"], pooling=pooling)
            B = case["B"]
            cols = []
            for t in range(case["T"]):
                o = case["offsets"][t * B:(t + 1) * B + 1]
                idx = torch.from_numpy(case["indices"][o[0]:o[-1]])
                cols.append(torch.nn.functional.embedding_bag(idx, torch.from_numpy(f64[t]),
                                                              torch.from_numpy(o[:-1] - o[0]),
                                                              mode=pooling).numpy())
            np.testing.assert_allclose(out, np.concatenate(cols, 1), rtol=1e-12, atol=1e-14)


def test_u8_weight_grad_equals_f32_path(oracle_lib):
    rng = np.random.default_rng(36)
    case, u8, f32 = _u8_case(rng, exact=True)
    G = rng.standard_normal((case["B"], int(case["dims"].sum()))).astype(np.float32)
    a, _ = oracle.weight_grad(case["rows"], case["dims"], "u8", u8, case["indices"], case["offsets"], case["B"], G)
    b, _ = oracle.weight_grad(case["rows"], case["dims"], "f32", [t.astype(np.float32) for t in f32],
                              case["indices"], case["offsets"], case["B"], G)
    np.testing.assert_array_equal(a, b)


# ------------------------------------------------------------ int32 indices and offsets


def test_int32_indices_and_offsets_are_the_same_values(oracle_lib):
    rng = np.random.default_rng(37)
    case = tiny_case(rng, dtype="bf16")
    a, _ = oracle.forward(case["rows"], case["dims"], "bf16", case["tables"], case["indices"], case["offsets"],
                          case["B"])
    b, _ = oracle.forward(case["rows"], case["dims"], "bf16", case["tables"], case["indices"].astype(np.int32),
                          case["offsets"].astype(np.int32), case["B"])
    np.testing.assert_array_equal(a, b)
