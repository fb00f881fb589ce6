"""Pins for the oracle's tolerance scale: the sum of |terms| that it returns
beside every pooled value and gradient element (absout), the denominator of
every parity check of the GPU path.

Independent of the oracle's loops:
  - hand-worked abs rows in the golden fixtures (signed terms, mean pooling);
  - with every term non-negative, |term| = term, so the scale must equal the
    value itself bit for bit (both are the same sum in the same order);
  - for signed inputs, the scale must equal the oracle's value on the
    elementwise absolute inputs (|W|, |w|, |grad_out|), whose pooled value is
    separately pinned against brute force and torch.
A scale that dropped the weight, forgot mean pooling's 1/L or took |x| of the
wrong factor fails at least one of these.
"""
import json
import os

import numpy as np
import pytest

import oracle
from tests.tiny_cases import tiny_case

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _fixture(name):
    return json.load(open(os.path.join(GOLDEN, name)))


def _u8_table(g):
    rows = []
    for c, s, b in zip(g["codes"], g["scale"], g["bias"]):
        rows.append(np.concatenate([np.array(c, np.uint8), np.array([s, b], np.float32).view(np.uint8),
                                    np.zeros(8, np.uint8)]))
    return np.stack(rows)


def _abs_table(t, dtype):
    """|W| in the table's own storage (clear the sign bit)."""
    if dtype == "f32":
        return np.abs(t)
    if dtype == "f16":
        return np.abs(t)
    return (t & np.uint16(0x7FFF)).astype(np.uint16)


# ---------------------------------------------------------------- hand-worked


def test_hand_worked_backward_scale():
    g = _fixture("hand_worked.json")
    seg = oracle.backward_segments(g["rows"], g["dims"], g["indices"], g["offsets"], g["B"])
    G = np.array(g["grad_out"], np.float32)
    rows, ab, _ = oracle.backward_rows(g["rows"], g["dims"], g["offsets"], g["B"], G, seg,
                                       weights=np.array(g["weights"], np.float32))
    np.testing.assert_array_equal(rows, g["grad_rows_weighted"])
    np.testing.assert_array_equal(ab, g["abs_grad_rows_weighted"])
    _, ab, _ = oracle.backward_rows(g["rows"], g["dims"], g["offsets"], g["B"], G, seg)
    np.testing.assert_array_equal(ab, g["grad_rows"])  # unweighted, G > 0: scale = value


@pytest.mark.parametrize("pooling", ["sum", "mean"])
def test_hand_worked_forward_scale_u8(pooling):
    g = _fixture("variants_hand_worked.json")
    _, ab = oracle.forward(g["rows"], g["dims"], "u8", [_u8_table(g)], g["indices"], g["offsets"], g["B"],
                           pooling=pooling)
    np.testing.assert_array_equal(ab, np.array(g["abs_out_" + pooling], np.float64))


@pytest.mark.parametrize("pooling", ["sum", "mean"])
def test_hand_worked_backward_scale_signed(pooling):
    g = _fixture("variants_hand_worked.json")
    seg = oracle.backward_segments(g["rows"], g["dims"], g["indices"], g["offsets"], g["B"])
    rows, ab, _ = oracle.backward_rows(g["rows"], g["dims"], g["offsets"], g["B"],
                                       np.array(g["grad_out_signed"], np.float32), seg, pooling=pooling)
    np.testing.assert_array_equal(rows, np.array(g["grad_rows_signed_" + pooling], np.float64).reshape(-1))
    np.testing.assert_array_equal(ab, np.array(g["abs_grad_rows_signed_" + pooling], np.float64).reshape(-1))


# ------------------------------------------------------- non-negative terms


def _nonneg_case(rng, dtype, weighted):
    case = tiny_case(rng, dtype="f32", weighted=weighted, max_L=20)
    tabs = []
    for t in case["tables"]:
        a = np.abs(t)
        if dtype == "f16":
            tabs.append(a.astype(np.float16))
        elif dtype == "bf16":
            u = a.view(np.uint32)
            tabs.append(((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16))
        else:
            tabs.append(a)
    case["tables"], case["dtype"] = tabs, dtype
    if weighted:
        case["weights"] = np.abs(case["weights"])
    return case


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("mode", ["sum", "weighted", "mean"])
def test_forward_scale_equals_value_on_nonnegative_terms(dtype, mode):
    rng = np.random.default_rng([31, ["f32", "f16", "bf16"].index(dtype), ["sum", "weighted", "mean"].index(mode)])
    for _ in range(25):
        case = _nonneg_case(rng, dtype, mode == "weighted")
        out, ab = oracle.forward(case["rows"], case["dims"], dtype, case["tables"], case["indices"],
                                 case["offsets"], case["B"], case["weights"], pooling="mean" if mode == "mean" else "sum")
        np.testing.assert_array_equal(ab, out)


def test_forward_scale_equals_value_on_nonnegative_u8():
    rng = np.random.default_rng(32)
    for _ in range(20):
        R, D, B = int(rng.integers(1, 30)), int(rng.choice([16, 32, 64])), int(rng.integers(1, 7))
        tab = np.zeros((R, D + 16), np.uint8)
        tab[:, :D] = rng.integers(0, 256, (R, D))
        sb = np.stack([rng.uniform(0, 1, R), rng.uniform(0, 1, R)], 1).astype(np.float32)
        tab[:, D:D + 8] = sb.view(np.uint8).reshape(R, 8)
        L = rng.integers(0, 12, B)
        off = np.concatenate([[0], np.cumsum(L)]).astype(np.int64)
        idx = rng.integers(0, R, int(off[-1]))
        for pooling in ("sum", "mean"):
            out, ab = oracle.forward([R], [D], "u8", [tab], idx, off, B, pooling=pooling)
            np.testing.assert_array_equal(ab, out)


@pytest.mark.parametrize("mode", ["sum", "weighted", "mean"])
def test_backward_scale_equals_value_on_nonnegative_terms(mode):
    rng = np.random.default_rng([33, ["sum", "weighted", "mean"].index(mode)])
    for _ in range(25):
        case = _nonneg_case(rng, "f32", mode == "weighted")
        seg = oracle.backward_segments(case["rows"], case["dims"], case["indices"], case["offsets"], case["B"])
        G = np.abs(rng.standard_normal((case["B"], int(case["dims"].sum())))).astype(np.float32)
        rows, ab, _ = oracle.backward_rows(case["rows"], case["dims"], case["offsets"], case["B"], G, seg,
                                           weights=case["weights"], pooling="mean" if mode == "mean" else "sum")
        np.testing.assert_array_equal(ab, rows)


def test_weight_grad_scale_equals_value_on_nonnegative_terms():
    rng = np.random.default_rng(34)
    for _ in range(25):
        case = _nonneg_case(rng, "f16", False)
        G = np.abs(rng.standard_normal((case["B"], int(case["dims"].sum())))).astype(np.float32)
        gw, ab = oracle.weight_grad(case["rows"], case["dims"], "f16", case["tables"], case["indices"],
                                    case["offsets"], case["B"], G)
        np.testing.assert_array_equal(ab, gw)


# ----------------------------------------------- signed terms: value on |inputs|


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("mode", ["sum", "weighted", "mean"])
def test_forward_scale_is_value_on_absolute_inputs(dtype, mode):
    rng = np.random.default_rng([35, ["f32", "f16", "bf16"].index(dtype), ["sum", "weighted", "mean"].index(mode)])
    pooling = "mean" if mode == "mean" else "sum"
    for _ in range(25):
        case = tiny_case(rng, dtype=dtype, weighted=mode == "weighted", max_L=20)
        _, ab = oracle.forward(case["rows"], case["dims"], dtype, case["tables"], case["indices"], case["offsets"],
                               case["B"], case["weights"], pooling=pooling)
        w_abs = None if case["weights"] is None else np.abs(case["weights"])
        val, _ = oracle.forward(case["rows"], case["dims"], dtype, [_abs_table(t, dtype) for t in case["tables"]],
                                case["indices"], case["offsets"], case["B"], w_abs, pooling=pooling)
        np.testing.assert_array_equal(ab, val)


@pytest.mark.parametrize("mode", ["sum", "weighted", "mean"])
def test_backward_scale_is_value_on_absolute_inputs(mode):
    rng = np.random.default_rng([36, ["sum", "weighted", "mean"].index(mode)])
    pooling = "mean" if mode == "mean" else "sum"
    for _ in range(25):
        case = tiny_case(rng, dtype="f32", weighted=mode == "weighted", max_L=20)
        seg = oracle.backward_segments(case["rows"], case["dims"], case["indices"], case["offsets"], case["B"])
        G = rng.standard_normal((case["B"], int(case["dims"].sum()))).astype(np.float32)
        _, ab, _ = oracle.backward_rows(case["rows"], case["dims"], case["offsets"], case["B"], G, seg,
                                        weights=case["weights"], pooling=pooling)
        w_abs = None if case["weights"] is None else np.abs(case["weights"])
        val, _, _ = oracle.backward_rows(case["rows"], case["dims"], case["offsets"], case["B"], np.abs(G), seg,
                                         weights=w_abs, pooling=pooling)
        np.testing.assert_array_equal(ab, val)


def test_weight_grad_scale_is_value_on_absolute_inputs():
    rng = np.random.default_rng(37)
    for _ in range(25):
        case = tiny_case(rng, dtype="bf16", max_L=20)
        G = rng.standard_normal((case["B"], int(case["dims"].sum()))).astype(np.float32)
        _, ab = oracle.weight_grad(case["rows"], case["dims"], "bf16", case["tables"], case["indices"],
                                   case["offsets"], case["B"], G)
        val, _ = oracle.weight_grad(case["rows"], case["dims"], "bf16", [_abs_table(t, "bf16") for t in case["tables"]],
                                    case["indices"], case["offsets"], case["B"], np.abs(G))
        np.testing.assert_array_equal(ab, val)
