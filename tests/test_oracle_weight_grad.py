"""Pins of the oracle's per-sample-weight gradient (CPU only): torch's own
autograd through embedding_bag, a matrix-product form, the linearity identity
and a hand-worked case."""
import numpy as np
import torch

import oracle
from tests.tiny_cases import table_as_f64, tiny_case


def gw_of(case, G):
    return oracle.weight_grad(case["rows"], case["dims"], case["dtype"], case["tables"], case["indices"],
                              case["offsets"], case["B"], G)


def grad_out_for(rng, case):
    return rng.standard_normal((case["B"], int(case["dims"].sum()))).astype(np.float32)


def test_weight_grad_matches_torch_autograd(oracle_lib):
    rng = np.random.default_rng(21)
    for _ in range(40):
        dtype = ["f32", "f16", "bf16"][int(rng.integers(3))]
        case = tiny_case(rng, dtype=dtype, weighted=True)
        G = grad_out_for(rng, case)
        gw, _ = gw_of(case, G)
        B = case["B"]
        dim_off = np.concatenate([[0], np.cumsum(case["dims"].astype(np.int64))])
        ref = np.zeros_like(gw)
        for t in range(case["T"]):
            o = case["offsets"][t * B:(t + 1) * B + 1]
            if o[-1] == o[0]:
                continue
            idx = torch.from_numpy(case["indices"][o[0]:o[-1]])
            w = torch.from_numpy(case["weights"][o[0]:o[-1]]).double().requires_grad_(True)
            W = torch.from_numpy(table_as_f64(case["tables"][t], dtype))
            out = torch.nn.functional.embedding_bag(idx, W, torch.from_numpy(o[:-1] - o[0]), mode="sum",
                                                    per_sample_weights=w)
            (out * torch.from_numpy(G[:, dim_off[t]:dim_off[t + 1]]).double()).sum().backward()
            ref[o[0]:o[-1]] = w.grad.numpy()
        np.testing.assert_allclose(gw, ref, rtol=1e-12, atol=1e-12)


def test_weight_grad_matrix_form_and_linearity(oracle_lib):
    rng = np.random.default_rng(22)
    for _ in range(30):
        case = tiny_case(rng, dtype="f32", weighted=True)
        G = grad_out_for(rng, case)
        gw, ab = gw_of(case, G)
        B = case["B"]
        dim_off = np.concatenate([[0], np.cumsum(case["dims"].astype(np.int64))])
        # matrix form: (G_t W_t^T)[b, r] is the gradient of every lookup of row r in bag (t, b)
        for t in range(case["T"]):
            P = G[:, dim_off[t]:dim_off[t + 1]].astype(np.float64) @ table_as_f64(case["tables"][t], "f32").T
            for b in range(B):
                k = t * B + b
                for j in range(case["offsets"][k], case["offsets"][k + 1]):
                    np.testing.assert_allclose(gw[j], P[b, case["indices"][j]], rtol=1e-12, atol=1e-12)
        assert np.all(ab >= np.abs(gw))
        # the output is linear in the weights: sum_j w_j dL/dw_j = <G, out>
        out, _ = oracle.forward(case["rows"], case["dims"], "f32", case["tables"], case["indices"],
                                case["offsets"], B, case["weights"])
        lhs = float(np.dot(case["weights"].astype(np.float64), gw))
        rhs = float((G.astype(np.float64) * out).sum())
        assert abs(lhs - rhs) <= 1e-9 * (1 + abs(rhs))


def test_weight_grad_hand_worked(oracle_lib):
    # two tables, B = 2.  Table 0 (D = 2): rows [1, 2], [3, 4], [5, 6].  Table 1 (D = 1): rows [10], [20].
    # bags: (t0, b0) = {row 2, row 0}, (t0, b1) = {}, (t1, b0) = {row 1}, (t1, b1) = {row 0, row 1}
    # G = [[1, -1, 2], [0, 3, -2]]  (columns: table 0 | table 1)
    # grad_w = <G[b, slice t], W_t[idx]>:
    #   j0 (t0 b0 row 2): 1*5 - 1*6 = -1;  j1 (t0 b0 row 0): 1*1 - 1*2 = -1
    #   j2 (t1 b0 row 1): 2*20 = 40;  j3 (t1 b1 row 0): -2*10 = -20;  j4 (t1 b1 row 1): -2*20 = -40
    tables = [np.array([[1, 2], [3, 4], [5, 6]], np.float32), np.array([[10], [20]], np.float32)]
    indices = np.array([2, 0, 1, 0, 1], np.int64)
    offsets = np.array([0, 2, 2, 3, 5], np.int64)
    G = np.array([[1, -1, 2], [0, 3, -2]], np.float32)
    gw, ab = oracle.weight_grad([3, 2], [2, 1], "f32", tables, indices, offsets, 2, G)
    np.testing.assert_array_equal(gw, [-1, -1, 40, -20, -40])
    np.testing.assert_array_equal(ab, [11, 3, 40, 20, 40])
