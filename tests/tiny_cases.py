"""Tiny random inputs for pinning the oracle (numpy only, no lookup arithmetic)
and the brute-force dense one-hot definition the oracle is checked against."""
from __future__ import annotations

import numpy as np

F16_TYPES = {"f32": np.float32, "f16": np.float16}


def tiny_case(rng: np.random.Generator, dtype: str = "f32", weighted: bool = False, max_T=4, max_R=64,
              max_B=8, max_L=12, dims=(4, 8, 16, 64), p_empty=0.2, integer_values=False):
    T = int(rng.integers(1, max_T + 1))
    B = int(rng.integers(1, max_B + 1))
    rows = rng.integers(1, max_R + 1, size=T).astype(np.int64)
    dim = rng.choice(np.array(dims), size=T).astype(np.int32)
    tables = []
    for t in range(T):
        if integer_values:
            v = rng.integers(-8, 9, size=(rows[t], dim[t])).astype(np.float32)
        else:
            v = rng.standard_normal((rows[t], dim[t])).astype(np.float32)
        if dtype == "f16":
            tables.append(v.astype(np.float16))
        elif dtype == "bf16":
            u = v.view(np.uint32)
            tables.append(((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16))
        else:
            tables.append(v)
    lengths = rng.integers(0, max_L + 1, size=T * B)
    lengths[rng.random(T * B) < p_empty] = 0
    offsets = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    idx = []
    for k in range(T * B):
        t = k // B
        idx.append(rng.integers(0, rows[t], size=lengths[k]))
    indices = np.concatenate(idx).astype(np.int64) if idx else np.zeros(0, np.int64)
    w = None
    if weighted:
        w = (rng.standard_normal(indices.size)).astype(np.float32)
    return dict(T=T, B=B, rows=rows, dims=dim, dtype=dtype, tables=tables, offsets=offsets,
                indices=indices, weights=w)


def table_as_f64(table: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return (table.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return table.astype(np.float64)


def dense_A(case, t: int) -> np.ndarray:
    """The multi-hot matrix A_t[b, r] = sum of w_j over bag (t, b)'s lookups of row r."""
    B, R = case["B"], int(case["rows"][t])
    A = np.zeros((B, R), np.float64)
    off, idx, w = case["offsets"], case["indices"], case["weights"]
    for b in range(B):
        k = t * B + b
        for j in range(off[k], off[k + 1]):
            A[b, idx[j]] += 1.0 if w is None else float(w[j])
    return A


def dense_forward(case) -> np.ndarray:
    """Brute force: concatenate A_t @ W_t over tables, in binary64."""
    return np.concatenate([dense_A(case, t) @ table_as_f64(case["tables"][t], case["dtype"])
                           for t in range(case["T"])], axis=1)


def dense_backward(case, grad_out: np.ndarray) -> dict:
    """Brute force: A_t^T @ G_t per table; returns {global row id: gradient row}."""
    dims = case["dims"].astype(np.int64)
    dim_off = np.concatenate([[0], np.cumsum(dims)])
    row_base = np.concatenate([[0], np.cumsum(case["rows"])])
    out = {}
    for t in range(case["T"]):
        A = dense_A(case, t)
        hit = np.zeros(int(case["rows"][t]), bool)
        s, e = case["offsets"][t * case["B"]], case["offsets"][(t + 1) * case["B"]]
        hit[case["indices"][s:e]] = True
        Gt = grad_out[:, dim_off[t]:dim_off[t + 1]].astype(np.float64)
        full = A.T @ Gt
        for r in np.nonzero(hit)[0]:
            out[int(row_base[t] + r)] = full[r]
    return out
