"""CPU oracle (fp64) for the pooled embedding-bag lookup and its sparse gradient.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the GPU product path.  The arithmetic
lives in ``tbe_oracle.c`` (plain C, binary64); this module only marshals
numpy arrays into it through ctypes.  See ``tbe_oracle.c`` for the definition
that is computed and for what pins it.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

from .build import LIB_PATH, build

F32, F16, BF16, U8_ROWWISE = 0, 1, 2, 3
DTYPE_CODES = {"f32": F32, "f16": F16, "bf16": BF16, "u8": U8_ROWWISE}
POOLING_CODES = {"sum": 0, "mean": 1}

_lib = None


class OracleError(RuntimeError):
    pass


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        lib = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        i32, i64 = ctypes.c_int32, ctypes.c_int64
        lib.oracle_forward.restype = ctypes.c_int
        lib.oracle_forward.argtypes = [i32, i64, P, P, i32, P, P, P, i64, P, i32, P, P]
        lib.oracle_encode.restype = ctypes.c_int
        lib.oracle_encode.argtypes = [ctypes.c_double, i32, P]
        lib.oracle_apply_gradient.restype = ctypes.c_int
        lib.oracle_apply_gradient.argtypes = [i32, P, P, i32, P, i32, ctypes.c_double, ctypes.c_double, P, P, P, P,
                                              i64]
        lib.oracle_map_ids.restype = ctypes.c_int
        lib.oracle_map_ids.argtypes = [P, i64, P, i64, P]
        lib.oracle_weight_grad.restype = ctypes.c_int
        lib.oracle_weight_grad.argtypes = [i32, i64, P, P, i32, P, P, P, i64, P, P, P]
        lib.oracle_backward_segments.restype = ctypes.c_int
        lib.oracle_backward_segments.argtypes = [i32, i64, P, P, P, P, i64, P, P, P, P, P, P]
        lib.oracle_backward_rows.restype = ctypes.c_int
        lib.oracle_backward_rows.argtypes = [i32, i64, P, P, P, P, P, P, P, P, i64, P, i32, P, P]
        lib.oracle_decode.restype = ctypes.c_double
        lib.oracle_decode.argtypes = [P, i32, i64]
        lib.oracle_decode_row.restype = ctypes.c_double
        lib.oracle_decode_row.argtypes = [P, i32, i64, i64, i64]
        _lib = lib
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _c(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a), dtype=dtype)


def _raw16(t: np.ndarray) -> np.ndarray:
    """Table storage as 16-bit words (fp16 / bf16 payloads)."""
    return np.ascontiguousarray(t).view(np.uint16)


def decode(words: np.ndarray, dtype: str) -> np.ndarray:
    """Decode stored elements to float64 with the oracle's own format decoder."""
    lib = _load()
    w = np.ascontiguousarray(words)
    return np.array([lib.oracle_decode(_p(w), DTYPE_CODES[dtype], i) for i in range(w.size)])


def decode_row(table: np.ndarray, dtype: str, D: int, r: int, d: int) -> float:
    """Element (r, d) of a table with rows of D values, decoded by the oracle
    (for "u8", rows of D codes, an fp32 scale and bias, 8 padding bytes)."""
    t = np.ascontiguousarray(table)
    return _load().oracle_decode_row(_p(t), DTYPE_CODES[dtype], D, r, d)


def forward(rows: Sequence[int], dims: Sequence[int], dtype: str, tables: Sequence[np.ndarray],
            indices, offsets, B: int, weights=None, pooling: str = "sum"):
    """Pooled lookup in binary64.

    tables[t] is table t as a [R_t, D_t] array of raw element storage: float32
    for "f32", and 16-bit words (uint16 / float16 / any 2-byte dtype, read as
    the raw bit pattern) for "f16" and "bf16"; for "u8" an [R_t, D_t + 16]
    uint8 array (each row's D_t codes, its fp32 scale and bias, 8 bytes of
    padding).
    Indices and offsets of any integer type are taken as int64 values.
    pooling is "sum" or "mean" (mean takes no weights).  Returns (out,
    absout), each [B, total_dim] float64.
    """
    lib = _load()
    T = len(rows)
    rows_a, dims_a = _c(rows, np.int64), _c(dims, np.int32)
    tabs = [np.ascontiguousarray(t) for t in tables]
    ptrs = (ctypes.c_void_p * T)(*[t.ctypes.data for t in tabs])
    idx, off = _c(indices, np.int64), _c(offsets, np.int64)
    w = None if weights is None else _c(weights, np.float32)
    total_dim = int(dims_a.astype(np.int64).sum())
    out = np.zeros((B, total_dim), np.float64)
    absout = np.zeros((B, total_dim), np.float64)
    rc = lib.oracle_forward(T, B, _p(rows_a), _p(dims_a), DTYPE_CODES[dtype], ptrs, _p(idx), _p(off),
                            idx.size, _p(w), POOLING_CODES[pooling], _p(out), _p(absout))
    if rc != 0:
        raise OracleError(f"oracle_forward returned {rc}")
    return out, absout


def weight_grad(rows: Sequence[int], dims: Sequence[int], dtype: str, tables: Sequence[np.ndarray],
                indices, offsets, B: int, grad_out):
    """Gradient of the pooled output with respect to the per-sample weights,
    in binary64: grad_w[j] = <grad_out[b(j), slice of t(j)], W_t[idx_j]>.
    Tables as in forward(); grad_out is float32 [B, total_dim].  Returns
    (grad_w, abs_terms), each [N] float64."""
    lib = _load()
    T = len(rows)
    rows_a, dims_a = _c(rows, np.int64), _c(dims, np.int32)
    tabs = [np.ascontiguousarray(t) for t in tables]
    ptrs = (ctypes.c_void_p * T)(*[t.ctypes.data for t in tabs])
    idx, off = _c(indices, np.int64), _c(offsets, np.int64)
    g = _c(grad_out, np.float32)
    gw = np.zeros(idx.size, np.float64)
    ab = np.zeros(idx.size, np.float64)
    rc = lib.oracle_weight_grad(T, B, _p(rows_a), _p(dims_a), DTYPE_CODES[dtype], ptrs, _p(idx), _p(off),
                                idx.size, _p(g), _p(gw), _p(ab))
    if rc != 0:
        raise OracleError(f"oracle_weight_grad returned {rc}")
    return gw, ab


SGD, ROWWISE_ADAGRAD = 0, 1


def encode(value: float, dtype: str) -> int:
    """The oracle's rounding of one binary64 value to the table format, as the
    stored bit pattern (uint32 for f32, uint16 otherwise)."""
    out = np.zeros(1, np.uint32 if dtype == "f32" else np.uint16)
    rc = _load().oracle_encode(float(value), DTYPE_CODES[dtype], _p(out))
    if rc != 0:
        raise OracleError(f"oracle_encode returned {rc}")
    return int(out[0])


def apply_gradient(rows, dims, dtype: str, tables, kind: int, lr: float, eps: float, state, grad_idx,
                   grad_row_offsets, grad_rows):
    """One optimizer step (SGD or row-wise Adagrad) on the listed rows, in
    binary64 with one rounding per stored element.  Updates `tables` (raw
    storage arrays, as in forward()) and `state` (float64 [sum R], Adagrad
    only) in place."""
    lib = _load()
    T = len(rows)
    rows_a, dims_a = _c(rows, np.int64), _c(dims, np.int32)
    for t in tables:
        if not (t.flags.c_contiguous and t.flags.writeable):
            raise ValueError("tables must be writeable contiguous arrays")
    ptrs = (ctypes.c_void_p * T)(*[t.ctypes.data for t in tables])
    gidx, gro = _c(grad_idx, np.int64), _c(grad_row_offsets, np.int64)
    gr = _c(grad_rows, np.float32)
    st = None
    if state is not None:
        if state.dtype != np.float64 or not state.flags.c_contiguous:
            raise ValueError("state must be contiguous float64")
        st = state
    rc = lib.oracle_apply_gradient(T, _p(rows_a), _p(dims_a), DTYPE_CODES[dtype], ptrs, kind, float(lr), float(eps),
                                   _p(st), _p(gidx), _p(gro), _p(gr), gidx.size)
    if rc != 0:
        raise OracleError(f"oracle_apply_gradient returned {rc}")


def map_ids(values, mapping) -> np.ndarray:
    """MapId preprocessing: 1-based position of each value in the sorted
    mapping, 0 for an unknown value (int64 [n])."""
    lib = _load()
    v, mp = _c(values, np.int64), _c(mapping, np.int64)
    out = np.empty(v.size, np.int64)
    rc = lib.oracle_map_ids(_p(v), v.size, _p(mp), mp.size, _p(out))
    if rc != 0:
        raise OracleError(f"oracle_map_ids returned {rc}")
    return out


def backward_segments(rows, dims, indices, offsets, B: int):
    """Integer part of the sparse gradient.

    Returns a dict with perm, sorted_keys, grad_idx, seg_offsets and
    grad_row_offsets (trimmed to U and U+1 entries) and U.
    """
    lib = _load()
    T = len(rows)
    rows_a, dims_a = _c(rows, np.int64), _c(dims, np.int32)
    idx, off = _c(indices, np.int64), _c(offsets, np.int64)
    N = idx.size
    perm = np.empty(max(N, 1), np.int64)
    keys = np.empty(max(N, 1), np.int64)
    gidx = np.empty(max(N, 1), np.int64)
    seg = np.empty(N + 1, np.int64)
    gro = np.empty(N + 1, np.int64)
    U = np.zeros(1, np.int64)
    rc = lib.oracle_backward_segments(T, B, _p(rows_a), _p(dims_a), _p(idx), _p(off), N, _p(perm),
                                      _p(keys), _p(gidx), _p(seg), _p(gro), _p(U))
    if rc != 0:
        raise OracleError(f"oracle_backward_segments returned {rc}")
    u = int(U[0])
    return {"perm": perm[:N], "sorted_keys": keys[:N], "grad_idx": gidx[:u],
            "seg_offsets": seg[: u + 1], "grad_row_offsets": gro[: u + 1], "U": u}


def backward_rows(rows, dims, offsets, B: int, grad_out, seg: dict, weights=None, sel=None,
                  pooling: str = "sum"):
    """Gradient rows (binary64) of the selected unique ids (default: all),
    for sum or mean pooling (mean takes no weights).

    Returns (rows_packed, abs_packed, row_offsets) where row s of the
    selection occupies rows_packed[row_offsets[s]:row_offsets[s+1]].
    """
    lib = _load()
    T = len(rows)
    rows_a, dims_a = _c(rows, np.int64), _c(dims, np.int32)
    off = _c(offsets, np.int64)
    g = _c(grad_out, np.float32)
    w = None if weights is None else _c(weights, np.float32)
    gidx = _c(seg["grad_idx"], np.int64)
    if sel is None:
        sel_a, n_sel = None, int(seg["U"])
        lens = np.diff(seg["grad_row_offsets"])
    else:
        sel_a = _c(sel, np.int64)
        n_sel = sel_a.size
        lens = np.diff(seg["grad_row_offsets"])[sel_a]
    ro = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    total = int(ro[-1])
    out = np.zeros(max(total, 1), np.float64)
    absout = np.zeros(max(total, 1), np.float64)
    rc = lib.oracle_backward_rows(T, B, _p(rows_a), _p(dims_a), _p(off), _p(w), _p(g),
                                  _p(_c(seg["perm"], np.int64)), _p(gidx), _p(_c(seg["seg_offsets"], np.int64)),
                                  n_sel, _p(sel_a), POOLING_CODES[pooling], _p(out), _p(absout))
    if rc != 0:
        raise OracleError(f"oracle_backward_rows returned {rc}")
    return out[:total], absout[:total], ro


def summation_error(y, y_ref, abs_ref) -> np.ndarray:
    """|y - y_ref| / sum|terms| elementwise, with 0/0 taken as 0.

    The scale is the sum of the absolute values of the summed terms, the
    backward-error scale for floating-point summation; a plain relative error
    is unbounded where the terms cancel.
    """
    y = np.asarray(y, np.float64)
    diff = np.abs(y - y_ref)
    with np.errstate(divide="ignore", invalid="ignore"):
        e = np.where(abs_ref > 0, diff / np.where(abs_ref > 0, abs_ref, 1.0), np.where(diff > 0, np.inf, 0.0))
    return e
