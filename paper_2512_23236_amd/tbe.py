"""Python binding of libtbe.so (include/tbe.h): argument marshalling only.

Torch tensors supply device memory and the current HIP stream; every step of
the lookup and of its gradient runs in the library's own kernels.  There is no
fallback: if the library is missing or was built for another ABI, loading
raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
# the in-tree build; TBE_LIBRARY names another build of the same ABI (for
# side-by-side timing of two builds)
LIB_PATH = os.environ.get("TBE_LIBRARY") or os.path.join(HERE, "libtbe.so")
ABI_VERSION = 3

F32, F16, BF16, U8_ROWWISE = 0, 1, 2, 3
# table storage type -> tbe_dtype; torch.uint8 tables are 8-bit row-wise (rows of
# D codes, an fp32 scale and bias, 8 padding bytes)
DTYPE_CODE = {torch.float32: F32, torch.float16: F16, torch.bfloat16: BF16, torch.uint8: U8_ROWWISE}
OUT_DTYPE_CODE = {torch.float32: F32, torch.float16: F16, torch.bfloat16: BF16}
POOLING_CODE = {"sum": 0, "mean": 1}
INDEX_TYPE_CODE = {torch.int64: 0, torch.int32: 1}

STATUS_INDEX_OOB, STATUS_OFFSETS, STATUS_CAPACITY = 1, 2, 4
PHASES = ("keys", "sort", "segments", "reduce", "combine")  # tbe_backward_phase order
NUM_PHASES = len(PHASES)

_lib = None


class TBEError(RuntimeError):
    def __init__(self, code: int, where: str):
        msg = _load().tbe_error_string(code).decode() if _lib is not None else str(code)
        super().__init__(f"{where}: {msg} (code {code})")
        self.code = code


class _Desc(ctypes.Structure):
    _fields_ = [
        ("num_tables", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("batch_size", ctypes.c_int64),
        ("rows", ctypes.c_void_p),
        ("dims", ctypes.c_void_p),
        ("table_offsets", ctypes.c_void_p),
        ("table_elems", ctypes.c_int64),
        ("bounds_check", ctypes.c_int32),
        ("pooling", ctypes.c_int32),
        ("index_type", ctypes.c_int32),
        ("out_dtype", ctypes.c_int32),
    ]


class _Opt(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("learning_rate", ctypes.c_float), ("eps", ctypes.c_float)]


SGD, ROWWISE_ADAGRAD = 0, 1  # tbe_optimizer_kind


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(LIB_PATH)
        P, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        lib.tbe_abi_version.restype = i32
        lib.tbe_error_string.restype = ctypes.c_char_p
        lib.tbe_error_string.argtypes = [i32]
        lib.tbe_plan_create.restype = i32
        lib.tbe_plan_create.argtypes = [ctypes.POINTER(_Desc), ctypes.POINTER(P)]
        lib.tbe_plan_destroy.restype = i32
        lib.tbe_plan_destroy.argtypes = [P]
        lib.tbe_plan_info.restype = i32
        lib.tbe_plan_info.argtypes = [P, P, P, P]
        lib.tbe_forward.restype = i32
        lib.tbe_forward.argtypes = [P, P, P, P, i64, P, P, P, P]
        lib.tbe_apply_gradient.restype = i32
        lib.tbe_apply_gradient.argtypes = [P, P, ctypes.POINTER(_Opt), P, P, P, P, P, i64, P]
        lib.tbe_map_ids.restype = i32
        lib.tbe_map_ids.argtypes = [P, i64, P, i64, P, P]
        lib.tbe_weight_grad.restype = i32
        lib.tbe_weight_grad.argtypes = [P, P, P, P, P, i64, P, P, P]
        lib.tbe_backward_workspace_bytes.restype = i32
        lib.tbe_backward_workspace_bytes.argtypes = [P, i64, P]
        lib.tbe_backward.restype = i32
        lib.tbe_backward.argtypes = [P, P, P, P, i64, P, P, ctypes.c_size_t, P, i64, P, P, P, P, P, P]
        lib.tbe_backward_timed.restype = i32
        lib.tbe_backward_timed.argtypes = [P, P, P, P, i64, P, P, ctypes.c_size_t, P, i64, P, P, P, P, P, P, P]
        lib.tbe_backward_index.restype = i32
        lib.tbe_backward_index.argtypes = [P, P, P, i64, P, P, ctypes.c_size_t, P, P, P, P, P, P, P]
        lib.tbe_backward_reduce.restype = i32
        lib.tbe_backward_reduce.argtypes = [P, P, i64, P, P, ctypes.c_size_t, P, i64, P, P, P, P]
        lib.tbe_backward_reduce_apply.restype = i32
        lib.tbe_backward_reduce_apply.argtypes = [P, P, i64, P, P, ctypes.c_size_t, P, i64, P, P, P, P,
                                                  ctypes.POINTER(_Opt), P, P, P, P]
        lib.tbe_backward_noalloc.restype = i32
        lib.tbe_backward_noalloc.argtypes = [P, P, P, P, i64, P, P, i64, P, P, P, P, P, P]
        if lib.tbe_abi_version() != ABI_VERSION:
            raise ImportError(f"libtbe ABI {lib.tbe_abi_version()} != {ABI_VERSION}")
        _lib = lib
    return _lib


def lib():
    return _load()


STATUS_NAMES = {STATUS_INDEX_OOB: "index out of range", STATUS_OFFSETS: "malformed offsets",
                STATUS_CAPACITY: "grad_rows capacity too small"}


def check_status(status: torch.Tensor) -> None:
    """Waits for the status word's stream work and raises if the device set
    any TBE_STATUS_* bit (an out-of-range index, malformed offsets, too small
    a gradient capacity)."""
    bits = int(status.item())  # synchronises with the work that wrote it
    if bits:
        names = [n for b, n in STATUS_NAMES.items() if bits & b]
        raise RuntimeError(f"device status {bits}: " + ", ".join(names))


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _check(rc: int, where: str):
    if rc != 0:
        raise TBEError(rc, where)


def _stream(dev: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)


class Plan:
    """A validated table layout with its per-table metadata on the device."""

    def __init__(self, rows: Sequence[int], dims: Sequence[int], dtype: torch.dtype, batch_size: int,
                 table_offsets: Optional[Sequence[int]] = None, table_elems: Optional[int] = None,
                 bounds_check: bool = True, device=None, pooling: str = "sum",
                 index_dtype: torch.dtype = torch.int64, out_dtype: torch.dtype = torch.float32):
        lib_ = _load()
        self.rows = np.ascontiguousarray(rows, dtype=np.int64)
        self.dims = np.ascontiguousarray(dims, dtype=np.int32)
        self.T = int(self.rows.size)
        self.B = int(batch_size)
        self.dtype = dtype
        self.pooling = pooling
        self.index_dtype = index_dtype
        self.out_dtype = out_dtype
        self.bounds_check = bool(bounds_check)
        self.table_offsets = None if table_offsets is None else np.ascontiguousarray(table_offsets, dtype=np.int64)
        if table_elems is None:
            extra = 16 if dtype == torch.uint8 else 0
            table_elems = int((self.rows * (self.dims.astype(np.int64) + extra)).sum())
        self.table_elems = int(table_elems)
        if dtype not in DTYPE_CODE or out_dtype not in OUT_DTYPE_CODE or index_dtype not in INDEX_TYPE_CODE:
            raise TBEError(-3, "Plan")
        if pooling not in POOLING_CODE:
            raise TBEError(-8, "Plan")
        d = _Desc(self.T, DTYPE_CODE[dtype], self.B, self.rows.ctypes.data, self.dims.ctypes.data,
                  None if self.table_offsets is None else self.table_offsets.ctypes.data,
                  self.table_elems, int(self.bounds_check), POOLING_CODE[pooling], INDEX_TYPE_CODE[index_dtype],
                  OUT_DTYPE_CODE[out_dtype])
        self.device = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
        self._h = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            _check(lib_.tbe_plan_create(ctypes.byref(d), ctypes.byref(self._h)), "tbe_plan_create")
        td, tr, kb = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int32()
        _check(lib_.tbe_plan_info(self._h, ctypes.byref(td), ctypes.byref(tr), ctypes.byref(kb)), "tbe_plan_info")
        self.total_dim, self.total_rows, self.key_bits = td.value, tr.value, kb.value

    @property
    def handle(self):
        return self._h

    def close(self):
        if self._h is not None and self._h.value:
            _check(_load().tbe_plan_destroy(self._h), "tbe_plan_destroy")
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _dev_tensor(t: torch.Tensor, dtype, name: str, plan: Plan):
    if t.device != plan.device:
        raise ValueError(f"{name} is on {t.device}, the plan is on {plan.device}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def forward(plan: Plan, tables: torch.Tensor, indices: torch.Tensor, offsets: torch.Tensor,
            per_sample_weights: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
            status: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Pooled lookup: returns out [B, total_dim] of the plan's out_dtype
    (written on the current stream)."""
    _dev_tensor(tables, plan.dtype, "tables", plan)
    _dev_tensor(indices, plan.index_dtype, "indices", plan)
    _dev_tensor(offsets, plan.index_dtype, "offsets", plan)
    if offsets.numel() != plan.T * plan.B + 1:
        raise ValueError(f"offsets has {offsets.numel()} entries, expected T*B+1 = {plan.T * plan.B + 1}")
    if per_sample_weights is not None:
        _dev_tensor(per_sample_weights, torch.float32, "per_sample_weights", plan)
        if per_sample_weights.numel() != indices.numel():
            raise ValueError("per_sample_weights must have one weight per index")
    if out is None:
        out = torch.empty((plan.B, plan.total_dim), dtype=plan.out_dtype, device=plan.device)
    _dev_tensor(out, plan.out_dtype, "out", plan)
    if out.numel() != plan.B * plan.total_dim:
        raise ValueError("out must be [B, total_dim]")
    if status is not None:
        _dev_tensor(status, torch.int32, "status", plan)
    rc = _load().tbe_forward(plan.handle, _ptr(tables), _ptr(indices), _ptr(offsets), indices.numel(),
                             _ptr(per_sample_weights), _ptr(out), _ptr(status), _stream(plan.device))
    _check(rc, "tbe_forward")
    return out


def apply_gradient(plan: Plan, tables: torch.Tensor, grad: "SparseGrad", kind: int, lr: float, eps: float = 0.0,
                   state: Optional[torch.Tensor] = None, max_unique: Optional[int] = None) -> None:
    """One optimizer step (SGD or row-wise Adagrad) on the rows `grad` lists,
    in place on `tables` (and `state`, fp32 [total_rows], for Adagrad)."""
    _dev_tensor(tables, plan.dtype, "tables", plan)
    for t, dt, name in ((grad.grad_idx, torch.int64, "grad_idx"), (grad.grad_row_offsets, torch.int64,
                        "grad_row_offsets"), (grad.grad_rows, torch.float32, "grad_rows"),
                        (grad.num_unique_dev, torch.int64, "num_unique")):
        _dev_tensor(t, dt, name, plan)
    if state is not None:
        _dev_tensor(state, torch.float32, "state", plan)
        if state.numel() != int(plan.rows.sum()):
            raise ValueError("state must have one entry per table row (total_rows)")
    if max_unique is None:
        max_unique = grad.grad_idx.numel()
    opt = _Opt(int(kind), float(lr), float(eps))
    rc = _load().tbe_apply_gradient(plan.handle, _ptr(tables), ctypes.byref(opt), _ptr(state), _ptr(grad.grad_idx),
                                    _ptr(grad.grad_row_offsets), _ptr(grad.grad_rows), _ptr(grad.num_unique_dev),
                                    int(max_unique), _stream(plan.device))
    _check(rc, "tbe_apply_gradient")


def map_ids(values: torch.Tensor, mapping: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """MapId preprocessing: 1-based position of each raw id in the sorted
    mapping, 0 when unknown (int64, queued on the current stream)."""
    for t, name in ((values, "values"), (mapping, "mapping")):
        if t.dtype != torch.int64 or not t.is_contiguous() or t.device.type != "cuda":
            raise TypeError(f"{name} must be a contiguous int64 device tensor")
    if mapping.device != values.device:
        raise ValueError("values and mapping must be on the same device")
    if out is None:
        out = torch.empty_like(values)
    if out.dtype != torch.int64 or out.numel() != values.numel() or out.device != values.device:
        raise ValueError("out must be int64 with one entry per value")
    rc = _load().tbe_map_ids(_ptr(values), values.numel(), _ptr(mapping), mapping.numel(), _ptr(out),
                             _stream(values.device))
    _check(rc, "tbe_map_ids")
    return out


def weight_grad(plan: Plan, tables: torch.Tensor, grad_out: torch.Tensor, indices: torch.Tensor,
                offsets: torch.Tensor, out: Optional[torch.Tensor] = None,
                status: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Gradient with respect to the per-sample weights: fp32 [N] (queued on the current stream).
    grad_out has the plan's out_dtype."""
    N = indices.numel()
    _dev_tensor(tables, plan.dtype, "tables", plan)
    _dev_tensor(grad_out, plan.out_dtype, "grad_out", plan)
    _dev_tensor(indices, plan.index_dtype, "indices", plan)
    _dev_tensor(offsets, plan.index_dtype, "offsets", plan)
    if grad_out.numel() != plan.B * plan.total_dim:
        raise ValueError("grad_out must be [B, total_dim]")
    if offsets.numel() != plan.T * plan.B + 1:
        raise ValueError("offsets must have T*B+1 entries")
    if out is None:
        out = torch.empty(N, dtype=torch.float32, device=plan.device)
    _dev_tensor(out, torch.float32, "out", plan)
    if out.numel() != N:
        raise ValueError("out must have num_indices entries")
    rc = _load().tbe_weight_grad(plan.handle, _ptr(tables), _ptr(grad_out), _ptr(indices), _ptr(offsets), N,
                                 _ptr(out), _ptr(status), _stream(plan.device))
    _check(rc, "tbe_weight_grad")
    return out


def backward_workspace_bytes(plan: Plan, num_indices: int) -> int:
    n = ctypes.c_size_t()
    _check(_load().tbe_backward_workspace_bytes(plan.handle, int(num_indices), ctypes.byref(n)),
           "tbe_backward_workspace_bytes")
    return n.value


class SparseGrad:
    """Result of backward(): the first num_unique() entries are meaningful."""

    def __init__(self, grad_rows, grad_idx, seg_offsets, grad_row_offsets, num_unique_dev):
        self.grad_rows = grad_rows
        self.grad_idx = grad_idx
        self.seg_offsets = seg_offsets
        self.grad_row_offsets = grad_row_offsets
        self.num_unique_dev = num_unique_dev

    def num_unique(self) -> int:
        return int(self.num_unique_dev.item())

    def trimmed(self):
        """Host copies trimmed to U: (grad_idx, seg_offsets, grad_row_offsets, grad_rows)."""
        U = self.num_unique()
        gro = self.grad_row_offsets[: U + 1].cpu()
        return (self.grad_idx[:U].cpu(), self.seg_offsets[: U + 1].cpu(), gro,
                self.grad_rows[: int(gro[-1])].cpu())


def _event_handles(events, n: int, where: str):
    """HIP event handles of torch events (None -> NULL)."""
    if events is None:
        return None
    if len(events) != n:
        raise ValueError(f"{where} needs {n} events")
    handles = (ctypes.c_void_p * n)()
    for i, ev in enumerate(events):
        if not ev.cuda_event:  # torch creates the HIP event on first use
            ev.record()
        handles[i] = ev.cuda_event
    return handles


def _check_backward_inputs(plan: Plan, indices, offsets, per_sample_weights):
    N = indices.numel()
    _dev_tensor(indices, plan.index_dtype, "indices", plan)
    _dev_tensor(offsets, plan.index_dtype, "offsets", plan)
    if offsets.numel() != plan.T * plan.B + 1:
        raise ValueError("offsets must have T*B+1 entries")
    if per_sample_weights is not None:
        _dev_tensor(per_sample_weights, torch.float32, "per_sample_weights", plan)
        if per_sample_weights.numel() != N:
            raise ValueError("per_sample_weights must have one weight per index")
    return N


def _check_grad_out(plan: Plan, grad_out):
    _dev_tensor(grad_out, plan.out_dtype, "grad_out", plan)  # the gradient of out has out's type
    if grad_out.numel() != plan.B * plan.total_dim:
        raise ValueError("grad_out must be [B, total_dim]")


def _new_outputs(plan: Plan, offsets, N: int, grad_rows_capacity: Optional[int]) -> "SparseGrad":
    dev = plan.device
    if grad_rows_capacity is None:
        # bound: every lookup its own row; needs the per-table lookup counts
        # (one small device-to-host copy of T+1 offsets)
        bounds = offsets[:: plan.B].cpu().numpy().astype(np.int64) if plan.B else np.zeros(plan.T + 1, np.int64)
        grad_rows_capacity = int((np.diff(bounds) * plan.dims.astype(np.int64)).sum()) if N else 0
    return SparseGrad(
        torch.empty(max(grad_rows_capacity, 1), dtype=torch.float32, device=dev),
        torch.empty(max(N, 1), dtype=torch.int64, device=dev),
        torch.empty(N + 1, dtype=torch.int64, device=dev),
        torch.empty(N + 1, dtype=torch.int64, device=dev),
        torch.zeros(1, dtype=torch.int64, device=dev))


def _check_outputs(plan: Plan, outputs: "SparseGrad", N: int, cap: Optional[int]) -> int:
    """Sizes of caller-supplied outputs against N; returns the capacity in floats."""
    for t, dt, name, need in ((outputs.grad_idx, torch.int64, "grad_idx", N),
                              (outputs.seg_offsets, torch.int64, "seg_offsets", N + 1),
                              (outputs.grad_row_offsets, torch.int64, "grad_row_offsets", N + 1),
                              (outputs.num_unique_dev, torch.int64, "num_unique", 1),
                              (outputs.grad_rows, torch.float32, "grad_rows", 0)):
        _dev_tensor(t, dt, name, plan)
        if t.numel() < need:
            raise ValueError(f"{name} holds {t.numel()} entries, needs at least {need} for {N} lookups")
    if cap is None:
        return outputs.grad_rows.numel()
    if cap < 0 or cap > outputs.grad_rows.numel():
        raise ValueError(f"grad_rows_capacity {cap} is outside grad_rows ({outputs.grad_rows.numel()} floats)")
    return int(cap)


def _workspace(plan: Plan, N: int, workspace: Optional[torch.Tensor]) -> torch.Tensor:
    need = backward_workspace_bytes(plan, N)
    if workspace is None:
        return torch.empty(max(need, 1), dtype=torch.uint8, device=plan.device)
    _dev_tensor(workspace, torch.uint8, "workspace", plan)
    return workspace  # its size is checked by the library (TBE_ERR_WORKSPACE)


def backward(plan: Plan, grad_out: torch.Tensor, indices: torch.Tensor, offsets: torch.Tensor,
             per_sample_weights: Optional[torch.Tensor] = None, grad_rows_capacity: Optional[int] = None,
             workspace: Optional[torch.Tensor] = None, status: Optional[torch.Tensor] = None,
             outputs: Optional[SparseGrad] = None,
             phase_events: Optional[Sequence[torch.cuda.Event]] = None) -> SparseGrad:
    """Sparse gradient of the tables (queued on the current stream).

    phase_events: NUM_PHASES + 1 events recorded at the phase boundaries of
    the backward (tbe_backward_timed); event i .. i+1 brackets phase i."""
    N = _check_backward_inputs(plan, indices, offsets, per_sample_weights)
    _check_grad_out(plan, grad_out)
    if outputs is None:
        outputs = _new_outputs(plan, offsets, N, grad_rows_capacity)
    cap = _check_outputs(plan, outputs, N, grad_rows_capacity)
    workspace = _workspace(plan, N, workspace)
    args = (plan.handle, _ptr(grad_out), _ptr(indices), _ptr(offsets), N, _ptr(per_sample_weights),
            _ptr(workspace), workspace.numel(), _ptr(outputs.grad_rows), cap, _ptr(outputs.grad_idx),
            _ptr(outputs.seg_offsets), _ptr(outputs.grad_row_offsets), _ptr(outputs.num_unique_dev), _ptr(status),
            _stream(plan.device))
    if phase_events is None:
        _check(_load().tbe_backward(*args), "tbe_backward")
    else:
        handles = _event_handles(phase_events, NUM_PHASES + 1, "phase_events")
        _check(_load().tbe_backward_timed(*args, handles), "tbe_backward_timed")
    return outputs


def backward_index(plan: Plan, indices: torch.Tensor, offsets: torch.Tensor,
                   per_sample_weights: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                   status: Optional[torch.Tensor] = None, outputs: Optional[SparseGrad] = None,
                   grad_rows_capacity: Optional[int] = None,
                   events: Optional[Sequence[torch.cuda.Event]] = None):
    """Index phase of the backward (tbe_backward_index), queued on the current
    stream: row ids, segment offsets, row offsets and U are final when it
    completes.  Returns (outputs, workspace) for backward_reduce.
    events: 4 events (keys, sort, segments begin; the phase ends)."""
    N = _check_backward_inputs(plan, indices, offsets, per_sample_weights)
    if outputs is None:
        outputs = _new_outputs(plan, offsets, N, grad_rows_capacity)
    _check_outputs(plan, outputs, N, grad_rows_capacity)
    workspace = _workspace(plan, N, workspace)
    rc = _load().tbe_backward_index(plan.handle, _ptr(indices), _ptr(offsets), N, _ptr(per_sample_weights),
                                    _ptr(workspace), workspace.numel(), _ptr(outputs.grad_idx),
                                    _ptr(outputs.seg_offsets), _ptr(outputs.grad_row_offsets),
                                    _ptr(outputs.num_unique_dev), _ptr(status), _stream(plan.device),
                                    _event_handles(events, 4, "events"))
    _check(rc, "tbe_backward_index")
    return outputs, workspace


def backward_reduce(plan: Plan, grad_out: torch.Tensor, num_indices: int, workspace: torch.Tensor,
                    outputs: SparseGrad, per_sample_weights: Optional[torch.Tensor] = None,
                    grad_rows_capacity: Optional[int] = None, status: Optional[torch.Tensor] = None,
                    events: Optional[Sequence[torch.cuda.Event]] = None) -> SparseGrad:
    """Reduce phase of the backward (tbe_backward_reduce), queued on the
    current stream after a backward_index of the same num_indices, workspace,
    outputs and per_sample_weights (whose values that phase already read).
    events: 3 events (reduce, combine begin; the phase ends)."""
    N = int(num_indices)
    _check_grad_out(plan, grad_out)
    if per_sample_weights is not None:
        _dev_tensor(per_sample_weights, torch.float32, "per_sample_weights", plan)
    cap = _check_outputs(plan, outputs, N, grad_rows_capacity)
    workspace = _workspace(plan, N, workspace)
    rc = _load().tbe_backward_reduce(plan.handle, _ptr(grad_out), N, _ptr(per_sample_weights), _ptr(workspace),
                                     workspace.numel(),
                                     _ptr(outputs.grad_rows), cap, _ptr(outputs.grad_row_offsets), _ptr(status),
                                     _stream(plan.device), _event_handles(events, 3, "events"))
    _check(rc, "tbe_backward_reduce")
    return outputs


def backward_reduce_apply(plan: Plan, grad_out: torch.Tensor, num_indices: int, workspace: torch.Tensor,
                          outputs: SparseGrad, tables: torch.Tensor, kind: int, lr: float, eps: float = 0.0,
                          state: Optional[torch.Tensor] = None, per_sample_weights: Optional[torch.Tensor] = None,
                          grad_rows_capacity: Optional[int] = None, status: Optional[torch.Tensor] = None,
                          events: Optional[Sequence[torch.cuda.Event]] = None) -> SparseGrad:
    """tbe_backward_reduce_apply: the reduce phase after a backward_index, with
    the optimizer step (SGD or row-wise Adagrad) made on `tables` (and
    `state`) in place by the same kernels.  The gradient rows are written too.
    events: 3 events (reduce, combine begin; the phase ends)."""
    N = int(num_indices)
    _check_grad_out(plan, grad_out)
    _dev_tensor(tables, plan.dtype, "tables", plan)
    if per_sample_weights is not None:
        _dev_tensor(per_sample_weights, torch.float32, "per_sample_weights", plan)
    if state is not None:
        _dev_tensor(state, torch.float32, "state", plan)
        if state.numel() != int(plan.rows.sum()):
            raise ValueError("state must have one entry per table row (total_rows)")
    cap = _check_outputs(plan, outputs, N, grad_rows_capacity)
    workspace = _workspace(plan, N, workspace)
    opt = _Opt(int(kind), float(lr), float(eps))
    rc = _load().tbe_backward_reduce_apply(plan.handle, _ptr(grad_out), N, _ptr(per_sample_weights),
                                           _ptr(workspace), workspace.numel(), _ptr(outputs.grad_rows), cap,
                                           _ptr(outputs.grad_idx), _ptr(outputs.seg_offsets),
                                           _ptr(outputs.grad_row_offsets), _ptr(tables), ctypes.byref(opt),
                                           _ptr(state), _ptr(status), _stream(plan.device),
                                           _event_handles(events, 3, "events"))
    _check(rc, "tbe_backward_reduce_apply")
    return outputs


NOALLOC_SCRATCH_BYTES = 64 << 20  # TBE_NOALLOC_SCRATCH_BYTES


def backward_noalloc(plan: Plan, grad_out: torch.Tensor, indices: torch.Tensor, offsets: torch.Tensor,
                     outputs: SparseGrad, per_sample_weights: Optional[torch.Tensor] = None,
                     grad_rows_capacity: Optional[int] = None, status: Optional[torch.Tensor] = None) -> SparseGrad:
    """tbe_backward_noalloc: the backward with the library's fixed device
    scratch as its workspace.  Neither this call nor the library allocates:
    the caller passes every output.  Calls that may overlap on one GPU race."""
    N = _check_backward_inputs(plan, indices, offsets, per_sample_weights)
    _check_grad_out(plan, grad_out)
    cap = _check_outputs(plan, outputs, N, grad_rows_capacity)
    rc = _load().tbe_backward_noalloc(plan.handle, _ptr(grad_out), _ptr(indices), _ptr(offsets), N,
                                      _ptr(per_sample_weights), _ptr(outputs.grad_rows), cap, _ptr(outputs.grad_idx),
                                      _ptr(outputs.seg_offsets), _ptr(outputs.grad_row_offsets),
                                      _ptr(outputs.num_unique_dev), _ptr(status), _stream(plan.device))
    _check(rc, "tbe_backward_noalloc")
    return outputs
