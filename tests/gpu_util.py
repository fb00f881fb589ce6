"""Helpers for the GPU parity tests: run the HIP path through the C ABI on
seeded inputs and compare it with the CPU oracle."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import workloads
from paper_2512_23236_amd import tbe

# Tolerances under the summation-normalised error |y - y_ref| / sum|terms|:
# 1e-5 for fp32 tables and for 8-bit row-wise tables (dequantised by one fp32
# fma, then the same fp32 accumulation), 2e-3 for fp16 / bf16 tables.
RTOL = {"f32": 1e-5, "f16": 2e-3, "bf16": 2e-3, "u8": 1e-5}
# Every forward accumulates in fp32, whatever the table type: two interleaved
# chains of at most ceil(L/2) terms per bag (L <= 200 here) bound the error by
# about (100 + 2) * 2^-24 = 6.1e-6 of sum|terms|.  Held for 16-bit tables too,
# so that accumulation in 16 bits (error near 2^-11) cannot hide under their
# 2e-3 bar.
FP32_ACC_BOUND = 2e-5


def note(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def device():
    return torch.device("cuda", 0)


def raw_tables(spec, flat_host: torch.Tensor):
    """Per-table numpy views of the flat buffer in the oracle's storage form."""
    offs = spec.table_offsets
    re = spec.row_elems
    tabs = []
    for t in range(spec.T):
        R, E = int(spec.rows[t]), int(re[t])
        v = flat_host[int(offs[t]): int(offs[t]) + R * E].view(R, E)
        tabs.append(_storage(spec, v))
    return tabs


def _storage(spec, v: torch.Tensor) -> np.ndarray:
    """A table slice as the oracle reads it: fp32 as is, 16-bit types as raw
    words, 8-bit row-wise rows as bytes."""
    if spec.dtype in ("f32", "u8"):
        return v.numpy()
    return v.view(torch.int16).numpy()


def plan_for(spec, bounds_check=True):
    return tbe.Plan(spec.rows, spec.dims, spec.torch_dtype, spec.B, bounds_check=bounds_check, device=device())


def run_forward(spec, d, bounds_check=True):
    plan = plan_for(spec, bounds_check)
    status = torch.zeros(1, dtype=torch.int32, device=device())
    out = tbe.forward(plan, d["tables"], d["indices"], d["offsets"], d.get("weights"), status=status)
    torch.cuda.synchronize()
    return out, int(status.item())


def oracle_forward_full(spec, d, pooling="sum"):
    h = {k: (v.cpu() if torch.is_tensor(v) else v) for k, v in d.items()}
    w = None if h.get("weights") is None else h["weights"].numpy()
    return oracle.forward(spec.rows, spec.dims, spec.dtype, raw_tables(spec, h["tables"]), h["indices"].numpy(),
                          h["offsets"].numpy(), spec.B, w, pooling=pooling)


def oracle_forward_bags(spec, d, bags, pooling="sum"):
    """Oracle results of selected bags k = t*B + b only, from the rows those
    bags touch (copied from the generated tables).  Returns {k: (ref, abs)}."""
    off = d["offsets"]
    bounds = off.cpu().numpy()
    res = {}
    for k in bags:
        t = int(k) // spec.B
        s, e = int(bounds[k]), int(bounds[k + 1])
        idx = d["indices"][s:e].cpu().numpy()
        uniq, inv = np.unique(idx, return_inverse=True)
        R, D, E = int(spec.rows[t]), int(spec.dims[t]), int(spec.row_elems[t])
        base = int(spec.table_offsets[t])
        full = d["tables"][base: base + R * E].view(R, E)
        rows = full[torch.as_tensor(uniq, device=full.device)].cpu() if len(uniq) else full[:0].cpu()
        tab = _storage(spec, rows)
        w = None if d.get("weights") is None else d["weights"][s:e].cpu().numpy()
        n_rows = max(len(uniq), 1)
        if len(uniq) == 0:
            tab = np.zeros((1, E), tab.dtype)
        ref, ab = oracle.forward([n_rows], [D], spec.dtype, [tab], inv.astype(np.int64), [0, e - s], 1, w,
                                 pooling=pooling)
        res[int(k)] = (ref[0], ab[0])
    return res


def forward_error(spec, out: torch.Tensor, ref, ab):
    return float(oracle.summation_error(out.cpu().numpy(), ref, ab).max())
