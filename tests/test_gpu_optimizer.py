"""Parity of the sparse optimizer step (HIP path through the C ABI) against
the CPU oracle, on synthetic sparse gradients drawn on the host."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import workloads
from paper_2512_23236_amd import tbe
from tests.gpu_util import device, note, plan_for, raw_tables

pytestmark = pytest.mark.gpu

# fp32 arithmetic (a fixed-order mean of squares, a division, a square root
# and one fma) against binary64: each new element may differ from the oracle's
# by one unit in the last place of its format plus 32 * 2^-24 of its update,
# and the Adagrad state by 32 * 2^-24 relative.
REL = 32 * 2.0 ** -24


def ulp(vals: np.ndarray, dtype: str) -> np.ndarray:
    a = np.abs(vals)
    if dtype == "f32":
        return np.spacing(a.astype(np.float32)).astype(np.float64)
    if dtype == "f16":
        return np.spacing(a.astype(np.float16)).astype(np.float64)
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -126)))
    return 2.0 ** (e - 7)


def as_f64(raw: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return raw.astype(np.float64)
    if dtype == "f16":
        return raw.view(np.float16).astype(np.float64)
    return (raw.astype(np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def sparse_grad(rng, spec, n_rows):
    rb = np.concatenate([[0], np.cumsum(spec.rows)])
    gidx = np.sort(rng.choice(int(rb[-1]), n_rows, replace=False)).astype(np.int64)
    t_of = np.searchsorted(rb, gidx, side="right") - 1
    gro = np.concatenate([[0], np.cumsum(spec.dims[t_of].astype(np.int64))]).astype(np.int64)
    rows = (rng.standard_normal(int(gro[-1])) * 3).astype(np.float32)
    return gidx, gro, rows


def run_case(spec, kind, lr, eps, n_rows, seed, u_dev=None):
    rng = np.random.default_rng(seed)
    d = workloads.gen_all(spec, device())
    plan = plan_for(spec)
    gidx, gro, rows = sparse_grad(rng, spec, n_rows)
    U = n_rows if u_dev is None else u_dev
    g = tbe.SparseGrad(torch.as_tensor(rows, device=device()), torch.as_tensor(gidx, device=device()),
                       torch.zeros(n_rows + 1, dtype=torch.int64, device=device()),
                       torch.as_tensor(gro, device=device()), torch.tensor([U], dtype=torch.int64, device=device()))
    total_rows = int(spec.rows.sum())
    state0 = rng.uniform(0, 4, total_rows).astype(np.float32)
    state = torch.as_tensor(state0, device=device()) if kind == tbe.ROWWISE_ADAGRAD else None
    before = [t.copy() for t in raw_tables(spec, d["tables"].cpu())]
    tables = d["tables"].clone()
    tbe.apply_gradient(plan, tables, g, kind, lr, eps, state=state)
    torch.cuda.synchronize()
    got = raw_tables(spec, tables.cpu())
    ref = [t.copy() for t in before]
    st_ref = state0.astype(np.float64)
    oracle.apply_gradient(spec.rows, spec.dims, spec.dtype, ref, kind, np.float32(lr), np.float32(eps),
                          st_ref if kind == tbe.ROWWISE_ADAGRAD else None, gidx[:U], gro[:U + 1], rows)
    worst = 0.0
    for t in range(spec.T):
        gw, rw, bw = as_f64(got[t], spec.dtype), as_f64(ref[t], spec.dtype), as_f64(before[t], spec.dtype)
        tol = ulp(rw, spec.dtype) + REL * (np.abs(rw - bw) + ulp(rw, spec.dtype))
        excess = np.abs(gw - rw) - tol
        assert np.all(excess <= 0), (t, float(excess.max()))
        unchanged = np.all(ref[t] == before[t], axis=1)
        assert np.array_equal(got[t][unchanged], before[t][unchanged])  # untouched rows: bit for bit
        worst = max(worst, float((np.abs(gw - rw) / np.maximum(ulp(rw, spec.dtype), 1e-300)).max()))
    if kind == tbe.ROWWISE_ADAGRAD:
        np.testing.assert_allclose(state.cpu().numpy(), st_ref, rtol=REL)
    note(f"[opt] {spec.name} kind={kind} rows={n_rows} U={U}: max |diff| = {worst:.2f} ulp")


@pytest.mark.parametrize("k", [1, 3, 4])
@pytest.mark.parametrize("kind", [0, 1])
def test_small_configs(k, kind):
    spec = workloads.small_config(k, seed=21, T=4, B=8)
    run_case(spec, kind, lr=0.05, eps=1e-3, n_rows=min(500, int(spec.rows.sum()) // 2), seed=k + 10 * kind)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_dims_and_dtypes(dtype):
    dims = [8, 64, 96, 128, 256, 1536]
    base = workloads.small_config(3, seed=22, T=len(dims), B=4)
    spec = dataclasses.replace(base, dtype=dtype, dims=np.array(dims, np.int32), name=f"opt-{dtype}")
    run_case(spec, tbe.ROWWISE_ADAGRAD, lr=0.5, eps=1e-6, n_rows=300, seed=3)


def test_only_the_first_num_unique_rows():
    spec = workloads.small_config(3, seed=23, T=3, B=4)
    run_case(spec, tbe.SGD, lr=0.1, eps=0.0, n_rows=200, seed=4, u_dev=120)


def test_zero_learning_rate_changes_nothing():
    spec = workloads.small_config(4, seed=24, T=2, B=4)
    d = workloads.gen_all(spec, device())
    plan = plan_for(spec)
    rng = np.random.default_rng(5)
    gidx, gro, rows = sparse_grad(rng, spec, 100)
    g = tbe.SparseGrad(torch.as_tensor(rows, device=device()), torch.as_tensor(gidx, device=device()),
                       torch.zeros(101, dtype=torch.int64, device=device()), torch.as_tensor(gro, device=device()),
                       torch.tensor([100], dtype=torch.int64, device=device()))
    tables = d["tables"].clone()
    tbe.apply_gradient(plan, tables, g, tbe.SGD, 0.0)
    torch.cuda.synchronize()
    assert torch.equal(tables, d["tables"])


def test_after_backward():
    """The step consumes tbe_backward's outputs directly (SparseGrad as written)."""
    spec = dataclasses.replace(workloads.small_config(5, seed=25, T=3, B=200), grad=True)
    d = workloads.gen_all(spec, device())
    plan = plan_for(spec)
    status = torch.zeros(1, dtype=torch.int32, device=device())
    g = tbe.backward(plan, d["grad_out"], d["indices"], d["offsets"], status=status)
    tables = d["tables"].clone()
    tbe.apply_gradient(plan, tables, g, tbe.SGD, 0.01)
    torch.cuda.synchronize()
    U = g.num_unique()
    gidx = g.grad_idx[:U].cpu().numpy()
    rb = np.concatenate([[0], np.cumsum(spec.rows)])
    changed = np.zeros(int(rb[-1]), bool)
    after, before = raw_tables(spec, tables.cpu()), raw_tables(spec, d["tables"].cpu())
    for t in range(spec.T):
        changed[rb[t]:rb[t + 1]] = np.any(after[t] != before[t], axis=1)
    assert int(status.item()) == 0
    assert not changed[np.setdiff1d(np.arange(rb[-1]), gidx)].any()  # only listed rows move


def test_ids_outside_the_plan_are_skipped():
    """Ids past the plan's rows change nothing; the valid ids around them are
    updated as usual."""
    spec = workloads.small_config(4, seed=26, T=3, B=4)
    d = workloads.gen_all(spec, device())
    plan = plan_for(spec)
    rng = np.random.default_rng(6)
    gidx, gro, rows = sparse_grad(rng, spec, 150)
    total = int(spec.rows.sum())
    bad = gidx.copy()
    bad[-3:] = total + np.arange(3)  # still ascending
    g = tbe.SparseGrad(torch.as_tensor(rows, device=device()), torch.as_tensor(bad, device=device()),
                       torch.zeros(151, dtype=torch.int64, device=device()), torch.as_tensor(gro, device=device()),
                       torch.tensor([150], dtype=torch.int64, device=device()))
    ref_g = tbe.SparseGrad(torch.as_tensor(rows, device=device()), torch.as_tensor(gidx[:-3], device=device()),
                           torch.zeros(148, dtype=torch.int64, device=device()),
                           torch.as_tensor(gro[:-3], device=device()),
                           torch.tensor([147], dtype=torch.int64, device=device()))
    a, b = d["tables"].clone(), d["tables"].clone()
    tbe.apply_gradient(plan, a, g, tbe.SGD, 0.1)
    tbe.apply_gradient(plan, b, ref_g, tbe.SGD, 0.1)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    assert not torch.equal(a, d["tables"])
