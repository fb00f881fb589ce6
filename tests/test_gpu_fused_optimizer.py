"""The backward's reduce phase with the optimizer step made by the same
kernels (tbe_backward_reduce_apply) against the two-pass path (tbe_backward,
then tbe_apply_gradient): tables, Adagrad state and gradient outputs bitwise
equal; and, on one case, the updated tables against the oracle's gradient
rows and optimizer step."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import workloads
from paper_2512_23236_amd import tbe
from tests.gpu_util import device, note, raw_tables
from tests.test_gpu_optimizer import REL, as_f64, ulp

pytestmark = pytest.mark.gpu


def _inputs(spec, hot_table=None):
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    if hot_table is not None:  # one row of the table takes every lookup: a long segment (pieces, combine)
        off = d["offsets"].cpu()
        d["indices"][int(off[hot_table * spec.B]):int(off[(hot_table + 1) * spec.B])] = 2
    return d


def _both(spec, d, kind, lr, eps, pooling="sum", out_dtype=torch.float32):
    plan = tbe.Plan(spec.rows, spec.dims, spec.torch_dtype, spec.B, bounds_check=True, device=device(),
                    pooling=pooling, out_dtype=out_dtype)
    w = d.get("weights") if pooling == "sum" else None
    g_out = d["grad_out"].to(out_dtype)
    status = torch.zeros(1, dtype=torch.int32, device=device())
    rng = np.random.default_rng(7)
    state0 = torch.as_tensor(rng.uniform(0, 4, int(spec.rows.sum())).astype(np.float32), device=device())
    ada = kind == tbe.ROWWISE_ADAGRAD
    # two passes
    t_a, s_a = d["tables"].clone(), state0.clone() if ada else None
    ga = tbe.backward(plan, g_out, d["indices"], d["offsets"], w, status=status)
    tbe.apply_gradient(plan, t_a, ga, kind, lr, eps, state=s_a, max_unique=d["N"])
    # fused
    t_b, s_b = d["tables"].clone(), state0.clone() if ada else None
    gb, ws = tbe.backward_index(plan, d["indices"], d["offsets"], w, status=status)
    tbe.backward_reduce_apply(plan, g_out, d["N"], ws, gb, t_b, kind, lr, eps, state=s_b, per_sample_weights=w,
                              status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    return plan, (t_a, s_a, ga), (t_b, s_b, gb), state0


@pytest.mark.parametrize("kind", [tbe.SGD, tbe.ROWWISE_ADAGRAD])
@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_fused_equals_two_passes(kind, dtype):
    spec = dataclasses.replace(workloads.small_config(5, seed=61, T=4, B=600), dtype=dtype)
    d = _inputs(spec, hot_table=1)
    _, (t_a, s_a, ga), (t_b, s_b, gb), _ = _both(spec, d, kind, lr=0.05, eps=1e-3)
    assert torch.equal(t_a, t_b)
    assert not torch.equal(t_a, d["tables"])
    if kind == tbe.ROWWISE_ADAGRAD:
        assert torch.equal(s_a, s_b)
    for x, y in zip(ga.trimmed(), gb.trimmed()):
        assert torch.equal(x, y)


@pytest.mark.parametrize("variant", ["weighted", "mean", "bf16_grad", "wide_rows"])
def test_fused_variants(variant):
    k = 4 if variant == "weighted" else 5
    spec = workloads.small_config(k, seed=62, T=3, B=500)
    pooling, out = "sum", torch.float32
    if variant == "mean":
        spec, pooling = dataclasses.replace(spec, weighted=False), "mean"
    if variant == "bf16_grad":
        out = torch.bfloat16
    if variant == "wide_rows":  # rows wider than 64 lanes of 4 columns: updated in passes
        spec = dataclasses.replace(spec, dtype="f32", dims=np.array([1536, 64, 264], np.int32))
    d = _inputs(spec, hot_table=0)
    _, (t_a, s_a, ga), (t_b, s_b, gb), _ = _both(spec, d, tbe.ROWWISE_ADAGRAD, lr=0.1, eps=1e-4, pooling=pooling,
                                                 out_dtype=out)
    assert torch.equal(t_a, t_b) and torch.equal(s_a, s_b)
    for x, y in zip(ga.trimmed(), gb.trimmed()):
        assert torch.equal(x, y)


@pytest.mark.parametrize("kind", [tbe.SGD, tbe.ROWWISE_ADAGRAD])
def test_fused_against_the_oracle(kind):
    """Updated tables against the oracle's gradient rows followed by the
    oracle's optimizer step.  The GPU gradient differs from the oracle's by at
    most 1e-5 of its sum of |terms| (the backward's bound), which moves each
    element by at most lr_eff times that; on top of that the optimizer's own
    rounding bound (one ulp plus 32 * 2^-24 of the update)."""
    spec = workloads.small_config(5, seed=63, T=3, B=400)
    d = _inputs(spec, hot_table=2)
    lr, eps = 0.05, 1e-3
    _, _, (t_b, s_b, _), state0 = _both(spec, d, kind, lr, eps)
    idx, off = d["indices"].cpu().numpy(), d["offsets"].cpu().numpy()
    seg = oracle.backward_segments(spec.rows, spec.dims, idx, off, spec.B)
    rows64, ab, _ = oracle.backward_rows(spec.rows, spec.dims, off, spec.B, d["grad_out"].cpu().numpy(), seg)
    before = [t.copy() for t in raw_tables(spec, d["tables"].cpu())]
    ref = [t.copy() for t in before]
    st_ref = state0.cpu().numpy().astype(np.float64)
    oracle.apply_gradient(spec.rows, spec.dims, spec.dtype, ref, kind, np.float32(lr), np.float32(eps),
                          st_ref if kind == tbe.ROWWISE_ADAGRAD else None, seg["grad_idx"], seg["grad_row_offsets"],
                          rows64.astype(np.float32))
    # the largest step size any row takes (Adagrad: lr / (sqrt(s) + eps) with s >= the initial state)
    s_min = float(state0.min()) if kind == tbe.ROWWISE_ADAGRAD else 0.0
    lr_eff = lr / (np.sqrt(s_min) + eps) if kind == tbe.ROWWISE_ADAGRAD else lr
    got = raw_tables(spec, t_b.cpu())
    rb = np.concatenate([[0], np.cumsum(spec.rows)])
    # per element of each listed row: the gradient's error bound, scattered to table positions
    worst = 0.0
    for t in range(spec.T):
        gw, rw, bw = as_f64(got[t], spec.dtype), as_f64(ref[t], spec.dtype), as_f64(before[t], spec.dtype)
        gbound = np.zeros_like(rw)
        sel = np.nonzero((seg["grad_idx"] >= rb[t]) & (seg["grad_idx"] < rb[t + 1]))[0]
        D = int(spec.dims[t])
        for u in sel:
            o = int(seg["grad_row_offsets"][u])
            gbound[int(seg["grad_idx"][u] - rb[t])] = 1e-5 * ab[o:o + D] * lr_eff * 1.01
        tol = 2 * ulp(rw, spec.dtype) + REL * (np.abs(rw - bw) + ulp(rw, spec.dtype)) + gbound
        if kind == tbe.ROWWISE_ADAGRAD:  # the state moved by the gradient's error too: relative 2e-5 of the update
            tol += 2e-5 * np.abs(rw - bw)
        excess = np.abs(gw - rw) - tol
        assert np.all(excess <= 0), (t, float(excess.max()))
        worst = max(worst, float((np.abs(gw - rw) / np.maximum(tol, 1e-300)).max()))
    note(f"[fused-opt] kind={kind}: worst |diff| / bound = {worst:.3f}")


def test_fused_capacity_too_small_updates_nothing():
    spec = workloads.small_config(5, seed=64, T=2, B=80)
    d = _inputs(spec)
    plan = tbe.Plan(spec.rows, spec.dims, spec.torch_dtype, spec.B, bounds_check=True, device=device())
    status = torch.zeros(1, dtype=torch.int32, device=device())
    gb, ws = tbe.backward_index(plan, d["indices"], d["offsets"], status=status)
    tables = d["tables"].clone()
    tbe.backward_reduce_apply(plan, d["grad_out"], d["N"], ws, gb, tables, tbe.SGD, 0.1, status=status,
                              grad_rows_capacity=16)
    torch.cuda.synchronize()
    assert int(status.item()) == tbe.STATUS_CAPACITY
    assert torch.equal(tables, d["tables"])


def test_fused_rejects_8bit_tables_and_missing_state():
    spec = workloads.small_config(5, seed=65, T=2, B=40)
    d = _inputs(spec)
    plan = tbe.Plan(spec.rows, spec.dims, spec.torch_dtype, spec.B, bounds_check=True, device=device())
    status = torch.zeros(1, dtype=torch.int32, device=device())
    gb, ws = tbe.backward_index(plan, d["indices"], d["offsets"], status=status)
    with pytest.raises(tbe.TBEError) as e:
        tbe.backward_reduce_apply(plan, d["grad_out"], d["N"], ws, gb, d["tables"], tbe.ROWWISE_ADAGRAD, 0.1,
                                  status=status)
    assert e.value.code == -1  # Adagrad without its state
    u8 = dataclasses.replace(spec, dtype="u8")
    uplan = tbe.Plan(u8.rows, u8.dims, u8.torch_dtype, u8.B, bounds_check=True, device=device())
    ut = workloads.gen_tables_flat(u8, device())
    with pytest.raises(tbe.TBEError) as e:
        tbe.backward_reduce_apply(uplan, d["grad_out"], d["N"], ws, gb, ut, tbe.SGD, 0.1, status=status)
    assert e.value.code == -8
    torch.cuda.synchronize()
