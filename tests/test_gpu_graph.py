"""A training step (the forward, then the allocation-free backward) captured
in a HIP graph and replayed.  Neither entry point allocates, copies or
synchronises, so the whole step is graph nodes of the library's kernels.
Every replay must equal the eager step bitwise: three replays with eager
work and synchronisations between them, each after every output was
overwritten with junk, and one more after new values were written into the
same input buffers (the graph reads its inputs at replay)."""
import dataclasses

import numpy as np
import pytest
import torch

import workloads
from paper_2512_23236_amd import tbe
from tests.gpu_util import device, note

pytestmark = pytest.mark.gpu


def _buffers(spec, plan, d):
    dev = device()
    N = d["N"]
    off = d["offsets"][:: plan.B].cpu().numpy().astype(np.int64)
    cap = int((np.diff(off) * plan.dims.astype(np.int64)).sum())
    out = torch.empty(spec.B, plan.total_dim, dtype=torch.float32, device=dev)
    grad = tbe.SparseGrad(torch.empty(max(cap, 1), device=dev), torch.empty(max(N, 1), dtype=torch.int64, device=dev),
                          torch.empty(N + 1, dtype=torch.int64, device=dev),
                          torch.empty(N + 1, dtype=torch.int64, device=dev),
                          torch.zeros(1, dtype=torch.int64, device=dev))
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    return out, grad, status


def _step(plan, d, out, grad, status):
    w = d.get("weights")
    tbe.forward(plan, d["tables"], d["indices"], d["offsets"], w, out=out, status=status)
    tbe.backward_noalloc(plan, d["grad_out"], d["indices"], d["offsets"], grad, w, status=status)


def _junk(out, grad):
    out.fill_(float("nan"))
    grad.grad_rows.fill_(float("nan"))
    for t in (grad.grad_idx, grad.seg_offsets, grad.grad_row_offsets, grad.num_unique_dev):
        t.fill_(-7)


def _result(out, grad, status):
    """The meaningful part of every output (host copies)."""
    U = int(grad.num_unique_dev.item())
    floats = int(grad.grad_row_offsets[U].item())
    return (out.cpu(), grad.grad_idx[:U].cpu(), grad.seg_offsets[: U + 1].cpu(),
            grad.grad_row_offsets[: U + 1].cpu(), grad.grad_rows[:floats].cpu(), U, int(status.item()))


def _same(a, b):
    assert a[5] == b[5] and a[6] == b[6] == 0
    for x, y in zip(a[:5], b[:5]):
        assert torch.equal(x, y)


@pytest.mark.parametrize("k", [4, 5])
def test_captured_step_replays_equal_eager(k):
    spec = dataclasses.replace(workloads.small_config(k, seed=71 + k, T=4, B=300), grad=True)
    d = workloads.gen_all(spec, device())
    plan = tbe.Plan(spec.rows, spec.dims, spec.torch_dtype, spec.B, bounds_check=True, device=device())
    out, grad, status = _buffers(spec, plan, d)
    note(f"[graph] cfg{k}: T={spec.T} B={spec.B} N={d['N']} weighted={spec.weighted}")

    _step(plan, d, out, grad, status)
    torch.cuda.synchronize()
    eager = _result(out, grad, status)

    # warm up on a side stream, then capture on torch's capture stream
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        _step(plan, d, out, grad, status)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _step(plan, d, out, grad, status)
    torch.cuda.synchronize()

    for rep in range(3):
        _junk(out, grad)
        x = torch.randn(4096, device=device()).cumsum(0)  # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        _same(eager, _result(out, grad, status))
        assert torch.isfinite(x).all()

    # new values in the same input buffers: the replay reads them
    torch.manual_seed(k)
    d["grad_out"].copy_(torch.randn_like(d["grad_out"]))
    rows = torch.as_tensor(np.repeat(spec.rows, spec.B), device=device())
    bag = torch.repeat_interleave(torch.arange(spec.T * spec.B, device=device()),
                                  d["offsets"][1:] - d["offsets"][:-1])
    d["indices"].copy_((d["indices"] * 7 + 3) % rows[bag])
    _step(plan, d, out, grad, status)
    torch.cuda.synchronize()
    eager2 = _result(out, grad, status)
    assert not torch.equal(eager2[1], eager[1]) or not torch.equal(eager2[4], eager[4])
    _junk(out, grad)
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    _same(eager2, _result(out, grad, status))
    note(f"[graph] cfg{k}: 4 replays equal the eager step (U={eager[5]}, then {eager2[5]})")
