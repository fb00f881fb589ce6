"""The allocation-free backward (tbe_backward_noalloc, the library's fixed
device scratch as workspace) against tbe_backward with a caller workspace:
the same kernels, so every output is bitwise the same.  Two calls in a row
share the one scratch array, the second with a smaller (and weighted) input;
an input whose workspace exceeds the scratch is rejected before anything is
queued."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import workloads
from paper_2512_23236_amd import tbe
from tests.gpu_util import device, note

pytestmark = pytest.mark.gpu


def _outputs(plan, d):
    N = d["N"]
    off = d["offsets"][:: plan.B].cpu().numpy().astype(np.int64)
    cap = int((np.diff(off) * plan.dims.astype(np.int64)).sum())
    dev = device()
    return tbe.SparseGrad(torch.full((max(cap, 1),), -3.0, device=dev),
                          torch.full((max(N, 1),), -1, dtype=torch.int64, device=dev),
                          torch.full((N + 1,), -1, dtype=torch.int64, device=dev),
                          torch.full((N + 1,), -1, dtype=torch.int64, device=dev),
                          torch.zeros(1, dtype=torch.int64, device=dev))


def _case(k, seed, T, B):
    spec = workloads.small_config(k, seed=seed, T=T, B=B)
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    plan = tbe.Plan(spec.rows, spec.dims, spec.torch_dtype, spec.B, bounds_check=True, device=device())
    return spec, d, plan


def _compare(spec, d, plan):
    need = tbe.backward_workspace_bytes(plan, d["N"])
    note(f"[noalloc] {spec.name} N={d['N']} workspace {need} of {tbe.NOALLOC_SCRATCH_BYTES} bytes")
    assert need <= tbe.NOALLOC_SCRATCH_BYTES
    w = d.get("weights")
    st_a = torch.zeros(1, dtype=torch.int32, device=device())
    st_b = torch.zeros(1, dtype=torch.int32, device=device())
    ref = tbe.backward(plan, d["grad_out"], d["indices"], d["offsets"], w, status=st_a, outputs=_outputs(plan, d))
    got = tbe.backward_noalloc(plan, d["grad_out"], d["indices"], d["offsets"], _outputs(plan, d),
                               per_sample_weights=w, status=st_b)
    torch.cuda.synchronize()
    assert int(st_a.item()) == 0 and int(st_b.item()) == 0
    for x, y in zip(ref.trimmed(), got.trimmed()):
        assert torch.equal(x, y)
    # and the integer part against the oracle, as every backward is held to
    seg = oracle.backward_segments(spec.rows, spec.dims, d["indices"].cpu().numpy(), d["offsets"].cpu().numpy(),
                                   spec.B)
    gidx, segs, gro, _ = got.trimmed()
    np.testing.assert_array_equal(gidx.numpy(), seg["grad_idx"])
    np.testing.assert_array_equal(segs.numpy(), seg["seg_offsets"])
    np.testing.assert_array_equal(gro.numpy(), seg["grad_row_offsets"])


def test_noalloc_matches_backward_twice_second_smaller():
    spec, d, plan = _case(5, seed=41, T=4, B=6000)   # about 0.7 M lookups
    _compare(spec, d, plan)
    spec2, d2, plan2 = _case(4, seed=42, T=3, B=400)  # smaller, weighted
    assert d2["N"] < d["N"]
    _compare(spec2, d2, plan2)


def test_noalloc_rejects_inputs_beyond_the_scratch():
    spec = workloads.small_config(5, seed=43, T=2, B=64)
    plan = tbe.Plan(spec.rows, spec.dims, spec.torch_dtype, spec.B, bounds_check=True, device=device())
    n = 1
    while tbe.backward_workspace_bytes(plan, n) <= tbe.NOALLOC_SCRATCH_BYTES:
        n *= 2
    note(f"[noalloc] {n} lookups need {tbe.backward_workspace_bytes(plan, n)} bytes")
    lib = tbe.lib()
    rc = lib.tbe_backward_noalloc(plan.handle, None, None, None, n, None, None, 0, None, None, None, None, None,
                                  None)
    assert rc == -5  # TBE_ERR_WORKSPACE, nothing queued
