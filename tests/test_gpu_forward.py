"""Forward parity of the HIP path (through the C ABI) against the CPU oracle."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import workloads
from paper_2512_23236_amd import tbe
from tests.gpu_util import (FP32_ACC_BOUND, RTOL, device, forward_error, note, oracle_forward_bags, oracle_forward_full,
                            plan_for, run_forward)

pytestmark = pytest.mark.gpu


def _check_full(spec, d=None, bitexact=False):
    note(f"[fwd] {spec.name} T={spec.T} B={spec.B} dtype={spec.dtype} seed={spec.seed}")
    if d is None:
        d = workloads.gen_all(spec, device())
    out, st = run_forward(spec, d)
    assert st == 0, f"status {st}"
    ref, ab = oracle_forward_full(spec, d)
    if bitexact:
        np.testing.assert_array_equal(out.cpu().numpy().astype(np.float64), ref)
    err = forward_error(spec, out, ref, ab)
    note(f"[fwd] {spec.name} max summation error {err:.3g}")
    assert err <= RTOL[spec.dtype]
    assert err <= FP32_ACC_BOUND  # fp32 accumulation, also for 16-bit tables
    return out


def test_cfg1_full():
    _check_full(workloads.make_config(1))


def test_cfg2_full_bitexact():
    # one lookup per bag: the pooled row is the table row widened exactly
    _check_full(workloads.make_config(2), bitexact=True)


@pytest.mark.parametrize("k", [3, 4])
@pytest.mark.parametrize("seed", [1, 2])
def test_small_configs(k, seed):
    _check_full(workloads.small_config(k, seed=seed, T=7, B=131))


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("weighted", [False, True])
def test_dims_and_dtypes(dtype, weighted):
    """Row widths from one 16-byte vector to more than one wave (1 KiB) wide,
    including widths that are not a power of two."""
    es = 4 if dtype == "f32" else 2
    dims = [16 // es, 32 // es * 3, 64, 128, 96, 256, 512, 8 * 48 // es, 2048 // es * 3]
    base = workloads.small_config(3, seed=3, T=len(dims), B=37)
    spec = dataclasses.replace(base, dtype=dtype, dims=np.array(dims, np.int32), weighted=weighted,
                               name=f"dims-{dtype}-{'w' if weighted else 'u'}")
    _check_full(spec)


def test_long_and_empty_bags():
    spec = workloads.small_config(4, seed=5, T=3, B=64)
    d = workloads.gen_all(spec, device())
    L = torch.diff(d["offsets"]).cpu()
    L[0] = 200          # a long bag
    L[1:5] = 0          # empty bags
    L[spec.B:2 * spec.B] = 0   # a table whose bags are all empty
    L[5] = 64           # exactly one index chunk
    L[6] = 65           # one more than a chunk
    off = torch.zeros(L.numel() + 1, dtype=torch.int64)
    torch.cumsum(L, 0, out=off[1:])
    d["offsets"] = off.to(device())
    d["indices"] = workloads.gen_indices(spec, d["offsets"])
    d["weights"] = workloads.gen_weights(spec, int(off[-1]), device())
    out = _check_full(spec, d)
    o = out.cpu()
    D = int(spec.dims[0])
    assert torch.all(o[1:5, :D] == 0) and not torch.any(torch.signbit(o[1:5, :D]))
    dim_off = spec.dim_off
    assert torch.all(o[:, dim_off[1]:dim_off[2]] == 0)


@pytest.mark.parametrize("dtype,weighted", [("f32", False), ("f32", True), ("u8", False), ("u8", True),
                                            ("f16", False), ("bf16", True)])
def test_longest_bags_meet_the_fp32_bar(dtype, weighted):
    """Bags of L = 200 lookups (the longest the configurations draw) on fp32
    and 8-bit row-wise tables meet the 1e-5 bar, and 16-bit tables the fp32
    accumulation bound, at row widths from 1 to 64 lanes per row."""
    es = {"f32": 4, "f16": 2, "bf16": 2, "u8": 1}[dtype]
    dims = [16 // es, 128 // es, 64, 256, 512 // es]
    dims = [max(d, 16) if dtype == "u8" else d for d in dims]
    base = workloads.small_config(3, seed=21, T=len(dims), B=24)
    spec = dataclasses.replace(base, dtype=dtype, dims=np.array(dims, np.int32), weighted=weighted,
                               name=f"long-{dtype}-{'w' if weighted else 'u'}")
    d = workloads.gen_all(spec, device())
    L = torch.full((spec.T * spec.B,), 200, dtype=torch.int64)
    L[3::7] = 199       # odd lengths: the two chains differ by one term
    L[5::11] = 0
    off = torch.zeros(L.numel() + 1, dtype=torch.int64)
    torch.cumsum(L, 0, out=off[1:])
    d["offsets"] = off.to(device())
    d["indices"] = workloads.gen_indices(spec, d["offsets"])
    d["weights"] = workloads.gen_weights(spec, int(off[-1]), device()) if weighted else None
    d["N"] = int(off[-1])
    _check_full(spec, d)


def test_one_row_table_and_identical_indices():
    spec = workloads.small_config(3, seed=9, T=2, B=50)
    spec = dataclasses.replace(spec, rows=np.array([1, 300], np.int64))
    d = workloads.gen_all(spec, device())
    d["indices"][:] = torch.where(torch.arange(d["N"], device=device()) < int(d["offsets"][spec.B]),
                                  torch.zeros_like(d["indices"]), torch.full_like(d["indices"], 17))
    _check_full(spec, d)


def test_deterministic_repeat():
    spec = workloads.small_config(4, seed=11, T=5, B=200)
    d = workloads.gen_all(spec, device())
    a, _ = run_forward(spec, d)
    b, _ = run_forward(spec, d)
    assert torch.equal(a, b)


def test_bounds_check_flags_and_skips():
    spec = workloads.small_config(3, seed=12, T=2, B=20)
    d = workloads.gen_all(spec, device())
    bad_j = int(d["offsets"][3]) if int(d["offsets"][4]) > int(d["offsets"][3]) else 0
    good = d["indices"].clone()
    d["indices"][bad_j] = int(spec.rows[0]) + 5   # out of range for table 0
    out, st = run_forward(spec, d)
    assert st & tbe.STATUS_INDEX_OOB
    # the offending lookup contributes nothing: compare against weight 0 there
    ref_d = dict(d, indices=good, weights=torch.ones(d["N"], device=device()))
    ref_d["weights"][bad_j] = 0.0
    ref, ab = oracle_forward_full(dataclasses.replace(spec, weighted=True), ref_d)
    err = oracle.summation_error(out.cpu().numpy(), ref, ab).max()
    assert err <= RTOL[spec.dtype]
    d["indices"][bad_j] = -1
    _, st = run_forward(spec, d)
    assert st & tbe.STATUS_INDEX_OOB


def test_bounds_check_offsets():
    spec = workloads.small_config(3, seed=13, T=2, B=20)
    d = workloads.gen_all(spec, device())
    off = d["offsets"].clone()
    off[5], off[6] = off[6].item(), off[5].item()   # decreasing pair
    d2 = dict(d, offsets=off)
    _, st = run_forward(spec, d2)
    assert st & tbe.STATUS_OFFSETS
    off = d["offsets"].clone()
    off[-1] += 3                                     # last offset beyond N
    _, st = run_forward(spec, dict(d, offsets=off))
    assert st & tbe.STATUS_OFFSETS


def test_empty_batch_and_no_lookups():
    spec = workloads.small_config(3, seed=14, T=2, B=0)
    d = workloads.gen_all(spec, device())
    out, st = run_forward(spec, d)
    assert out.numel() == 0 and st == 0
    spec = dataclasses.replace(workloads.small_config(3, seed=14, T=2, B=8), empty_p=1.0)
    d = workloads.gen_all(spec, device())
    assert d["N"] == 0
    out, st = run_forward(spec, d)
    assert st == 0 and torch.all(out == 0)


def test_python_binding_validates():
    spec = workloads.small_config(1, seed=1, T=1, B=4)
    d = workloads.gen_all(spec, device())
    plan = plan_for(spec)
    with pytest.raises(TypeError):
        tbe.forward(plan, d["tables"].half(), d["indices"], d["offsets"])
    with pytest.raises(ValueError):
        tbe.forward(plan, d["tables"], d["indices"], d["offsets"][:-1])
    with pytest.raises(tbe.TBEError):
        tbe.forward(plan, d["tables"][1:], d["indices"], d["offsets"])  # 4-byte misaligned tables


@pytest.mark.slow
@pytest.mark.parametrize("k", [3, 4])
def test_full_size_sampled(k):
    """Configurations 3 and 4 at full size, in the benchmark's launch
    configuration (bounds checking on), checked on sampled bags (plus the
    longest and empty bags)."""
    spec = workloads.make_config(k)
    note(f"[fwd-full] cfg{k}: generating {spec.table_bytes / 1e9:.1f} GB of tables")
    d = workloads.gen_all(spec, device())
    out, st = run_forward(spec, d, bounds_check=True)
    assert st == 0
    L = torch.diff(d["offsets"]).cpu().numpy()
    rng = np.random.default_rng(k)
    bags = set(rng.choice(L.size, 300, replace=False).tolist())
    bags.add(int(np.argmax(L)))
    empties = np.nonzero(L == 0)[0]
    bags.update(empties[:5].tolist())
    res = oracle_forward_bags(spec, d, sorted(bags))
    o = out.cpu().numpy()
    worst = 0.0
    for kk, (ref, ab) in res.items():
        t, b = kk // spec.B, kk % spec.B
        c0, c1 = int(spec.dim_off[t]), int(spec.dim_off[t + 1])
        worst = max(worst, float(oracle.summation_error(o[b, c0:c1], ref, ab).max()))
    note(f"[fwd-full] cfg{k}: {len(res)} bags, max summation error {worst:.3g}")
    assert worst <= RTOL[spec.dtype]
    assert worst <= FP32_ACC_BOUND
    # every output element was written with a finite value
    assert np.isfinite(o).all()
    del d
    torch.cuda.empty_cache()
