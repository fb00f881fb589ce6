"""Parity of the per-sample-weight gradient (HIP path through the C ABI)
against the CPU oracle."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import workloads
from paper_2512_23236_amd import tbe
from tests.gpu_util import device, note, plan_for, raw_tables

pytestmark = pytest.mark.gpu

# fp32 arithmetic on exactly widened table elements, one short fixed-order sum
# per lookup (at most 8 terms per lane, then a tree over <= 64 lanes)
RTOL_W = 1e-5


def run_wg(spec, d, bounds_check=True):
    plan = plan_for(spec, bounds_check)
    status = torch.zeros(1, dtype=torch.int32, device=device())
    gw = tbe.weight_grad(plan, d["tables"], d["grad_out"], d["indices"], d["offsets"], status=status)
    torch.cuda.synchronize()
    return gw, int(status.item())


def oracle_wg(spec, d):
    h = {k: (v.cpu() if torch.is_tensor(v) else v) for k, v in d.items()}
    return oracle.weight_grad(spec.rows, spec.dims, spec.dtype, raw_tables(spec, h["tables"]),
                              h["indices"].numpy(), h["offsets"].numpy(), spec.B, h["grad_out"].numpy())


def check(spec, d=None):
    note(f"[wgrad] {spec.name} T={spec.T} B={spec.B} dtype={spec.dtype} dims={list(spec.dims)[:6]}")
    if d is None:
        d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    gw, st = run_wg(spec, d)
    assert st == 0, f"status {st}"
    ref, ab = oracle_wg(spec, d)
    err = float(oracle.summation_error(gw.cpu().numpy(), ref, ab).max()) if ref.size else 0.0
    note(f"[wgrad] {spec.name}: N={d['N']} max summation error {err:.3g}")
    assert err <= RTOL_W
    return gw, d


@pytest.mark.parametrize("k", [1, 3, 4])
@pytest.mark.parametrize("seed", [1, 2])
def test_small_configs(k, seed):
    check(workloads.small_config(k, seed=seed, T=5, B=97))


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_dims_and_dtypes(dtype):
    """Row widths from one 16-byte vector to several 64-lane chunks, including
    widths that are not a power of two."""
    es = 4 if dtype == "f32" else 2
    dims = [16 // es, 32 // es * 3, 64, 128, 96, 256, 512, 8 * 48 // es, 2048 // es * 3]
    base = workloads.small_config(4, seed=3, T=len(dims), B=37)
    check(dataclasses.replace(base, dtype=dtype, dims=np.array(dims, np.int32), name=f"wgrad-dims-{dtype}"))


def test_long_and_empty_bags():
    """Bags longer than the 64 indices one load covers, and empty bags."""
    spec = workloads.small_config(4, seed=5, T=3, B=64)
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    lens = np.resize([0, 1, 63, 64, 65, 200, 0, 130], spec.T * spec.B)
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    N = int(off[-1])
    rng = np.random.default_rng(5)
    idx = np.concatenate([rng.integers(0, spec.rows[k // spec.B], size=lens[k]) for k in range(spec.T * spec.B)])
    d = dict(d, offsets=torch.as_tensor(off, device=device()), indices=torch.as_tensor(idx, device=device()), N=N)
    check(spec, d)


def test_bounds_check_zeroes_bad_lookups():
    spec = workloads.small_config(4, seed=9, T=3, B=60)
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    N = d["N"]
    bad = [1, N // 2, N - 1]
    good = d["indices"].clone()
    d["indices"][torch.tensor(bad, device=device())] = torch.tensor([-1, 10 ** 9, int(spec.rows.max()) + 1],
                                                                     device=device())
    gw, st = run_wg(spec, d)
    assert st & tbe.STATUS_INDEX_OOB
    ref, ab = oracle_wg(spec, dict(d, indices=good))
    got = gw.cpu().numpy()
    assert np.all(got[bad] == 0)
    keep = np.ones(N, bool)
    keep[bad] = False
    assert float(oracle.summation_error(got[keep], ref[keep], ab[keep]).max()) <= RTOL_W


def test_bounds_check_flags_bad_offsets():
    """Malformed offsets under the bounds check (a bag ending past N, a bag
    ending before it starts): the offsets bit is set and every access stays
    inside the inputs (the weight gradients are then unspecified)."""
    spec = workloads.small_config(4, seed=11, T=2, B=40)
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    N = d["N"]
    off = d["offsets"].cpu().numpy().copy()
    off[5] = N + 7            # bag 4 ends past N
    off[13] = off[12] - 1     # bag 12 ends before it starts
    d["offsets"] = torch.as_tensor(off, device=device())
    _, st = run_wg(spec, d)
    assert st & tbe.STATUS_OFFSETS


def test_deterministic_repeat():
    spec = workloads.small_config(3, seed=8, T=4, B=200)
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    a, _ = run_wg(spec, d)
    b, _ = run_wg(spec, d)
    assert torch.equal(a, b)


def test_rejects_bad_arguments():
    spec = workloads.small_config(4, seed=10, T=2, B=8)
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    plan = plan_for(spec)
    with pytest.raises(ValueError):
        tbe.weight_grad(plan, d["tables"], d["grad_out"][:-1], d["indices"], d["offsets"])
    with pytest.raises(TypeError):
        tbe.weight_grad(plan, d["tables"], d["grad_out"].double(), d["indices"], d["offsets"])


@pytest.mark.slow
def test_full_size_cfg4_sampled():
    """Configuration 4 at full size (40 bf16 tables of 5e6 x 128, B = 32768,
    weighted): every lookup of 3000 sampled bags against the oracle."""
    spec = dataclasses.replace(workloads.make_config(4), grad=True)
    note(f"[wgrad-full] cfg4: generating inputs ({spec.table_bytes / 1e9:.1f} GB tables)")
    d = workloads.gen_all(spec, device())
    gw, st = run_wg(spec, d)
    assert st == 0
    rng = np.random.default_rng(4)
    bags = np.unique(rng.integers(0, spec.T * spec.B, size=3000))
    off = d["offsets"].cpu().numpy()
    dim_off = np.concatenate([[0], np.cumsum(spec.dims.astype(np.int64))])
    worst = 0.0
    got_all = gw.cpu().numpy()
    for k in bags:
        t, b = int(k) // spec.B, int(k) % spec.B
        s, e = int(off[k]), int(off[k + 1])
        if e == s:
            continue
        idx = d["indices"][s:e].cpu().numpy()
        uniq, inv = np.unique(idx, return_inverse=True)
        R, D = int(spec.rows[t]), int(spec.dims[t])
        base = int(spec.table_offsets[t])
        rows = d["tables"][base: base + R * D].view(R, D)[torch.as_tensor(uniq, device=device())].cpu()
        G = d["grad_out"].view(spec.B, -1)[b, dim_off[t]:dim_off[t + 1]].cpu().numpy()[None, :]
        ref, ab = oracle.weight_grad([len(uniq)], [D], spec.dtype, [rows.view(torch.int16).numpy()],
                                     inv.astype(np.int64), [0, e - s], 1, G)
        worst = max(worst, float(oracle.summation_error(got_all[s:e], ref, ab).max()))
    note(f"[wgrad-full] {len(bags)} bags, max summation error {worst:.3g}")
    assert worst <= RTOL_W
