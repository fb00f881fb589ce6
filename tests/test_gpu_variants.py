"""Parity of the variants through the C ABI: mean pooling, int32 indices and
offsets, fp16 / bf16 output, and 8-bit row-wise tables, alone and combined,
against the CPU oracle (and, where the arithmetic is the same, bit for bit
against the default path)."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import workloads
from paper_2512_23236_amd import tbe
from tests.gpu_util import RTOL, device, note, oracle_forward_bags, oracle_forward_full, raw_tables

pytestmark = pytest.mark.gpu

GRAD_RTOL = 1e-5
OUT_TORCH = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
# half an ulp of the output format, relative: the rounding of the fp32 result
OUT_HALF_ULP = {"f32": 0.0, "f16": 2.0 ** -11, "bf16": 2.0 ** -8}


def make_plan(spec, pooling="sum", index="i64", out="f32", bounds_check=True):
    return tbe.Plan(spec.rows, spec.dims, spec.torch_dtype, spec.B, bounds_check=bounds_check, device=device(),
                    pooling=pooling, index_dtype=torch.int32 if index == "i32" else torch.int64,
                    out_dtype=OUT_TORCH[out])


def inputs(spec, index="i64"):
    d = workloads.gen_all(spec, device())
    if index == "i32":
        d["indices"] = d["indices"].to(torch.int32)
        d["offsets"] = d["offsets"].to(torch.int32)
    return d


def forward(spec, d, **kw):
    plan = make_plan(spec, **kw)
    st = torch.zeros(1, dtype=torch.int32, device=device())
    out = tbe.forward(plan, d["tables"], d["indices"], d["offsets"], d.get("weights"), status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    return out


def check_forward(spec, d, out, pooling, out_dt):
    ref, ab = oracle_forward_full(spec, d, pooling=pooling)
    y = out.float().cpu().numpy().astype(np.float64)
    # the fp32 result is within RTOL * sum|terms| of the oracle; the stored
    # value adds at most half an ulp of the output format (plus fp16's
    # subnormal spacing)
    bound = RTOL[spec.dtype] * ab + OUT_HALF_ULP[out_dt] * np.abs(ref) + (2.0 ** -25 if out_dt == "f16" else 0.0)
    excess = np.abs(y - ref) - bound
    note(f"[var] {spec.name} {spec.dtype} pooling={pooling} out={out_dt}: max excess {excess.max():.3g}")
    assert excess.max() <= 0


def small(k=3, seed=1, T=5, B=97, **kw):
    return dataclasses.replace(workloads.small_config(k, seed=seed, T=T, B=B), **kw)


# ------------------------------------------------------------------ forward


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16", "u8"])
def test_mean_forward(dtype):
    spec = small(dtype=dtype, name=f"mean-{dtype}")
    d = inputs(spec)
    check_forward(spec, d, forward(spec, d, pooling="mean"), "mean", "f32")


@pytest.mark.parametrize("weighted", [False, True])
@pytest.mark.parametrize("k", [3, 4])
def test_int32_forward_equals_int64(k, weighted):
    spec = small(k=k, seed=2, weighted=weighted, name=f"i32-cfg{k}")
    d64 = inputs(spec)
    d32 = dict(d64, indices=d64["indices"].to(torch.int32), offsets=d64["offsets"].to(torch.int32))
    a = forward(spec, d64)
    b = forward(spec, d32, index="i32")
    assert torch.equal(a, b)  # the same arithmetic in the same order
    check_forward(spec, d64, b, "sum", "f32")


@pytest.mark.parametrize("out_dt", ["f16", "bf16"])
@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16", "u8"])
def test_reduced_precision_output(dtype, out_dt):
    spec = small(seed=3, dtype=dtype, name=f"out-{out_dt}")
    d = inputs(spec)
    ref32 = forward(spec, d)
    out = forward(spec, d, out=out_dt)
    assert out.dtype == OUT_TORCH[out_dt]
    # the stored value is the fp32 result rounded to nearest even
    assert torch.equal(out, ref32.to(OUT_TORCH[out_dt]))
    check_forward(spec, d, out, "sum", out_dt)


@pytest.mark.parametrize("weighted", [False, True])
def test_u8_rowwise_dims(weighted):
    """8-bit rows from one 16-byte vector of codes to more than one wave of
    vectors (1040 codes: 65 vectors); rows of D + 8 bytes start 8-byte aligned."""
    dims = [16, 48, 64, 128, 96, 256, 528, 1040]
    spec = small(T=len(dims), B=41, dtype="u8", dims=np.array(dims, np.int32), weighted=weighted,
                 name=f"u8-dims-{'w' if weighted else 'u'}")
    d = inputs(spec)
    check_forward(spec, d, forward(spec, d), "sum", "f32")


def test_all_options_together():
    spec = small(k=3, seed=5, T=6, B=211, dtype="u8", name="u8-mean-i32-bf16")
    d = inputs(spec, "i32")
    check_forward(spec, d, forward(spec, d, pooling="mean", index="i32", out="bf16"), "mean", "bf16")


def test_mean_counts_dropped_lookups():
    """With bounds checking a bad lookup adds nothing but is still one of the
    bag's L lookups: the mean is (sum of the good rows) / L."""
    spec = small(seed=6, dtype="f32", name="mean-oob")
    d = inputs(spec)
    off = d["offsets"].cpu().numpy()
    k = int(np.nonzero(np.diff(off) >= 2)[0][0])
    t, b = divmod(k, spec.B)
    s, e = int(off[k]), int(off[k + 1])
    bad = d["indices"].clone()
    bad[s] = int(spec.rows[t]) + 5
    plan = make_plan(spec, pooling="mean")
    st = torch.zeros(1, dtype=torch.int32, device=device())
    out = tbe.forward(plan, d["tables"], bad, d["offsets"], status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == tbe.STATUS_INDEX_OOB
    with pytest.raises(RuntimeError, match="index out of range"):
        tbe.check_status(st)
    tab = raw_tables(spec, d["tables"].cpu())[t]
    ref, ab = oracle.forward([int(spec.rows[t])], [int(spec.dims[t])], "f32", [tab],
                             d["indices"][s + 1:e].cpu().numpy(), [0, e - s - 1], 1)
    c0 = int(spec.dim_off[t])
    got = out[b, c0:c0 + int(spec.dims[t])].cpu().numpy().astype(np.float64) * (e - s)
    assert oracle.summation_error(got, ref[0], ab[0]).max() <= 2 * RTOL["f32"]


@pytest.mark.slow
def test_full_size_cfg3_variants_sampled():
    """cfg3 at full size (31.7 GB of fp16 tables) with mean pooling, int32
    indices and bf16 output, in the launch configuration the benchmark uses;
    1000 sampled bags against the oracle."""
    spec = workloads.make_config(3)
    d = inputs(spec, "i32")
    out = forward(spec, d, pooling="mean", index="i32", out="bf16")
    rng = np.random.default_rng(0)
    bags = sorted(rng.choice(spec.T * spec.B, 1000, replace=False))
    d64 = dict(d, indices=d["indices"].to(torch.int64), offsets=d["offsets"].to(torch.int64))
    res = oracle_forward_bags(spec, d64, bags, pooling="mean")
    worst = -1.0
    for k, (ref, ab) in res.items():
        t, b = divmod(k, spec.B)
        c0 = int(spec.dim_off[t])
        y = out[b, c0:c0 + int(spec.dims[t])].float().cpu().numpy().astype(np.float64)
        excess = np.abs(y - ref) - (RTOL["f16"] * ab + OUT_HALF_ULP["bf16"] * np.abs(ref))
        worst = max(worst, float(excess.max()))
    note(f"[var] cfg3 full mean/i32/bf16: max excess {worst:.3g}")
    assert worst <= 0


# ------------------------------------------------------------------ backward


def backward(spec, d, **kw):  # kw: make_plan options
    plan = make_plan(spec, **kw)
    st = torch.zeros(1, dtype=torch.int32, device=device())
    g = tbe.backward(plan, d["grad_out"], d["indices"], d["offsets"], d.get("weights"), status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    return g


def check_backward(spec, d, g, pooling):
    idx = d["indices"].cpu().numpy().astype(np.int64)
    off = d["offsets"].cpu().numpy().astype(np.int64)
    seg = oracle.backward_segments(spec.rows, spec.dims, idx, off, spec.B)
    w = None if d.get("weights") is None else d["weights"].cpu().numpy()
    ref, ab, _ = oracle.backward_rows(spec.rows, spec.dims, off, spec.B, d["grad_out"].cpu().numpy(), seg,
                                      weights=w, pooling=pooling)
    gidx, segs, gro, rows = g.trimmed()
    np.testing.assert_array_equal(gidx.numpy(), seg["grad_idx"])
    np.testing.assert_array_equal(segs.numpy(), seg["seg_offsets"])
    np.testing.assert_array_equal(gro.numpy(), seg["grad_row_offsets"])
    err = float(oracle.summation_error(rows.numpy(), ref, ab).max()) if ref.size else 0.0
    note(f"[var] bwd {spec.name} pooling={pooling}: U={seg['U']} max summation error {err:.3g}")
    assert err <= GRAD_RTOL


def test_mean_backward_counts_dropped_lookups():
    """Mean-pooled backward with bounds checking: a bad lookup is dropped but
    still counts in its bag's L, so every good lookup of the bag carries
    fl32(1/L) of the full bag.  Expected: the oracle's weighted backward of the
    good lookups alone, each weighted by fl32(1/L) of its original bag."""
    spec = small(k=5, seed=4, T=3, B=150, name="mean-bwd-oob")
    d = inputs(spec)
    N = d["N"]
    off = d["offsets"].cpu().numpy().astype(np.int64)
    lens = np.diff(off)
    bags = np.nonzero(lens >= 2)[0][:5]
    bad = off[bags]  # the first lookup of five bags
    good = d["indices"].clone()
    d["indices"][torch.as_tensor(bad, device=device())] = int(spec.rows.max()) + 7
    plan = make_plan(spec, pooling="mean")
    st = torch.zeros(1, dtype=torch.int32, device=device())
    g = tbe.backward(plan, d["grad_out"], d["indices"], d["offsets"], None, status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == tbe.STATUS_INDEX_OOB
    keep = np.ones(N, bool)
    keep[bad] = False
    bag_of = np.repeat(np.arange(lens.size), lens)
    with np.errstate(divide="ignore"):  # empty bags have no lookups to weight
        inv = (np.float32(1.0) / lens.astype(np.float32)).astype(np.float32)  # fl32(1/L) of every bag
    w = inv[bag_of][keep]
    off2 = np.zeros_like(off)
    np.cumsum(np.bincount(bag_of[keep], minlength=lens.size), out=off2[1:])
    idx = good.cpu().numpy().astype(np.int64)[keep]
    seg = oracle.backward_segments(spec.rows, spec.dims, idx, off2, spec.B)
    ref, ab, _ = oracle.backward_rows(spec.rows, spec.dims, off2, spec.B, d["grad_out"].cpu().numpy(), seg,
                                      weights=w, pooling="sum")
    gidx, segs, gro, rows = g.trimmed()
    np.testing.assert_array_equal(gidx.numpy(), seg["grad_idx"])
    np.testing.assert_array_equal(segs.numpy(), seg["seg_offsets"])
    np.testing.assert_array_equal(gro.numpy(), seg["grad_row_offsets"])
    assert float(oracle.summation_error(rows.numpy(), ref, ab).max()) <= GRAD_RTOL


@pytest.mark.parametrize("B", [1, 2])
def test_mean_backward_tiny_batches(B):
    # one or two batch rows: packed records with 0 or 1 batch-row bits, and
    # each bag's fl32(1/L) read back by batch row
    spec = dataclasses.replace(small(k=5, seed=2, T=4, B=B, name=f"mean-bwd-B{B}"),
                               rows=np.array([1, 7, 300, 70000], np.int64))
    d = inputs(spec)
    check_backward(spec, d, backward(spec, d, pooling="mean"), "mean")


@pytest.mark.parametrize("index", ["i64", "i32"])
def test_mean_backward(index):
    spec = small(k=5, seed=1, T=4, B=300, name=f"mean-bwd-{index}")
    d = inputs(spec, index)
    check_backward(spec, d, backward(spec, d, pooling="mean", index=index), "mean")


@pytest.mark.slow
def test_full_size_cfg5_mean_backward_sampled():
    """cfg5 at full size with mean pooling and int32 indices, in the
    benchmark's launch configuration: the sort runs on 4-byte values (packed
    records for the tables that fit) and the reduce reads each bag's
    fl32(1/L).  Integer outputs bit-exact; gradient rows on a sample that
    includes the longest segments."""
    spec = workloads.make_config(5)
    offsets = workloads.gen_offsets(spec, device())
    d = {"offsets": offsets.to(torch.int32), "indices": workloads.gen_indices(spec, offsets).to(torch.int32),
         "N": int(offsets[-1]), "grad_out": workloads.gen_grad_out(spec, device())}
    g = backward(spec, d, pooling="mean", index="i32")
    note("[var] cfg5 full mean/i32 backward: GPU done; oracle integer part")
    idx = d["indices"].cpu().numpy().astype(np.int64)
    off = d["offsets"].cpu().numpy().astype(np.int64)
    seg = oracle.backward_segments(spec.rows, spec.dims, idx, off, spec.B)
    gidx, segs, gro, rows = g.trimmed()
    np.testing.assert_array_equal(gidx.numpy(), seg["grad_idx"])
    np.testing.assert_array_equal(segs.numpy(), seg["seg_offsets"])
    np.testing.assert_array_equal(gro.numpy(), seg["grad_row_offsets"])
    lens = np.diff(seg["seg_offsets"])
    rng = np.random.default_rng(6)
    sel = np.unique(np.concatenate([np.argsort(lens)[-20:], rng.choice(seg["U"], 2000, replace=False)]))
    ref, ab, _ = oracle.backward_rows(spec.rows, spec.dims, off, spec.B, d["grad_out"].cpu().numpy(), seg, sel=sel,
                                      pooling="mean")
    got = np.concatenate([rows[int(gro[u]):int(gro[u + 1])].numpy() for u in sel])
    err = float(oracle.summation_error(got, ref, ab).max())
    note(f"[var] cfg5 full mean/i32 backward: U={seg['U']}, max summation error {err:.3g}")
    assert err <= GRAD_RTOL


@pytest.mark.parametrize("k", [5, 4])
def test_int32_backward_equals_int64(k):
    spec = small(k=k, seed=2, T=4, B=300, grad=True, name=f"i32-bwd-cfg{k}")
    d64 = inputs(spec)
    d32 = dict(d64, indices=d64["indices"].to(torch.int32), offsets=d64["offsets"].to(torch.int32))
    a = backward(spec, d64)
    b = backward(spec, d32, index="i32")
    for x, y in zip(a.trimmed(), b.trimmed()):
        assert torch.equal(x, y)
    check_backward(spec, d32, b, "sum")


@pytest.mark.parametrize("gdt", ["f16", "bf16"])
@pytest.mark.parametrize("weighted", [False, True])
def test_reduced_precision_grad_out(gdt, weighted):
    """With a 16-bit output the gradient of the output is 16-bit too; its
    values widen exactly, so the oracle gets them as fp32."""
    spec = small(k=4 if weighted else 5, seed=7, T=4, B=300, grad=True, name=f"grad-{gdt}")
    d = inputs(spec)
    d["grad_out"] = d["grad_out"].to(OUT_TORCH[gdt])
    g = backward(spec, d, out=gdt)
    check_backward(spec, dict(d, grad_out=d["grad_out"].float()), g, "sum")


def test_reduced_precision_grad_out_past_2gib():
    """16-bit grad_out of more than 2 GiB (rows addressed with 64-bit pointers
    instead of 32-bit buffer offsets): one-hot bags over two wide tables."""
    base = workloads.small_config(2, seed=17, T=2, B=440000)
    spec = dataclasses.replace(base, dims=np.array([1536, 1024], np.int32), grad=True, name="grad-bf16-wide")
    assert spec.B * int(spec.dims.sum()) * 2 >= 2 ** 31
    d = inputs(spec)
    d["grad_out"] = d["grad_out"].to(torch.bfloat16)
    g = backward(spec, d, out="bf16")
    check_backward(spec, dict(d, grad_out=d["grad_out"].float()), g, "sum")


def test_backward_with_u8_tables():
    """The gradient never reads the tables: an 8-bit row-wise plan gives the
    same sparse gradient as an fp16 plan of the same shapes."""
    spec = small(k=5, seed=3, T=4, B=200, name="u8-bwd")
    d = inputs(spec)
    a = backward(spec, d)
    b = backward(dataclasses.replace(spec, dtype="u8"), d)
    for x, y in zip(a.trimmed(), b.trimmed()):
        assert torch.equal(x, y)


# ------------------------------------------------------------------ weight gradient


@pytest.mark.parametrize("gdt", ["f16", "bf16"])
def test_weight_grad_reduced_precision_grad_out(gdt):
    spec = small(k=4, seed=9, T=3, B=120, grad=True, name=f"wgrad-{gdt}")
    d = inputs(spec)
    g16 = d["grad_out"].to(OUT_TORCH[gdt])
    st = torch.zeros(1, dtype=torch.int32, device=device())
    gw = tbe.weight_grad(make_plan(spec, out=gdt), d["tables"], g16, d["indices"], d["offsets"], status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    ref, ab = oracle.weight_grad(spec.rows, spec.dims, spec.dtype, raw_tables(spec, d["tables"].cpu()),
                                 d["indices"].cpu().numpy(), d["offsets"].cpu().numpy(), spec.B,
                                 g16.float().cpu().numpy())
    assert oracle.summation_error(gw.cpu().numpy(), ref, ab).max() <= RTOL[spec.dtype]


def test_int32_weight_grad_equals_int64():
    spec = small(k=4, seed=4, T=3, B=120, grad=True, name="i32-wgrad")
    d64 = inputs(spec)
    d32 = dict(d64, indices=d64["indices"].to(torch.int32), offsets=d64["offsets"].to(torch.int32))
    st = torch.zeros(1, dtype=torch.int32, device=device())
    a = tbe.weight_grad(make_plan(spec), d64["tables"], d64["grad_out"], d64["indices"], d64["offsets"], status=st)
    b = tbe.weight_grad(make_plan(spec, index="i32"), d32["tables"], d32["grad_out"], d32["indices"],
                        d32["offsets"], status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    assert torch.equal(a, b)


# ------------------------------------------------------------------ unsupported combinations


def test_unsupported_combinations_rejected():
    spec = small(k=4, seed=5, T=2, B=16, grad=True, name="unsupported")
    d = inputs(spec)
    st = torch.zeros(1, dtype=torch.int32, device=device())
    mean = make_plan(spec, pooling="mean")
    with pytest.raises(tbe.TBEError) as e:
        tbe.forward(mean, d["tables"], d["indices"], d["offsets"], d["weights"], status=st)
    assert e.value.code == -8
    with pytest.raises(tbe.TBEError) as e:
        tbe.backward(mean, d["grad_out"], d["indices"], d["offsets"], d["weights"], status=st)
    assert e.value.code == -8
    with pytest.raises(tbe.TBEError) as e:
        tbe.weight_grad(mean, d["tables"], d["grad_out"], d["indices"], d["offsets"], status=st)
    assert e.value.code == -8
    u8spec = dataclasses.replace(spec, dtype="u8")
    u8 = workloads.gen_tables_flat(u8spec, device())
    with pytest.raises(tbe.TBEError) as e:
        tbe.weight_grad(make_plan(u8spec), u8, d["grad_out"], d["indices"], d["offsets"], status=st)
    assert e.value.code == -8
    g = tbe.backward(make_plan(spec), d["grad_out"], d["indices"], d["offsets"], status=st)
    with pytest.raises(tbe.TBEError) as e:
        tbe.apply_gradient(make_plan(u8spec), u8, g, tbe.SGD, 0.1)
    assert e.value.code == -8
    torch.cuda.synchronize()


def test_unchecked_plans_match_checked():
    """On valid inputs a plan without bounds checking (status may be NULL)
    gives the same bits as a checking plan: forward and backward, with the
    variants combined."""
    spec = small(k=5, seed=10, T=4, B=250, dtype="u8", name="unchecked")
    d = inputs(spec, "i32")
    outs, grads = [], []
    for check in (True, False):
        plan = make_plan(spec, pooling="mean", index="i32", out="bf16", bounds_check=check)
        st = torch.zeros(1, dtype=torch.int32, device=device()) if check else None
        outs.append(tbe.forward(plan, d["tables"], d["indices"], d["offsets"], status=st))
        gplan = make_plan(spec, pooling="mean", index="i32", bounds_check=check)
        grads.append(tbe.backward(gplan, d["grad_out"], d["indices"], d["offsets"], status=st))
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])
    for x, y in zip(grads[0].trimmed(), grads[1].trimmed()):
        assert torch.equal(x, y)
