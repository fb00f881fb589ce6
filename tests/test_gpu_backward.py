"""Backward (sparse gradient) parity of the HIP path against the CPU oracle:
row ids, segment boundaries and row offsets bit-exact; gradient rows within
the fp32 summation tolerance."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import workloads
from paper_2512_23236_amd import tbe
from tests.gpu_util import device, note, plan_for

pytestmark = pytest.mark.gpu

GRAD_RTOL = 1e-5   # the gradient touches only fp32 data


def run_backward(spec, d, bounds_check=True, capacity=None):
    plan = plan_for(spec, bounds_check)
    status = torch.zeros(1, dtype=torch.int32, device=device())
    g = tbe.backward(plan, d["grad_out"], d["indices"], d["offsets"], d.get("weights"),
                     grad_rows_capacity=capacity, status=status)
    torch.cuda.synchronize()
    return g, int(status.item())


def oracle_backward(spec, d):
    idx = d["indices"].cpu().numpy()
    off = d["offsets"].cpu().numpy()
    seg = oracle.backward_segments(spec.rows, spec.dims, idx, off, spec.B)
    w = None if d.get("weights") is None else d["weights"].cpu().numpy()
    rows, ab, _ = oracle.backward_rows(spec.rows, spec.dims, off, spec.B, d["grad_out"].cpu().numpy(), seg, weights=w)
    return seg, rows, ab


def check(spec, d=None, weighted=None):
    note(f"[bwd] {spec.name} T={spec.T} B={spec.B} dims={list(spec.dims)[:6]} weighted={spec.weighted}")
    if d is None:
        d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    g, st = run_backward(spec, d)
    assert st == 0, f"status {st}"
    gidx, segs, gro, rows = g.trimmed()
    seg, ref, ab = oracle_backward(spec, d)
    np.testing.assert_array_equal(gidx.numpy(), seg["grad_idx"])
    np.testing.assert_array_equal(segs.numpy(), seg["seg_offsets"])
    np.testing.assert_array_equal(gro.numpy(), seg["grad_row_offsets"])
    err = float(oracle.summation_error(rows.numpy(), ref, ab).max()) if ref.size else 0.0
    note(f"[bwd] {spec.name}: U={seg['U']} N={d['N']} max summation error {err:.3g}")
    assert err <= GRAD_RTOL
    return g, d


@pytest.mark.parametrize("k", [5, 4])
@pytest.mark.parametrize("seed", [1, 2])
def test_small_configs(k, seed):
    # B large enough that each table's range spans several 4096-position tiles
    check(workloads.small_config(k, seed=seed, T=4, B=300))


@pytest.mark.parametrize("weighted", [False, True])
def test_dims(weighted):
    dims = [4, 8, 24, 64, 128, 256, 512, 1536]
    base = workloads.small_config(5, seed=4, T=len(dims), B=90)
    spec = dataclasses.replace(base, dtype="f32", dims=np.array(dims, np.int32), weighted=weighted,
                               name=f"bwd-dims-{'w' if weighted else 'u'}")
    check(spec)


def test_hot_rows_and_block_edges():
    """One table hit only at row 3 (a single segment thousands long, cut by
    many block edges), and a table whose segments have lengths around the
    128-position block size."""
    spec = workloads.small_config(5, seed=6, T=3, B=400)
    d = workloads.gen_all(spec, device())
    off = d["offsets"].cpu()
    s0, e0 = int(off[0]), int(off[spec.B])
    d["indices"][s0:e0] = 3
    s1, e1 = int(off[spec.B]), int(off[2 * spec.B])
    n1 = e1 - s1
    pattern = np.repeat(np.arange(n1), np.resize([127, 128, 129, 1, 256, 300, 5], n1))[:n1]
    pattern = pattern % int(spec.rows[1])
    d["indices"][s1:e1] = torch.as_tensor(pattern, device=device())
    g, _ = check(spec, d)


@pytest.mark.parametrize("fill", [0x00, 0x5A, 0xFF])
def test_workspace_contents_ignored(fill):
    """The workspace may hold anything on entry (here: a byte pattern, then
    what a different call left there); outputs are bitwise the same.  The
    first table's one long segment leaves a tile with blocks past its end."""
    spec = workloads.small_config(5, seed=14, T=3, B=300)
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    off = d["offsets"].cpu()
    d["indices"][int(off[0]):int(off[spec.B])] = 1
    other = workloads.small_config(5, seed=15, T=3, B=300)
    od = workloads.gen_all(dataclasses.replace(other, grad=True), device())
    plan, oplan = plan_for(spec), plan_for(other)
    need = max(tbe.backward_workspace_bytes(plan, d["N"]), tbe.backward_workspace_bytes(oplan, od["N"]))
    ws = torch.full((need,), fill, dtype=torch.uint8, device=device())
    status = torch.zeros(1, dtype=torch.int32, device=device())
    first = tbe.backward(plan, d["grad_out"], d["indices"], d["offsets"], workspace=ws, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    # another workload through the same workspace, then the first again
    tbe.backward(oplan, od["grad_out"], od["indices"], od["offsets"], workspace=ws, status=status)
    again = tbe.backward(plan, d["grad_out"], d["indices"], d["offsets"], workspace=ws, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    for x, y in zip(first.trimmed(), again.trimmed()):
        assert torch.equal(x, y)
    seg, ref, ab = oracle_backward(spec, d)
    gidx, segs, gro, rows = first.trimmed()
    np.testing.assert_array_equal(gidx.numpy(), seg["grad_idx"])
    np.testing.assert_array_equal(gro.numpy(), seg["grad_row_offsets"])
    assert float(oracle.summation_error(rows.numpy(), ref, ab).max()) <= GRAD_RTOL


def test_phase_events():
    """tbe_backward_timed gives the same outputs as tbe_backward and records
    every phase boundary in order."""
    spec = workloads.small_config(5, seed=17, T=3, B=300)
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    plan = plan_for(spec)
    status = torch.zeros(1, dtype=torch.int32, device=device())
    plain = tbe.backward(plan, d["grad_out"], d["indices"], d["offsets"], status=status)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(tbe.NUM_PHASES + 1)]
    timed = tbe.backward(plan, d["grad_out"], d["indices"], d["offsets"], status=status, phase_events=evs)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    for x, y in zip(plain.trimmed(), timed.trimmed()):
        assert torch.equal(x, y)
    times = [evs[i].elapsed_time(evs[i + 1]) for i in range(tbe.NUM_PHASES)]
    assert all(t >= 0 for t in times), times
    with pytest.raises(ValueError):
        tbe.backward(plan, d["grad_out"], d["indices"], d["offsets"], status=status, phase_events=evs[:2])


def test_all_tables_one_row():
    spec = dataclasses.replace(workloads.small_config(5, seed=7, T=2, B=200), rows=np.array([1, 1], np.int64))
    check(spec)


@pytest.mark.parametrize("k", [5, 4])
def test_mixed_sort_passes(k):
    # tables sorted in 1, 2 and 3 radix passes of 8 bits in one call (each
    # table stops after the passes its row count needs), at the pass-count
    # boundaries; k = 4 carries weights (64-bit sort values)
    rows = np.array([3, 255, 256, 65535, 65536, 300000], np.int64)
    base = workloads.small_config(k, seed=11, T=len(rows), B=700)
    check(dataclasses.replace(base, rows=rows, name=f"bwd-passes-{k}"))


@pytest.mark.parametrize("B", [1024, 1025])
def test_packed_records_at_the_width_limit(B):
    # Unweighted sort records pack key field and batch row into one word when
    # both fit in 32 bits: at B = 1024 (10 batch-row bits) a table of
    # 2^22 - 1 rows (22 key bits) packs and one of 2^22 rows does not; at
    # B = 1025 (11 bits) neither does, the 2^21 - 1 row table does.  Bad
    # lookups (drop keys, whose key field is all ones) sit in every table, and
    # the last batch row (all ones in its bits) looks up every table.
    rows = np.array([3, (1 << 21) - 1, (1 << 22) - 1, 1 << 22], np.int64)
    spec = dataclasses.replace(workloads.small_config(5, seed=12, T=len(rows), B=B), rows=rows,
                               name=f"bwd-packed-{B}")
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    off = d["offsets"].cpu()
    N = d["N"]
    good = d["indices"].clone()
    # one bad lookup in the first bag with lookups of each table
    bad = []
    for t in range(spec.T):
        s0, s1 = int(off[t * B]), int(off[(t + 1) * B])
        if s1 > s0:
            bad.append(s0)
    bad = torch.tensor(bad, device=device())
    d["indices"][bad] = torch.tensor([int(rows.max()) + 5] * len(bad), device=device())
    lens = torch.diff(off)
    assert all(int(lens[(t + 1) * B - 1]) > 0 for t in range(spec.T)), "the last batch row looks up every table"
    g, st = run_backward(spec, d)
    assert st & tbe.STATUS_INDEX_OOB
    keep = torch.ones(N, dtype=torch.bool)
    keep[bad.cpu()] = False
    bag = torch.repeat_interleave(torch.arange(off.numel() - 1), lens)
    off2 = torch.zeros_like(off)
    torch.cumsum(torch.bincount(bag[keep], minlength=off.numel() - 1), 0, out=off2[1:])
    d2 = dict(d, indices=good[keep.to(device())], offsets=off2.to(device()))
    seg, ref, ab = oracle_backward(spec, d2)
    gidx, segs, gro, grows = g.trimmed()
    np.testing.assert_array_equal(gidx.numpy(), seg["grad_idx"])
    np.testing.assert_array_equal(segs.numpy(), seg["seg_offsets"])
    np.testing.assert_array_equal(gro.numpy(), seg["grad_row_offsets"])
    assert float(oracle.summation_error(grows.numpy(), ref, ab).max()) <= GRAD_RTOL


@pytest.mark.parametrize("k", [5, 4])
@pytest.mark.parametrize("B", [1, 2])
def test_tiny_batches(k, B):
    # a batch row of 0 (B = 1) or 1 (B = 2) bits: every unweighted table's
    # records pack with the key field alone (B = 1) or above one bit; k = 4
    # carries weights (8-byte values, never packed)
    rows = np.array([1, 7, 300, 70000], np.int64)
    spec = dataclasses.replace(workloads.small_config(k, seed=13, T=len(rows), B=B), rows=rows,
                               name=f"bwd-tiny-{k}-{B}")
    check(spec)


def test_deterministic_repeat():
    spec = workloads.small_config(4, seed=8, T=3, B=400)
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    a, _ = run_backward(spec, d)
    b, _ = run_backward(spec, d)
    for x, y in zip(a.trimmed(), b.trimmed()):
        assert torch.equal(x, y)


def test_bounds_check_drops_bad_lookups():
    spec = workloads.small_config(5, seed=9, T=3, B=60)
    d = workloads.gen_all(spec, device())
    N = d["N"]
    bad = torch.tensor([1, N // 2, N - 1], device=device())
    good = d["indices"].clone()
    d["indices"][bad] = torch.tensor([-1, 10 ** 9, int(spec.rows.max()) + 1], device=device())
    g, st = run_backward(spec, d)
    assert st & tbe.STATUS_INDEX_OOB
    # expected: the oracle on the same lookups with the bad ones removed
    keep = torch.ones(N, dtype=torch.bool)
    keep[bad.cpu()] = False
    off = d["offsets"].cpu()
    bag = torch.repeat_interleave(torch.arange(off.numel() - 1), torch.diff(off))
    lens = torch.bincount(bag[keep], minlength=off.numel() - 1)
    off2 = torch.zeros_like(off)
    torch.cumsum(lens, 0, out=off2[1:])
    d2 = dict(d, indices=good[keep.to(device())], offsets=off2.to(device()))
    seg, ref, ab = oracle_backward(spec, d2)
    gidx, segs, gro, rows = g.trimmed()
    np.testing.assert_array_equal(gidx.numpy(), seg["grad_idx"])
    np.testing.assert_array_equal(segs.numpy(), seg["seg_offsets"])
    np.testing.assert_array_equal(gro.numpy(), seg["grad_row_offsets"])
    assert float(oracle.summation_error(rows.numpy(), ref, ab).max()) <= GRAD_RTOL


def test_bad_offsets_flagged():
    spec = workloads.small_config(5, seed=10, T=2, B=30)
    d = workloads.gen_all(spec, device())
    off = d["offsets"].clone()
    off[3], off[4] = off[4].item(), off[3].item()
    g, st = run_backward(spec, dict(d, offsets=off))
    assert st & tbe.STATUS_OFFSETS
    assert g.num_unique() == 0


def test_capacity_too_small():
    spec = workloads.small_config(5, seed=11, T=2, B=50)
    d = workloads.gen_all(spec, device())
    g, st = run_backward(spec, d, capacity=16)
    assert st & tbe.STATUS_CAPACITY
    seg, _, _ = oracle_backward(spec, d)
    gidx, segs, gro, _ = g.trimmed()
    np.testing.assert_array_equal(gidx.numpy(), seg["grad_idx"])
    np.testing.assert_array_equal(gro.numpy(), seg["grad_row_offsets"])


def test_no_lookups():
    spec = dataclasses.replace(workloads.small_config(5, seed=12, T=2, B=8), empty_p=1.0)
    d = workloads.gen_all(spec, device())
    assert d["N"] == 0
    g, st = run_backward(spec, d)
    assert st == 0 and g.num_unique() == 0
    assert int(g.seg_offsets[0]) == 0 and int(g.grad_row_offsets[0]) == 0


def test_workspace_too_small_rejected():
    spec = workloads.small_config(5, seed=13, T=2, B=8)
    d = workloads.gen_all(spec, device())
    plan = plan_for(spec)
    ws = torch.empty(16, dtype=torch.uint8, device=device())
    with pytest.raises(tbe.TBEError):
        tbe.backward(plan, d["grad_out"], d["indices"], d["offsets"], workspace=ws)


@pytest.mark.slow
def test_grad_out_past_2gib():
    """grad_out of more than 2 GiB (rows addressed with 64-bit pointers
    instead of 32-bit buffer offsets): one-hot bags over two wide tables."""
    base = workloads.small_config(2, seed=16, T=2, B=220000)
    spec = dataclasses.replace(base, dims=np.array([1536, 1024], np.int32), name="bwd-wide")
    assert spec.B * int(spec.dims.sum()) * 4 >= 2 ** 31
    check(spec)


@pytest.mark.slow
def test_full_size_cfg5():
    """Configuration 5 at full size in the benchmark's launch configuration:
    every integer output bit-exact against the oracle, gradient rows checked
    on a sample that includes the longest segments."""
    spec = workloads.make_config(5)
    note(f"[bwd-full] cfg5: generating inputs ({spec.table_bytes / 1e9:.1f} GB tables)")
    offsets = workloads.gen_offsets(spec, device())
    d = {"offsets": offsets, "indices": workloads.gen_indices(spec, offsets), "N": int(offsets[-1]),
         "grad_out": workloads.gen_grad_out(spec, device())}
    g, st = run_backward(spec, d)
    assert st == 0
    note("[bwd-full] GPU done; oracle integer part")
    idx = d["indices"].cpu().numpy()
    off = d["offsets"].cpu().numpy()
    seg = oracle.backward_segments(spec.rows, spec.dims, idx, off, spec.B)
    gidx, segs, gro, rows = g.trimmed()
    np.testing.assert_array_equal(gidx.numpy(), seg["grad_idx"])
    np.testing.assert_array_equal(segs.numpy(), seg["seg_offsets"])
    np.testing.assert_array_equal(gro.numpy(), seg["grad_row_offsets"])
    lens = np.diff(seg["seg_offsets"])
    rng = np.random.default_rng(5)
    sel = np.unique(np.concatenate([np.argsort(lens)[-20:], rng.choice(seg["U"], 2000, replace=False)]))
    note(f"[bwd-full] U={seg['U']}, oracle rows for {sel.size} segments (longest {lens.max()})")
    ref, ab, ro = oracle.backward_rows(spec.rows, spec.dims, off, spec.B, d["grad_out"].cpu().numpy(), seg, sel=sel)
    got = np.concatenate([rows[int(gro[u]):int(gro[u + 1])].numpy() for u in sel])
    err = float(oracle.summation_error(got, ref, ab).max())
    note(f"[bwd-full] max summation error {err:.3g}")
    assert err <= GRAD_RTOL


# ------------------------------------------------------------- two phases


@pytest.mark.parametrize("k,pooling", [(5, "sum"), (4, "sum"), (5, "mean")])
def test_split_phases_bitwise_equal(k, pooling):
    """tbe_backward_index then tbe_backward_reduce give exactly what
    tbe_backward gives, also when the index phase runs on a second stream
    beside a forward on the first (both only read indices and offsets)."""
    spec = workloads.small_config(k, seed=31, T=4, B=500)
    if pooling == "mean":
        spec = dataclasses.replace(spec, weighted=False)
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    plan = tbe.Plan(spec.rows, spec.dims, spec.torch_dtype, spec.B, bounds_check=True, device=device(),
                    pooling=pooling)
    w = d.get("weights")
    status = torch.zeros(1, dtype=torch.int32, device=device())
    whole = tbe.backward(plan, d["grad_out"], d["indices"], d["offsets"], w, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    side = torch.cuda.Stream(device())  # default priority, like the current stream
    main = torch.cuda.current_stream(device())
    side.wait_stream(main)
    with torch.cuda.stream(side):
        parts, ws = tbe.backward_index(plan, d["indices"], d["offsets"], w, status=status)
    out = tbe.forward(plan, d["tables"], d["indices"], d["offsets"], w, status=status)
    main.wait_stream(side)
    tbe.backward_reduce(plan, d["grad_out"], d["N"], ws, parts, per_sample_weights=w, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    for x, y in zip(whole.trimmed(), parts.trimmed()):
        assert torch.equal(x, y)
    assert torch.isfinite(out).all()
    # phase events of the split calls are recorded in order
    ie = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    re = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    tbe.backward_index(plan, d["indices"], d["offsets"], w, workspace=ws, status=status, outputs=parts, events=ie)
    tbe.backward_reduce(plan, d["grad_out"], d["N"], ws, parts, per_sample_weights=w, status=status, events=re)
    torch.cuda.synchronize()
    assert all(ie[i].elapsed_time(ie[i + 1]) >= 0 for i in range(3))
    assert all(re[i].elapsed_time(re[i + 1]) >= 0 for i in range(2))
    for x, y in zip(whole.trimmed(), parts.trimmed()):
        assert torch.equal(x, y)


def test_null_status_and_small_capacity():
    """A plan without bounds checking may pass no status word.  A capacity too
    small for the gradient then returns cleanly, writes no gradient row and
    leaves grad_row_offsets[U] > capacity for the caller to see; the integer
    outputs are still complete.  With a status word the shortfall is the
    capacity bit."""
    spec = workloads.small_config(5, seed=32, T=2, B=60)
    d = workloads.gen_all(spec, device())
    plan = plan_for(spec, bounds_check=False)
    outs = tbe.SparseGrad(torch.full((64,), 7.0, device=device()),
                          torch.empty(d["N"], dtype=torch.int64, device=device()),
                          torch.empty(d["N"] + 1, dtype=torch.int64, device=device()),
                          torch.empty(d["N"] + 1, dtype=torch.int64, device=device()),
                          torch.zeros(1, dtype=torch.int64, device=device()))
    g = tbe.backward(plan, d["grad_out"], d["indices"], d["offsets"], grad_rows_capacity=16, outputs=outs)
    torch.cuda.synchronize()
    seg, ref, ab = oracle_backward(spec, d)
    U = g.num_unique()
    assert U == seg["U"] and int(g.grad_row_offsets[U]) > 16
    np.testing.assert_array_equal(g.grad_idx[:U].cpu().numpy(), seg["grad_idx"])
    assert torch.all(g.grad_rows == 7.0)  # no gradient row written
    status = torch.zeros(1, dtype=torch.int32, device=device())
    tbe.backward(plan, d["grad_out"], d["indices"], d["offsets"], grad_rows_capacity=16, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == tbe.STATUS_CAPACITY
    g = tbe.backward(plan, d["grad_out"], d["indices"], d["offsets"])
    torch.cuda.synchronize()
    gidx, segs, gro, rows = g.trimmed()
    np.testing.assert_array_equal(gro.numpy(), seg["grad_row_offsets"])
    assert float(oracle.summation_error(rows.numpy(), ref, ab).max()) <= GRAD_RTOL


def test_segment_beyond_the_pairwise_levels():
    """One row looked up more than 2^12 * 128 = 524,288 times: its segment has
    more pieces than the combine's pairwise levels hold, so the combine's last
    accumulator is used; a second table keeps ordinary segments beside it."""
    spec = dataclasses.replace(workloads.small_config(5, seed=33, T=2, B=22000), dims=np.array([64, 128], np.int32))
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    off = d["offsets"].cpu()
    s0, e0 = int(off[0]), int(off[spec.B])
    assert e0 - s0 > 524288 + 3 * 128
    d["indices"][s0:e0] = 7
    note(f"[bwd] one segment of {e0 - s0} lookups")
    check(spec, d)


@pytest.mark.slow
def test_full_size_cfg4_weighted():
    """The training step's backward on configuration 4's shapes (40 tables of
    5e6 rows, B = 32768, Poisson(50) bags, Zipf(1.2) ids, per-sample weights;
    hottest segment about 3e5 lookups): integer outputs bit-exact, gradient
    rows on a sample that includes the 20 longest segments."""
    spec = dataclasses.replace(workloads.make_config(4), grad=True)
    note("[bwd-cfg4] generating offsets, indices, weights, grad_out")
    offsets = workloads.gen_offsets(spec, device())
    N = int(offsets[-1])
    d = {"offsets": offsets, "indices": workloads.gen_indices(spec, offsets), "N": N,
         "weights": workloads.gen_weights(spec, N, device()), "grad_out": workloads.gen_grad_out(spec, device())}
    g, st = run_backward(spec, d)
    assert st == 0
    note(f"[bwd-cfg4] GPU done (N={N}); oracle integer part")
    idx = d["indices"].cpu().numpy()
    off = d["offsets"].cpu().numpy()
    seg = oracle.backward_segments(spec.rows, spec.dims, idx, off, spec.B)
    gidx, segs, gro, rows = g.trimmed()
    np.testing.assert_array_equal(gidx.numpy(), seg["grad_idx"])
    np.testing.assert_array_equal(segs.numpy(), seg["seg_offsets"])
    np.testing.assert_array_equal(gro.numpy(), seg["grad_row_offsets"])
    lens = np.diff(seg["seg_offsets"])
    rng = np.random.default_rng(6)
    sel = np.unique(np.concatenate([np.argsort(lens)[-20:], rng.choice(seg["U"], 2000, replace=False)]))
    note(f"[bwd-cfg4] U={seg['U']}, oracle rows for {sel.size} segments (longest {lens.max()})")
    ref, ab, ro = oracle.backward_rows(spec.rows, spec.dims, off, spec.B, d["grad_out"].cpu().numpy(), seg,
                                       weights=d["weights"].cpu().numpy(), sel=sel)
    got = np.concatenate([rows[int(gro[u]):int(gro[u + 1])].numpy() for u in sel])
    err = float(oracle.summation_error(got, ref, ab).max())
    note(f"[bwd-cfg4] max summation error {err:.3g}")
    assert err <= GRAD_RTOL
    del g, d
    torch.cuda.empty_cache()


# -------------------------------------------------- long and hot segments


def _pattern_indices(spec, d, table, lengths):
    """Table `table`'s lookups, in order, as consecutive runs of rows 0, 1, 2,
    ... with the given run lengths (cycled; rows wrap at the table size)."""
    off = d["offsets"].cpu()
    s, e = int(off[table * spec.B]), int(off[(table + 1) * spec.B])
    n = e - s
    reps = np.resize(np.asarray(lengths), n)
    pat = np.repeat(np.arange(reps.size), reps)[:n] % int(spec.rows[table])
    d["indices"][s:e] = torch.as_tensor(pat, device=device())
    return n


@pytest.mark.parametrize("weighted", [False, True])
def test_hot_segments_around_the_threshold(weighted):
    """Segments of 1023 .. 1026 and 2000 lookups beside ones of 129 .. 1000
    and short ones, in runs that straddle block and tile edges (every long
    segment is summed from per-block pieces)."""
    spec = dataclasses.replace(workloads.small_config(4 if weighted else 5, seed=51, T=2, B=3000),
                               rows=np.array([40, 3000], np.int64), dims=np.array([64, 128], np.int32))
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    n = _pattern_indices(spec, d, 0, [1023, 1024, 1025, 1026, 2000, 129, 1000, 7, 1, 300])
    note(f"[bwd-long] {n} lookups in table 0")
    check(spec, d)


@pytest.mark.parametrize("weighted", [False, True])
def test_long_segments_at_run_edges(weighted):
    """Long segments whose piece counts lie around multiples of 16 and 32
    (the combine sums whole runs of 16 pieces as fixed trees, two runs at
    once on the wave's halves for rows of at most 128 fp32 columns, then the
    last pieces one by one), on rows of 64, 128 and 256 columns."""
    spec = dataclasses.replace(workloads.small_config(4 if weighted else 5, seed=55, T=3, B=3000),
                               rows=np.array([50, 50, 50], np.int64), dims=np.array([64, 128, 256], np.int32))
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    runs = [128 * p for p in (15, 16, 17, 31, 32, 33, 47, 48, 49, 64, 65, 97)]
    for t in range(3):
        n = _pattern_indices(spec, d, t, runs[t:] + runs[:t])
        note(f"[bwd-runs] table {t}: {n} lookups")
    check(spec, d)


def test_many_long_rows_in_one_table():
    """A table with about 100 rows of more than 1024 lookups each."""
    spec = dataclasses.replace(workloads.small_config(5, seed=52, T=1, B=4000), rows=np.array([500], np.int64),
                               dims=np.array([64], np.int32))
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    n = _pattern_indices(spec, d, 0, [1100])
    assert n // 1100 >= 90
    check(spec, d)


def test_hot_segment_in_a_small_batch():
    """A batch of 50 bags whose table is hit only at one row: one segment of
    more than 1024 lookups from few batch rows."""
    spec = dataclasses.replace(workloads.small_config(5, seed=53, T=2, B=50), rows=np.array([9, 20], np.int64),
                               dims=np.array([256, 64], np.int32))
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    off = d["offsets"].cpu()
    d["indices"][int(off[0]):int(off[spec.B])] = 4
    assert int(off[spec.B]) - int(off[0]) > 1024
    check(spec, d)


@pytest.mark.parametrize("out", ["bf16", "f16"])
def test_hot_segments_mean_pooling_16bit_grad_out(out):
    """Long segments under mean pooling (weight 1/L per lookup) with a 16-bit
    output gradient (two columns per lane, 128-column slices)."""
    spec = dataclasses.replace(workloads.small_config(5, seed=54, T=2, B=2500),
                               rows=np.array([30, 700], np.int64), dims=np.array([256, 96], np.int32),
                               weighted=False)
    d = workloads.gen_all(dataclasses.replace(spec, grad=True), device())
    _pattern_indices(spec, d, 0, [5000, 1500, 40, 1025])
    dt = {"bf16": torch.bfloat16, "f16": torch.float16}[out]
    plan = tbe.Plan(spec.rows, spec.dims, spec.torch_dtype, spec.B, bounds_check=True, device=device(),
                    pooling="mean", out_dtype=dt)
    g16 = d["grad_out"].to(dt)
    status = torch.zeros(1, dtype=torch.int32, device=device())
    g = tbe.backward(plan, g16, d["indices"], d["offsets"], status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    idx, off = d["indices"].cpu().numpy(), d["offsets"].cpu().numpy()
    seg = oracle.backward_segments(spec.rows, spec.dims, idx, off, spec.B)
    ref, ab, _ = oracle.backward_rows(spec.rows, spec.dims, off, spec.B, g16.float().cpu().numpy(), seg,
                                      pooling="mean")
    gidx, segs, gro, rows = g.trimmed()
    np.testing.assert_array_equal(gidx.numpy(), seg["grad_idx"])
    np.testing.assert_array_equal(gro.numpy(), seg["grad_row_offsets"])
    err = float(oracle.summation_error(rows.numpy(), ref, ab).max())
    note(f"[bwd-long] mean {out}: max summation error {err:.3g}")
    assert err <= GRAD_RTOL
