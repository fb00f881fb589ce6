"""The seeded input generator: published SplitMix64 vector, determinism,
element-wise regeneration, and the distributions each configuration asks for."""
import os

import numpy as np
import torch

import workloads
from workloads import gen

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_splitmix64_published_vector():
    line = [ln for ln in open(os.path.join(GOLDEN, "splitmix64.txt")) if ln.startswith("seed 1234567:")][0]
    want = [int(x) for x in line.split(":")[1].split()]
    assert [gen.splitmix64_py(1234567, n) for n in range(5)] == want
    got = gen.splitmix64(1234567, torch.arange(5)).tolist()
    assert [x & gen.MASK64 for x in got] == want


def test_same_seed_same_bytes_other_seed_differs():
    a = workloads.gen_all(workloads.small_config(3, seed=5))
    b = workloads.gen_all(workloads.small_config(3, seed=5))
    c = workloads.gen_all(workloads.small_config(3, seed=6))
    for k in ("tables", "offsets", "indices"):
        assert torch.equal(a[k], b[k])
    assert not torch.equal(a["tables"][:1000], c["tables"][:1000])


def test_rows_regenerate_bit_for_bit():
    for k in (1, 2, 3, 4):
        s = workloads.small_config(k, seed=77)
        t = s.T - 1
        full = workloads.gen_table(s, t)
        rows = [0, int(s.rows[t]) - 1, int(s.rows[t]) // 2]
        assert torch.equal(workloads.gen_table_rows(s, t, rows), full[rows])
    s = workloads.small_config(5, seed=77)
    g = workloads.gen_grad_out(s)
    assert torch.equal(workloads.gen_grad_out_rows(s, [3, 0, s.B - 1]), g[[3, 0, s.B - 1]])
    off = workloads.gen_offsets(s)
    idx = workloads.gen_indices(s, off)
    t = 1
    pos = torch.arange(int(off[t * s.B]), int(off[(t + 1) * s.B]))
    assert torch.equal(workloads.gen_indices_at(s, t, pos), idx[pos])


def test_config_shapes():
    c1, c2, c3, c4, c5 = (workloads.make_config(k) for k in range(1, 6))
    assert (c1.T, c1.B, c1.dtype, int(c1.rows[0]), int(c1.dims[0])) == (1, 512, "f32", 10000, 64)
    assert (c2.T, c2.B, c2.dtype) == (26, 2048, "f16") and set(c2.dims) == {128}
    assert c2.rows.min() >= 1000 and c2.rows.max() <= 1_000_000
    assert (c3.T, c3.B, c3.dtype) == (100, 16384, "f16") and set(c3.dims) <= {64, 128, 256}
    assert c3.rows.min() >= 10_000 and c3.rows.max() <= 10_000_000
    assert c3.table_bytes <= 40_000_000_000
    assert (c4.T, c4.B, c4.dtype, c4.weighted) == (40, 32768, "bf16", True)
    assert c4.table_bytes == 40 * 5_000_000 * 128 * 2
    # the training step draws exactly configuration 3's inputs
    assert c5.grad and np.array_equal(c5.rows, c3.rows) and np.array_equal(c5.dims, c3.dims)
    assert c5.seed == c3.seed


def test_length_distributions():
    L1 = workloads.gen_lengths(workloads.make_config(1)).numpy()
    assert L1.min() >= 1 and L1.max() <= 20 and abs(L1.mean() - 10.5) < 0.6
    assert np.all(workloads.gen_lengths(workloads.make_config(2)).numpy() == 1)
    L3 = workloads.gen_lengths(workloads.make_config(3)).numpy()
    assert abs((L3 == 0).mean() - 0.02) < 0.002
    nz = L3[L3 > 0]
    assert abs(nz.mean() - 30) < 0.1 and abs(nz.var() - 30) < 1.0 and L3.max() <= 200
    L4 = workloads.gen_lengths(workloads.make_config(4)).numpy()
    assert abs(L4.mean() - 50) < 0.1 and abs(L4.var() - 50) < 1.5


def test_value_distributions():
    s = workloads.small_config(3, seed=1)
    v = workloads.gen_table(s, 0).float().numpy()
    assert v.min() >= -0.05 and v.max() <= 0.05 and abs(v.mean()) < 2e-3
    assert abs(v.var() - 0.1 ** 2 / 12) < 2e-4
    s1 = workloads.make_config(1)
    w = workloads.gen_table(s1, 0).numpy()
    assert abs(w.mean()) < 2e-4 and abs(w.std() - 0.01) < 2e-4
    g = workloads.gen_grad_out(workloads.small_config(5, seed=2)).numpy()
    assert abs(g.mean()) < 0.02 and abs(g.std() - 1) < 0.02
    wt = workloads.gen_weights(workloads.make_config(4), 100_000).numpy()
    assert wt.min() >= 0 and wt.max() < 1 and abs(wt.mean() - 0.5) < 0.01


def test_zipf_rank_frequency_slope():
    """log count vs log rank has slope close to -alpha over the head."""
    for k, alpha in ((3, 1.05), (4, 1.2)):
        s = workloads.make_config(k)
        R = 1_000_000
        j = torch.arange(2_000_000)
        s = gen.dataclasses.replace(s, rows=np.full(s.T, R, np.int64))
        idx = gen._indices_at(s, 0, j).numpy()
        a, c = gen._affine_perm(s, 0)
        # invert the affine permutation to recover ranks
        ainv = pow(a, -1, R)
        rank = ((idx - c) % R) * ainv % R + 1
        cnt = np.bincount(rank, minlength=101)[1:101].astype(float)
        slope = np.polyfit(np.log(np.arange(1, 101)), np.log(cnt), 1)[0]
        assert abs(slope + alpha) < 0.05, slope
        assert idx.min() >= 0 and idx.max() < R
