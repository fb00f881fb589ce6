"""Parity of the MapId preprocessing kernel (HIP path through the C ABI)
against the CPU oracle: bit-exact integer outputs."""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import workloads
from paper_2512_23236_amd import tbe
from tests.gpu_util import device, note

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "mapid_example.json")


def run(values, mapping):
    v = torch.as_tensor(np.asarray(values, np.int64), device=device())
    m = torch.as_tensor(np.asarray(mapping, np.int64), device=device())
    out = tbe.map_ids(v, m)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def test_paper_worked_example():
    ex = json.load(open(GOLDEN))
    np.testing.assert_array_equal(run(ex["values"], ex["mapping"]), ex["expected"])


# the evaluation's shapes (unique ids x batch), smallest and largest of each sweep
@pytest.mark.parametrize("n_unique,batch", [(100, 10000), (5000, 10000), (10000, 2000), (10000, 50000)])
def test_evaluation_shapes(n_unique, batch):
    d = workloads.gen_map_ids(n_unique, batch, seed=n_unique + batch)
    got = run(d["values"].numpy(), d["mapping"].numpy())
    want = oracle.map_ids(d["values"].numpy(), d["mapping"].numpy())
    note(f"[mapid] {n_unique} x {batch}: {(want > 0).mean():.3f} known")
    np.testing.assert_array_equal(got, want)


def test_duplicates_extremes_and_sizes():
    rng = np.random.default_rng(33)
    big = np.iinfo(np.int64)
    for m in [1, 2, 3, 7, 64, 1000, 1 << 20]:
        M = np.sort(np.concatenate([rng.integers(-1000, 1000, size=m - 1), [big.max]])).astype(np.int64)
        v = np.concatenate([rng.integers(-1100, 1100, size=4000), [big.min, big.max, -1, 0]]).astype(np.int64)
        np.testing.assert_array_equal(run(v, M), oracle.map_ids(v, M))


def test_empty_mapping_and_no_values():
    np.testing.assert_array_equal(run([5, -3, 0], []), [0, 0, 0])
    assert run(np.zeros(0, np.int64), [1, 2]).size == 0


@pytest.mark.slow
def test_large():
    """A million-id mapping (20-step search) and 2^22 values (grid-stride
    loop); the oracle counts entries one by one, so a sample is checked."""
    d = workloads.gen_map_ids(1_000_000, 1 << 22, seed=5)
    got = run(d["values"].numpy(), d["mapping"].numpy())
    sel = np.random.default_rng(6).choice(got.size, 2000, replace=False)
    want = oracle.map_ids(d["values"].numpy()[sel], d["mapping"].numpy())
    np.testing.assert_array_equal(got[sel], want)
