"""Pins of the oracle's optimizer step and of its rounding to the table
formats (CPU only)."""
import numpy as np

import oracle


def bf16_values():
    """All finite bfloat16 values (as float64) with their bit patterns, sorted."""
    bits = np.arange(1 << 16, dtype=np.uint32)
    vals = (bits << 16).view(np.float32).astype(np.float64)
    ok = np.isfinite(vals)
    order = np.argsort(vals[ok], kind="stable")
    return vals[ok][order], bits[ok][order]


def nearest_even(x, vals, bits):
    """Brute force: the representable value nearest x, ties to the even pattern."""
    i = np.searchsorted(vals, x)
    cands = [j for j in (i - 1, i, i + 1) if 0 <= j < len(vals)]
    best = min(cands, key=lambda j: (abs(vals[j] - x), int(bits[j]) & 1))
    return int(bits[best])


def test_f16_rounding_matches_numpy(oracle_lib):
    rng = np.random.default_rng(41)
    xs = np.concatenate([rng.standard_normal(3000) * 10.0 ** rng.integers(-9, 5, 3000),
                         rng.uniform(-70000, 70000, 300)])
    # exact midpoints between neighbouring halves (ties) and their neighbours
    h = rng.integers(0, 0x7bff, 2000).astype(np.uint16)
    lo, hi = h.view(np.float16).astype(np.float64), (h + 1).view(np.float16).astype(np.float64)
    mid = (lo + hi) / 2
    xs = np.concatenate([xs, mid, np.nextafter(mid, 0), np.nextafter(mid, np.inf), -mid])
    for x in xs:
        assert oracle.encode(x, "f16") == int(np.float16(x).view(np.uint16)), x


def test_bf16_rounding_matches_brute_force(oracle_lib):
    vals, bits = bf16_values()
    rng = np.random.default_rng(42)
    xs = np.concatenate([rng.standard_normal(1500) * 10.0 ** rng.integers(-40, 38, 1500),
                         rng.uniform(-1, 1, 300) * 1e-39])  # subnormal range
    k = rng.integers(1, len(vals) - 1, 1500)
    mid = (vals[k] + vals[k + 1]) / 2  # ties
    for x in np.concatenate([xs, mid, np.nextafter(mid, np.inf)]):
        want = nearest_even(x, vals, bits)
        got = oracle.encode(x, "bf16")
        assert got == want or (vals[bits == got][0] == 0.0 and vals[bits == want][0] == 0.0), x


def test_f32_rounding_is_the_c_cast(oracle_lib):
    rng = np.random.default_rng(43)
    for x in rng.standard_normal(2000) * 10.0 ** rng.integers(-40, 38, 2000):
        assert oracle.encode(x, "f32") == int(np.array([x], np.float64).astype(np.float32).view(np.uint32)[0])


def layout(rows, dims):
    return np.concatenate([[0], np.cumsum(rows)]), np.asarray(dims, np.int64)


def test_sgd_exact_on_dyadic_values(oracle_lib):
    # W - lr * g with lr = 1/4 and small dyadic values is exact in every format
    rows, dims = [4, 3], [2, 8]
    rb, _ = layout(rows, dims)
    for dtype, npt in (("f32", np.float32), ("f16", np.float16)):
        tabs = [np.arange(r * d, dtype=np.float64).reshape(r, d).astype(npt) / 8 for r, d in zip(rows, dims)]
        before = [t.copy() for t in tabs]
        gidx = np.array([1, 4, 6], np.int64)  # table 0 row 1; table 1 rows 0 and 2
        gro = np.array([0, 2, 10, 18], np.int64)
        g = (np.arange(18, dtype=np.float32) - 9) / 2
        oracle.apply_gradient(rows, dims, dtype, tabs, oracle.SGD, 0.25, 0.0, None, gidx, gro, g)
        want = [b.astype(np.float64) for b in before]
        want[0][1] -= 0.25 * g[0:2]
        want[1][0] -= 0.25 * g[2:10]
        want[1][2] -= 0.25 * g[10:18]
        for t in range(2):
            np.testing.assert_array_equal(tabs[t].astype(np.float64), want[t])


def test_rowwise_adagrad_hand_worked(oracle_lib):
    # one table of 3 rows x 4; row 1 has state 3 and gradient [1, -1, 3, -3]:
    # mean g^2 = (1 + 1 + 9 + 9) / 4 = 5, s = 3 + 5 = 8, step = lr / (sqrt(8) + eps);
    # with lr = 2 * sqrt(8) and eps = 0, step = 2 and W[1] -= 2 * g.
    W = np.array([[1, 2, 3, 4], [10, 20, 30, 40], [5, 6, 7, 8]], np.float32)
    state = np.array([0.5, 3.0, 7.0])
    oracle.apply_gradient([3], [4], "f32", [W], oracle.ROWWISE_ADAGRAD, 2 * np.sqrt(8.0), 0.0, state,
                          np.array([1]), np.array([0, 4]), np.array([1, -1, 3, -3], np.float32))
    np.testing.assert_array_equal(W, [[1, 2, 3, 4], [8, 22, 24, 46], [5, 6, 7, 8]])
    np.testing.assert_array_equal(state, [0.5, 8.0, 7.0])


def test_matches_numpy_step(oracle_lib):
    """Against a numpy evaluation (binary64 arithmetic, numpy's rounding to the
    format); rows not listed stay untouched."""
    rng = np.random.default_rng(44)
    rows, dims = [50, 20, 7], [8, 64, 16]
    rb, _ = layout(rows, dims)
    for dtype, npt in (("f32", np.float32), ("f16", np.float16)):
        for kind in (oracle.SGD, oracle.ROWWISE_ADAGRAD):
            tabs = [rng.standard_normal((r, d)).astype(npt) for r, d in zip(rows, dims)]
            ref = [t.astype(np.float64) for t in tabs]
            gidx = np.sort(rng.choice(int(rb[-1]), 30, replace=False)).astype(np.int64)
            tof = np.searchsorted(rb, gidx, side="right") - 1
            lens = np.array([dims[t] for t in tof])
            gro = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
            g = rng.standard_normal(int(gro[-1])).astype(np.float32)
            state = rng.uniform(0, 2, int(rb[-1]))
            st_ref = state.copy()
            lr, eps = 0.05, 1e-3
            oracle.apply_gradient(rows, dims, dtype, tabs, kind, lr, eps,
                                  state if kind else None, gidx, gro, g)
            for u, gi in enumerate(gidx):
                t, r = tof[u], gi - rb[tof[u]]
                gu = g[gro[u]:gro[u + 1]].astype(np.float64)
                step = lr
                if kind:
                    st_ref[gi] += np.mean(gu * gu)
                    step = lr / (np.sqrt(st_ref[gi]) + eps)
                ref[t][r] = (ref[t][r] - step * gu).astype(npt).astype(np.float64)
            for t in range(3):
                np.testing.assert_array_equal(tabs[t].astype(np.float64), ref[t])
            if kind:
                np.testing.assert_allclose(state, st_ref, rtol=1e-15)
