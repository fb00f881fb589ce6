"""Seeded, counter-based synthetic workloads for the pooled embedding-bag path.

Every random draw is one output of SplitMix64 (Steele, Lea and Flood, "Fast
splittable pseudorandom number generators", OOPSLA 2014) at a counter that
names the element it feeds: table t, row r, column d; bag k; lookup j.  Any
single element can therefore be regenerated on its own, on the CPU or on a
GPU, bit for bit, without replaying a stream.  The integer hash runs as
wrapping int64 torch arithmetic, so the same code serves both devices; the
few floating-point steps are single IEEE operations (one multiply, one add,
one rounding cast) whose results do not depend on the device.

What the draws stand in for.  The paper motivates the workload (Introduction,
"Model Diversity Across Ranking Stages": embedding tables that stress memory
bandwidth; Background, "Feature Types and Memory Layout": sparse features are
variable-length int64 id lists, weighted sparse features pair each id with an
fp32 score) but ships no data.  The five configurations below are seeded
synthetic stand-ins for production DLRM sparse features:

  cfg1  1 fp32 table, 10,000 x 64, N(0, 0.01); B=512; L ~ U{1..20}; uniform ids
  cfg2  26 fp16 tables, rows log-uniform in [1e3, 1e6], D=128, U(-.05,.05);
        B=2048; L = 1; uniform ids
  cfg3  100 fp16 tables, rows log-uniform in [1e4, 1e7] (total <= 40e9 bytes),
        D in {64,128,256}, U(-.05,.05); B=16384; L = 0 with prob. 0.02, else
        min(Poisson(30), 200); ids Zipf(1.05) over a per-table permutation
  cfg4  40 bf16 tables, 5e6 x 128, U(-.05,.05); B=32768; L ~ Poisson(50);
        per-sample weights U(0,1) fp32; ids Zipf(1.2) over a permutation
  cfg5  cfg3's inputs plus an output gradient N(0,1) fp32 [B x total_dim]

Any configuration can be redrawn with dtype "u8" (8-bit row-wise tables):
each row is D uniform 8-bit codes plus a per-row fp32 scale U(2e-4, 6e-4)
and bias U(-0.06, -0.04), about what quantising U(-0.05, 0.05) rows gives,
then 8 zero bytes of padding.

Distribution recipes (the recipe is the definition):
  * uniform fp value in [lo, hi): u = 24 random bits as fp32 (exact),
    x = fl32(fl32(u * fl32((hi-lo)/2^24)) + fl32(lo)), then rounded to
    the table dtype with round-to-nearest-even.
  * normal(0, sigma): z = (sum of twelve 16-bit uniforms - 6*2^16) / 2^16,
    the classic sum-of-twelve-uniforms approximation (mean 0, variance 1,
    support [-6, 6]); z is exact in fp32; x = fl32(z * fl32(sigma)).
  * uniform integer in [0, n): ((32 random bits) * n) >> 32.
  * Zipf(alpha) over R rows: P(rank k) proportional to k^-alpha, k = 1..R,
    by inverse CDF on the fp64 prefix sums c_k = sum_{i<=k} i^-alpha:
    rank - 1 = #{k : c_k <= u * c_R} (clamped to R-1), u = 53 random bits;
    row = (a * (rank - 1) + c) mod R with gcd(a, R) = 1 drawn per table, an
    affine permutation that scatters hot ranks over the table.
  * Poisson(lam) clipped at m: inverse CDF on the fp64 table of
    P(X <= k), k < m, with u = 53 random bits; values >= m become m.
  * log-uniform rows in [lo, hi]: floor(exp(U(ln lo, ln hi))) clamped,
    drawn on the host with numpy's PCG64 (host metadata only).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np
import torch

MASK64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
MIX1 = 0xBF58476D1CE4E5B9
MIX2 = 0x94D049BB133111EB

ROLE_TABLE, ROLE_LEN, ROLE_EMPTY, ROLE_IDX, ROLE_W, ROLE_GRAD, ROLE_PERM = 1, 2, 3, 4, 5, 6, 7
ROLE_MAPID = 8
ROLE_QPARAM = 9

# name -> (torch storage dtype, bytes per stored element); "u8" is the 8-bit
# row-wise format: a row of D codes, its fp32 scale and bias, 8 zero bytes.
DTYPES = {"f32": (torch.float32, 4), "f16": (torch.float16, 2), "bf16": (torch.bfloat16, 2),
          "u8": (torch.uint8, 1)}
U8_ROW_EXTRA = 16  # bytes after a u8 row's codes: scale, bias, padding to 16
U8_SCALE = (2e-4, 6e-4)    # per-row scale range: about (0.1 / 255) x [0.5, 1.5]
U8_BIAS = (-0.06, -0.04)   # per-row bias range: about the minimum of U(-0.05, 0.05)

_CHUNK = 1 << 25


def _signed(x: int) -> int:
    x &= MASK64
    return x - (1 << 64) if x >= (1 << 63) else x


def _mix_py(z: int) -> int:
    z &= MASK64
    z = ((z ^ (z >> 30)) * MIX1) & MASK64
    z = ((z ^ (z >> 27)) * MIX2) & MASK64
    return z ^ (z >> 31)


def splitmix64_py(key: int, n: int) -> int:
    """Output n (0-based) of SplitMix64 started at state `key`, as a Python int."""
    return _mix_py((key + (n + 1) * GAMMA) & MASK64)


def _mix_t(z: torch.Tensor) -> torch.Tensor:
    # int64 tensors hold uint64 bit patterns; a logical right shift is an
    # arithmetic shift followed by a mask of the (64 - s) low bits.
    z = z ^ ((z >> 30) & ((1 << 34) - 1))
    z = z * _signed(MIX1)
    z = z ^ ((z >> 27) & ((1 << 37) - 1))
    z = z * _signed(MIX2)
    z = z ^ ((z >> 31) & ((1 << 33) - 1))
    return z


def splitmix64(key: int, n: torch.Tensor) -> torch.Tensor:
    """Outputs n (int64 tensor of counters) of SplitMix64 started at `key`."""
    return _mix_t((n + 1) * _signed(GAMMA) + _signed(key))


def stream_key(seed: int, role: int, t: int = 0) -> int:
    """Key of the stream that feeds one role (and one table) of one seed."""
    k = _mix_py((seed * GAMMA) & MASK64)
    k = _mix_py(k ^ (role * 0x632BE59BD9B4E019 & MASK64))
    return _mix_py(k ^ ((t + 1) * 0x8CB92BA72F3D8DD7 & MASK64))


def _bits(h: torch.Tensor, shift: int, nbits: int) -> torch.Tensor:
    return (h >> shift) & ((1 << nbits) - 1)


def _u53(h: torch.Tensor) -> torch.Tensor:
    return _bits(h, 11, 53).to(torch.float64) * (2.0 ** -53)


# --------------------------------------------------------------------------
# Specification


@dataclasses.dataclass
class Spec:
    name: str
    T: int
    B: int
    dtype: str
    rows: np.ndarray            # int64 [T]
    dims: np.ndarray            # int32 [T]
    values: tuple               # ("uniform", lo, hi) | ("normal", sigma)
    pooling: tuple              # ("uniform", lo, hi) | ("fixed", L) | ("poisson", mean, clip)
    empty_p: float
    index_dist: tuple           # ("uniform",) | ("zipf", alpha)
    weighted: bool
    seed: int
    attempt: int = 0
    grad: bool = False          # training step: an output gradient is drawn too

    @property
    def torch_dtype(self):
        return DTYPES[self.dtype][0]

    @property
    def elem_size(self) -> int:
        return DTYPES[self.dtype][1]

    @property
    def row_elems(self) -> np.ndarray:
        """Stored elements per row of each table (D_t, or D_t + 16 bytes for "u8")."""
        extra = U8_ROW_EXTRA if self.dtype == "u8" else 0
        return self.dims.astype(np.int64) + extra

    @property
    def dim_off(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.dims.astype(np.int64))])

    @property
    def total_dim(self) -> int:
        return int(self.dims.astype(np.int64).sum())

    @property
    def row_base(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.rows.astype(np.int64))])

    @property
    def table_offsets(self) -> np.ndarray:
        """Element offset of each table in a flat buffer, tables packed in order."""
        sizes = self.rows.astype(np.int64) * self.row_elems
        return np.concatenate([[0], np.cumsum(sizes)])[:-1]

    @property
    def table_elems(self) -> int:
        return int((self.rows.astype(np.int64) * self.row_elems).sum())

    @property
    def table_bytes(self) -> int:
        return self.table_elems * self.elem_size

    def describe(self) -> dict:
        return {
            "name": self.name, "T": self.T, "B": self.B, "dtype": self.dtype,
            "rows_total": int(self.rows.sum()), "total_dim": self.total_dim,
            "table_bytes": self.table_bytes, "pooling": list(self.pooling),
            "empty_p": self.empty_p, "index_dist": list(self.index_dist),
            "weighted": self.weighted, "seed": self.seed, "attempt": self.attempt,
        }


def _log_uniform_rows(rng: np.random.Generator, n: int, lo: int, hi: int) -> np.ndarray:
    r = np.floor(np.exp(rng.uniform(math.log(lo), math.log(hi), size=n)))
    return np.clip(r, lo, hi).astype(np.int64)


def make_config(k: int, seed: Optional[int] = None) -> Spec:
    """Full-size configuration k (1..5) with the given seed (default 1000 + k;
    configuration 5 is configuration 3's draw plus a gradient, so it defaults
    to configuration 3's seed)."""
    if seed is None:
        seed = 1003 if k == 5 else 1000 + k
    if k == 1:
        return Spec("cfg1", 1, 512, "f32", np.array([10_000], np.int64), np.array([64], np.int32),
                    ("normal", 0.01), ("uniform", 1, 20), 0.0, ("uniform",), False, seed)
    if k == 2:
        rng = np.random.default_rng([seed, 2])
        rows = _log_uniform_rows(rng, 26, 1_000, 1_000_000)
        return Spec("cfg2", 26, 2048, "f16", rows, np.full(26, 128, np.int32),
                    ("uniform", -0.05, 0.05), ("fixed", 1), 0.0, ("uniform",), False, seed)
    if k in (3, 5):
        # Redraw (rows, dims) with an attempt counter until the tables fit 40e9 bytes.
        attempt = 0
        while True:
            rng = np.random.default_rng([seed, 3, attempt])
            rows = _log_uniform_rows(rng, 100, 10_000, 10_000_000)
            dims = rng.choice(np.array([64, 128, 256], np.int32), size=100)
            if int((rows * dims).sum()) * 2 <= 40_000_000_000:
                break
            attempt += 1
        return Spec("cfg5" if k == 5 else "cfg3", 100, 16384, "f16", rows, dims.astype(np.int32),
                    ("uniform", -0.05, 0.05), ("poisson", 30.0, 200), 0.02, ("zipf", 1.05),
                    False, seed, attempt, grad=(k == 5))
    if k == 4:
        return Spec("cfg4", 40, 32768, "bf16", np.full(40, 5_000_000, np.int64), np.full(40, 128, np.int32),
                    ("uniform", -0.05, 0.05), ("poisson", 50.0, 200), 0.0, ("zipf", 1.2), True, seed)
    raise ValueError(f"unknown config {k}")


def small_config(k: int, seed: Optional[int] = None, T: Optional[int] = None, B: Optional[int] = None,
                 rows_lo: int = 64, rows_hi: int = 5000) -> Spec:
    """Configuration k's structure (dtype, dims, distributions) at a size the
    oracle finishes in seconds: fewer tables, a smaller batch, smaller tables."""
    full = make_config(k, seed)
    T = T if T is not None else min(full.T, 5)
    B = B if B is not None else min(full.B, 97)
    rng = np.random.default_rng([full.seed, 99, k])
    rows = _log_uniform_rows(rng, T, rows_lo, rows_hi)
    if k in (3, 5):
        dims = rng.choice(np.array([64, 128, 256], np.int32), size=T).astype(np.int32)
    else:
        dims = np.resize(full.dims, T).astype(np.int32)
    return dataclasses.replace(full, name=f"{full.name}-small", T=T, B=B, rows=rows, dims=dims)


# --------------------------------------------------------------------------
# Draws


def _poisson_cdf(lam: float, clip: int) -> np.ndarray:
    p = np.empty(clip, np.float64)
    p[0] = math.exp(-lam)
    for i in range(1, clip):
        p[i] = p[i - 1] * lam / i
    return np.cumsum(p)


_ZIPF_CACHE: dict = {}


def _zipf_prefix(alpha: float, rmax: int) -> np.ndarray:
    """fp64 prefix sums c_k = sum_{i<=k} i^-alpha for k = 1..rmax (cached)."""
    cur = _ZIPF_CACHE.get(alpha)
    if cur is None or cur.shape[0] < rmax:
        k = np.arange(1, rmax + 1, dtype=np.float64)
        cur = np.cumsum(k ** (-alpha))
        _ZIPF_CACHE[alpha] = cur
    return cur[:rmax]


_DEV_CACHE: dict = {}


def _on(arr: np.ndarray, device, tag) -> torch.Tensor:
    dev = torch.device(device)
    if dev.type == "cpu":
        return torch.from_numpy(arr)
    key = (tag, str(dev), arr.shape[0])
    t = _DEV_CACHE.get(key)
    if t is None:
        t = torch.from_numpy(arr).to(dev)
        _DEV_CACHE[key] = t
    return t


def gen_lengths(spec: Spec, device="cpu") -> torch.Tensor:
    """Bag lengths, int64 [T*B]; bag k = t*B + b (table-major)."""
    n = spec.T * spec.B
    k = torch.arange(n, dtype=torch.int64, device=device)
    kind = spec.pooling[0]
    if kind == "fixed":
        L = torch.full((n,), int(spec.pooling[1]), dtype=torch.int64, device=device)
    elif kind == "uniform":
        lo, hi = int(spec.pooling[1]), int(spec.pooling[2])
        h = splitmix64(stream_key(spec.seed, ROLE_LEN), k)
        L = lo + ((_bits(h, 32, 32) * (hi - lo + 1)) >> 32)
    elif kind == "poisson":
        lam, clip = float(spec.pooling[1]), int(spec.pooling[2])
        cdf = _on(_poisson_cdf(lam, clip), device, ("pois", lam, clip))
        u = _u53(splitmix64(stream_key(spec.seed, ROLE_LEN), k))
        L = torch.searchsorted(cdf, u, right=True)
    else:
        raise ValueError(kind)
    if spec.empty_p > 0:
        u = _u53(splitmix64(stream_key(spec.seed, ROLE_EMPTY), k))
        L = torch.where(u < spec.empty_p, torch.zeros_like(L), L)
    return L


def gen_offsets(spec: Spec, device="cpu", lengths: Optional[torch.Tensor] = None) -> torch.Tensor:
    """CSR offsets, int64 [T*B + 1], offsets[0] = 0, offsets[-1] = N."""
    L = gen_lengths(spec, device) if lengths is None else lengths
    off = torch.zeros(L.numel() + 1, dtype=torch.int64, device=L.device)
    torch.cumsum(L, 0, out=off[1:])
    return off


def _affine_perm(spec: Spec, t: int):
    R = int(spec.rows[t])
    rng = np.random.default_rng([stream_key(spec.seed, ROLE_PERM, t) & 0xFFFFFFFF, t])
    if R == 1:
        return 1, 0
    while True:
        a = int(rng.integers(1, R))
        if math.gcd(a, R) == 1:
            break
    c = int(rng.integers(0, R))
    return a, c


def _indices_at(spec: Spec, t: int, j: torch.Tensor) -> torch.Tensor:
    """Indices of table t at global lookup positions j (int64 tensor)."""
    R = int(spec.rows[t])
    h = splitmix64(stream_key(spec.seed, ROLE_IDX, t), j)
    if spec.index_dist[0] == "uniform":
        return (_bits(h, 32, 32) * R) >> 32
    alpha = float(spec.index_dist[1])
    cum = _zipf_prefix(alpha, R)
    full = _ZIPF_CACHE[alpha]
    cum_t = _on(full, j.device, ("zipf", alpha))[:R]
    target = _u53(h) * float(cum[R - 1])
    rank0 = torch.searchsorted(cum_t, target, right=True).clamp_(max=R - 1)
    a, c = _affine_perm(spec, t)
    return (rank0 * a + c) % R


def gen_indices(spec: Spec, offsets: torch.Tensor) -> torch.Tensor:
    """Lookup indices, int64 [N], local to each bag's table, on offsets' device."""
    N = int(offsets[-1])
    dev = offsets.device
    out = torch.empty(N, dtype=torch.int64, device=dev)
    if spec.B == 0 or N == 0:
        return out
    bounds = offsets[:: spec.B].cpu().tolist()  # start of each table's lookups, plus N
    for t in range(spec.T):
        s, e = int(bounds[t]), int(bounds[t + 1])
        for c0 in range(s, e, _CHUNK):
            c1 = min(e, c0 + _CHUNK)
            out[c0:c1] = _indices_at(spec, t, torch.arange(c0, c1, dtype=torch.int64, device=dev))
    return out


def gen_indices_at(spec: Spec, t: int, positions: torch.Tensor) -> torch.Tensor:
    """The indices at the given global lookup positions, all in table t."""
    return _indices_at(spec, t, positions.to(torch.int64))


def _values(spec: Spec, t: int, n: torch.Tensor) -> torch.Tensor:
    key = stream_key(spec.seed, ROLE_TABLE, t)
    return _value_draw(spec.values, key, n).to(spec.torch_dtype)


def _value_draw(values: tuple, key: int, n: torch.Tensor) -> torch.Tensor:
    dev = n.device
    if values[0] == "uniform":
        lo, hi = float(values[1]), float(values[2])
        u = _bits(splitmix64(key, n), 40, 24).to(torch.float32)
        scale = torch.tensor((hi - lo) / 2.0 ** 24, dtype=torch.float32, device=dev)
        shift = torch.tensor(lo, dtype=torch.float32, device=dev)
        return torch.add(torch.mul(u, scale), shift)
    if values[0] == "normal":
        return _normal12(key, n) * torch.tensor(float(values[1]), dtype=torch.float32, device=dev)
    raise ValueError(values[0])


def _normal12(key: int, n: torch.Tensor) -> torch.Tensor:
    s = torch.zeros_like(n)
    for q in range(3):
        h = splitmix64(key, n * 3 + q)
        for p in range(4):
            s += _bits(h, 16 * p, 16)
    return (s - 6 * 65536).to(torch.float32) * (2.0 ** -16)


def _u8_rows(spec: Spec, t: int, r: torch.Tensor) -> torch.Tensor:
    """Rows r of 8-bit row-wise table t as stored bytes [len(r), D_t + 16]:
    D_t uniform 8-bit codes, an fp32 scale drawn from U8_SCALE and an fp32
    bias drawn from U8_BIAS (little-endian), both per row, and 8 zero bytes."""
    D = int(spec.dims[t])
    r = r.view(-1, 1)
    n = r * D + torch.arange(D, dtype=torch.int64, device=r.device).view(1, -1)
    codes = _bits(splitmix64(stream_key(spec.seed, ROLE_TABLE, t), n.reshape(-1)), 56, 8).to(torch.uint8)
    key = stream_key(spec.seed, ROLE_QPARAM, t)
    rr = r.reshape(-1)
    scale = _value_draw(("uniform",) + U8_SCALE, key, 2 * rr)
    bias = _value_draw(("uniform",) + U8_BIAS, key, 2 * rr + 1)
    pad = torch.zeros_like(scale)
    sb = torch.stack([scale, bias, pad, pad], 1).contiguous().view(torch.uint8)
    return torch.cat([codes.view(-1, D), sb], 1)


def gen_table(spec: Spec, t: int, device="cpu", out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Table t, [R_t, D_t] in the spec's dtype (row-major); for "u8" the
    stored bytes [R_t, D_t + 16]."""
    R, D = int(spec.rows[t]), int(spec.dims[t])
    if spec.dtype == "u8":
        if out is None:
            out = torch.empty((R, D + U8_ROW_EXTRA), dtype=torch.uint8, device=device)
        step = max(1, _CHUNK // (D + U8_ROW_EXTRA))
        for r0 in range(0, R, step):
            r1 = min(R, r0 + step)
            out[r0:r1] = _u8_rows(spec, t, torch.arange(r0, r1, dtype=torch.int64, device=out.device))
        return out
    if out is None:
        out = torch.empty((R, D), dtype=spec.torch_dtype, device=device)
    flat = out.view(-1)
    dev = flat.device
    for c0 in range(0, R * D, _CHUNK):
        c1 = min(R * D, c0 + _CHUNK)
        flat[c0:c1] = _values(spec, t, torch.arange(c0, c1, dtype=torch.int64, device=dev))
    return out


def gen_table_rows(spec: Spec, t: int, row_ids, device="cpu") -> torch.Tensor:
    """Rows row_ids of table t, [len(row_ids), D_t] (same bits as gen_table)."""
    D = int(spec.dims[t])
    r = torch.as_tensor(row_ids, dtype=torch.int64, device=device).view(-1, 1)
    if spec.dtype == "u8":
        return _u8_rows(spec, t, r)
    n = r * D + torch.arange(D, dtype=torch.int64, device=device).view(1, -1)
    return _values(spec, t, n.reshape(-1)).view(-1, D)


def gen_tables_flat(spec: Spec, device="cpu") -> torch.Tensor:
    """All tables packed in table order into one flat buffer (spec.table_offsets)."""
    flat = torch.empty(spec.table_elems, dtype=spec.torch_dtype, device=device)
    offs = spec.table_offsets
    re = spec.row_elems
    for t in range(spec.T):
        R, E = int(spec.rows[t]), int(re[t])
        gen_table(spec, t, device, out=flat[int(offs[t]): int(offs[t]) + R * E].view(R, E))
    return flat


def gen_weights(spec: Spec, N: int, device="cpu", positions: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Per-sample weights U(0,1) fp32 [N] (or at the given lookup positions)."""
    j = torch.arange(N, dtype=torch.int64, device=device) if positions is None else positions
    out = torch.empty(j.numel(), dtype=torch.float32, device=j.device)
    key = stream_key(spec.seed, ROLE_W)
    for c0 in range(0, j.numel(), _CHUNK):
        c1 = min(j.numel(), c0 + _CHUNK)
        out[c0:c1] = _bits(splitmix64(key, j[c0:c1]), 40, 24).to(torch.float32) * (2.0 ** -24)
    return out


def gen_grad_out(spec: Spec, device="cpu") -> torch.Tensor:
    """Output gradient N(0,1) fp32 [B, total_dim]."""
    C = spec.total_dim
    out = torch.empty(spec.B * C, dtype=torch.float32, device=device)
    key = stream_key(spec.seed, ROLE_GRAD)
    for c0 in range(0, out.numel(), _CHUNK):
        c1 = min(out.numel(), c0 + _CHUNK)
        out[c0:c1] = _normal12(key, torch.arange(c0, c1, dtype=torch.int64, device=device))
    return out.view(spec.B, C)


def gen_grad_out_rows(spec: Spec, b_ids, device="cpu") -> torch.Tensor:
    """Rows b_ids of the output gradient (same bits as gen_grad_out)."""
    C = spec.total_dim
    b = torch.as_tensor(b_ids, dtype=torch.int64, device=device).view(-1, 1)
    n = b * C + torch.arange(C, dtype=torch.int64, device=device).view(1, -1)
    return _normal12(stream_key(spec.seed, ROLE_GRAD), n.reshape(-1)).view(-1, C)


def gen_all(spec: Spec, device="cpu") -> dict:
    """Every input of one call: flat tables, offsets, indices, weights, grad_out."""
    offsets = gen_offsets(spec, device)
    N = int(offsets[-1])
    d = {
        "tables": gen_tables_flat(spec, device),
        "offsets": offsets,
        "indices": gen_indices(spec, offsets),
        "weights": gen_weights(spec, N, device) if spec.weighted else None,
        "N": N,
    }
    if spec.grad:
        d["grad_out"] = gen_grad_out(spec, device)
    return d


# --------------------------------------------------------------------------
# MapId preprocessing inputs


def gen_map_ids(n_unique: int, batch: int, seed: int = 7, hit_p: float = 0.8, device="cpu") -> dict:
    """Inputs of the MapId preprocessing step, shaped as its evaluation
    (UniqueIDs x Batch): `mapping` holds n_unique distinct raw 62-bit ids in
    ascending order (SplitMix64 draws; a repeat is dropped, so the count can
    in principle fall short); each of the `batch` values is, with probability
    hit_p, a mapping entry chosen uniformly, else a fresh 62-bit id (unknown
    with overwhelming probability)."""
    n = torch.arange(n_unique, dtype=torch.int64, device=device)
    raw = splitmix64(stream_key(seed, ROLE_MAPID, 0), n) & ((1 << 62) - 1)
    mapping = torch.unique(raw)  # ascending
    i = torch.arange(batch, dtype=torch.int64, device=device)
    pick = splitmix64(stream_key(seed, ROLE_MAPID, 1), i)
    fresh = splitmix64(stream_key(seed, ROLE_MAPID, 2), i) & ((1 << 62) - 1)
    if mapping.numel() == 0:
        return {"values": fresh, "mapping": mapping}
    hit = _bits(pick, 11, 24).to(torch.float64) * (2.0 ** -24) < hit_p
    pos = (_bits(pick, 32, 32) * mapping.numel()) >> 32
    return {"values": torch.where(hit, mapping[pos], fresh), "mapping": mapping}

