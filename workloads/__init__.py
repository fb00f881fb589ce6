"""Seeded synthetic inputs for the pooled embedding-bag path.

This package is shared by the CPU oracle's tests and by the GPU path's tests
and benchmark.  It only draws inputs (table values, bag lengths, indices,
per-sample weights, output gradients, raw ids for the MapId step); it holds
none of the lookup, pooling, gradient or id-mapping arithmetic.
"""
from .gen import (  # noqa: F401
    Spec,
    make_config,
    small_config,
    splitmix64,
    gen_lengths,
    gen_offsets,
    gen_indices,
    gen_table,
    gen_table_rows,
    gen_tables_flat,
    gen_weights,
    gen_grad_out,
    gen_grad_out_rows,
    gen_indices_at,
    gen_all,
    gen_map_ids,
)
