"""Test utilities: oracle references for workload batches and the parity bar."""
from __future__ import annotations

import numpy as np

import oracle

# parity bar for bf16 arithmetic against the fp64 oracle
MAX_ABS = 2e-2
REL_L2 = 1e-2


def oracle_for_batch(batch, w64, rows=None, stages=False, x_bits=None):
    """Run the oracle on a workload batch. Only requests owning a requested row
    get their cached context seeded (the others' new K/V are still written)."""
    shape = batch.shape
    cache = oracle.PagedKVCache(batch.num_blocks, shape.n_kv_heads, shape.head_dim)
    starts = batch.token_offsets()
    if rows is None:
        need = range(len(batch.requests))
    else:
        rows_a = np.asarray(rows)
        need = [r for r in range(len(batch.requests))
                if np.any((rows_a >= starts[r]) & (rows_a < starts[r + 1]))]
    for r in need:
        req = batch.requests[r]
        if req.context_len:
            k, v = batch.prior_kv(r)
            cache.write(req.block_table, 0, oracle.bf16_bits_to_f64(k), oracle.bf16_bits_to_f64(v))
    x = oracle.bf16_bits_to_f64(batch.x_in() if x_bits is None else x_bits)
    return oracle.layer_forward(w64, shape, cache, batch.requests, x, rows=rows, stages=stages)


def sample_rows(batch, seed=0, chunk_edge=8, chunk_mid=16, n_dec=16):
    """Rows checked at full size: each chunk's first and last rows, some middle
    rows, and a random subset of the decodes."""
    rng = np.random.default_rng(seed)
    starts = batch.token_offsets()
    rows = set()
    decs = []
    for r, req in enumerate(batch.requests):
        s, c = int(starts[r]), req.chunk_len
        if c == 1:
            decs.append(s)
            continue
        rows.update(range(s, s + min(chunk_edge, c)))
        rows.update(range(s + max(0, c - chunk_edge), s + c))
        if c > 2 * chunk_edge:
            rows.update(int(i) for i in rng.choice(np.arange(s + chunk_edge, s + c - chunk_edge),
                                                   size=min(chunk_mid, c - 2 * chunk_edge), replace=False))
    if decs:
        rows.update(int(i) for i in rng.choice(decs, size=min(n_dec, len(decs)), replace=False))
    return np.array(sorted(rows), dtype=np.int64)


def errors(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    d = got - ref
    return float(np.max(np.abs(d))), float(np.linalg.norm(d) / max(np.linalg.norm(ref), 1e-300))


def assert_parity(got, ref, what="y", max_abs=MAX_ABS, rel_l2=REL_L2):
    ma, rl = errors(got, ref)
    assert np.all(np.isfinite(got)), f"{what}: non-finite values"
    assert ma <= max_abs and rl <= rel_l2, f"{what}: max-abs {ma:.3e} (bar {max_abs}), rel-L2 {rl:.3e} (bar {rel_l2})"
    return ma, rl


def assert_stage(got, ref, what):
    """Intermediate bf16 values, which carry the rounding of every bf16 value
    they were computed from: |err| <= 2e-2 * max(1, |ref|) and rel-L2 <= 1e-2."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert np.all(np.isfinite(got)), f"{what}: non-finite values"
    err = np.abs(got - ref)
    bound = MAX_ABS * np.maximum(1.0, np.abs(ref))
    bad = err > bound
    ma, rl = errors(got, ref)
    worst = np.unravel_index(np.argmax(err / bound), err.shape)
    assert not bad.any() and rl <= REL_L2, (f"{what}: {bad.sum()} values off, max-abs {ma:.3e}, rel-L2 {rl:.3e}, "
                                            f"worst at {worst}: got {got[worst]:.5f} ref {ref[worst]:.5f}")
