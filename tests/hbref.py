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


def bf16_half_ulp(v):
    """Half the bf16 spacing at |v| (the largest rounding error of a value
    stored in bf16, round to nearest)."""
    a = np.maximum(np.abs(np.asarray(v, dtype=np.float64)), 2.0 ** -126)
    return np.ldexp(1.0, np.floor(np.log2(a)).astype(np.int64) - 8)


def assert_parity_bf16_out(got, ref, what):
    """A layer output stored in bf16 (the model passes hidden states between
    layers in bf16): the layer bar plus the storage rounding,
    |err| <= 2e-2 + half a bf16 ulp at max(|got|, |ref|), and rel-L2 <= 1e-2."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert np.all(np.isfinite(got)), f"{what}: non-finite values"
    err = np.abs(got - ref)
    bound = MAX_ABS + bf16_half_ulp(np.maximum(np.abs(got), np.abs(ref)))
    ma, rl = errors(got, ref)
    worst = np.unravel_index(np.argmax(err / bound), err.shape)
    assert np.all(err <= bound) and rl <= REL_L2, (f"{what}: {(err > bound).sum()} values off, max-abs {ma:.3e}, "
                                                   f"rel-L2 {rl:.3e}, worst at {worst}: got {got[worst]:.5f} "
                                                   f"ref {ref[worst]:.5f}")
    return ma, rl


def assert_swiglu_stage(got, st, w64, eps, what="silu(gate)*up"):
    """The SwiGLU product m = silu(g) * u of two GEMM outputs g, u (unit
    scale). Holding g and u each to the 2e-2 bar, the product rule bounds
    m's error to first order by 2e-2 * (|silu(g)| + |silu'(g) u|), plus half a
    bf16 ulp for its storage; rel-L2 <= 1e-2. g and u are the oracle's, from
    its h2 rows (st["h2"]); the reference m is the oracle's st["m"]."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(st["m"], dtype=np.float64)
    assert np.all(np.isfinite(got)), f"{what}: non-finite values"
    f = oracle.rmsnorm(st["h2"], w64["g_ffn"], eps)
    F = w64["w_gate_up"].shape[0] // 2
    g = oracle.linear(f, w64["w_gate_up"][:F])
    u = oracle.linear(f, w64["w_gate_up"][F:])
    sig = 1.0 / (1.0 + np.exp(-g))
    dsilu = sig * (1.0 + g * (1.0 - sig))  # d/dg of g * sigmoid(g)
    bound = MAX_ABS * np.maximum(1.0, np.abs(oracle.silu(g)) + np.abs(dsilu * u)) + bf16_half_ulp(ref)
    err = np.abs(got - ref)
    ma, rl = errors(got, ref)
    worst = np.unravel_index(np.argmax(err / bound), err.shape)
    assert np.all(err <= bound) and rl <= REL_L2, (
        f"{what}: {(err > bound).sum()} values off, max-abs {ma:.3e}, rel-L2 {rl:.3e}, worst at {worst}: "
        f"got {got[worst]:.5f} ref {ref[worst]:.5f} bound {bound[worst]:.4f}")
    return ma, rl


def check_attention_kernel(dl, batch, rows, q_bits, o_bits, what="attention"):
    """The attention kernel in isolation: its output rows against the oracle's
    causal attention evaluated on the kernel's own inputs -- the device's
    bf16 q (after RoPE) and the K/V the device's paged pool holds for each
    request (read back through its block table). The inputs being identical,
    what remains is the kernel's arithmetic: the probabilities enter the PV
    product as bf16 (relative error <= 2^-9 each), the output is stored as
    bf16, and fp32 accumulation is far below both. Bound per element:
    2^-8 * sum_j p_j |v_j| + half a bf16 ulp of the output + 1e-6 (twice the
    probability rounding, for the fp32 exponentials and sums).
    q_bits, o_bits: uint16 [len(rows)][n_q head_dim] of the sampled rows."""
    import torch
    from paper_2503_22562_amd.harness import bf16_bits, k_by_slot, v_by_slot
    shape = batch.shape
    nq, nkv, hd = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    rows = np.asarray(rows)
    starts = batch.token_offsets()
    q = oracle.bf16_bits_to_f64(q_bits).reshape(len(rows), nq, hd)
    got = oracle.bf16_bits_to_f64(o_bits).reshape(len(rows), nq, hd)
    worst = 0.0
    for r, req in enumerate(batch.requests):
        sel = np.nonzero((rows >= starts[r]) & (rows < starts[r + 1]))[0]
        if len(sel) == 0:
            continue
        kv = req.context_len + req.chunk_len
        nb = -(-kv // 16)
        idx = torch.from_numpy(np.asarray(req.block_table[:nb], dtype=np.int64)).to(dl.k_pool.device)
        kb = k_by_slot(bf16_bits(dl.k_pool.index_select(0, idx)))       # [nb][nkv][16][hd]
        vb = v_by_slot(bf16_bits(dl.v_pool.index_select(0, idx)))       # [nb][nkv][16][hd]
        k = oracle.bf16_bits_to_f64(kb.transpose(0, 2, 1, 3).reshape(nb * 16, nkv, hd)[:kv])
        v = oracle.bf16_bits_to_f64(vb.transpose(0, 2, 1, 3).reshape(nb * 16, nkv, hd)[:kv])
        pos = req.context_len + (rows[sel] - starts[r])
        ref = oracle.causal_attention(q[sel], k, v, pos, nkv)
        mass = oracle.causal_attention(q[sel], k, np.abs(v), pos, nkv)  # sum_j p_j |v_j|
        bound = 2.0 ** -8 * mass + bf16_half_ulp(ref) + 1e-6
        err = np.abs(got[sel] - ref)
        assert np.all(np.isfinite(got[sel])), f"{what}: non-finite values (request {r})"
        bad = err > bound
        if bad.any():
            i = np.unravel_index(np.argmax(err / bound), err.shape)
            raise AssertionError(f"{what}: request {r} (chunk {req.chunk_len} at {req.context_len}): {bad.sum()} "
                                 f"values off; worst row {rows[sel][i[0]]} head {i[1]} dim {i[2]}: got "
                                 f"{got[sel][i]:.6f} ref {ref[i]:.6f} bound {bound[i]:.2e}")
        worst = max(worst, float((err / bound).max()))
    return worst
