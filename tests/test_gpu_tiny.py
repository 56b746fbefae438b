"""GPU parity of the hybrid-batch layer against the fp64 oracle on small
shapes, KV placement bit-exactness, invariants and edge cases. Every call
goes through the C ABI (libhb.so)."""
import numpy as np
import pytest

import oracle
from hb_workloads import (TINY, LayerShape, f32_to_bf16_bits, make_batch, make_weights, tiny_batch)
from hbref import assert_parity, assert_stage, assert_swiglu_stage, errors, oracle_for_batch

pytestmark = pytest.mark.gpu


def _setup(hb, batch, weights=None, max_T=None, max_R=None, seed_prior=True):
    from paper_2503_22562_amd.harness import DeviceLayer
    w = make_weights(batch.shape) if weights is None else weights
    dl = DeviceLayer(batch.shape, w, batch.num_blocks, max_T or max(batch.n_tokens, 1),
                     max_R or max(len(batch.requests), 1))
    if seed_prior:
        for r, req in enumerate(batch.requests):
            if req.context_len:
                k, v = batch.prior_kv(r)
                dl.append_kv(req.block_table, 0, k, v)
    return dl, w


def _reqs(batch):
    return [(r.chunk_len, r.context_len, r.block_table) for r in batch.requests]


def _run(dl, batch, x_bits=None):
    import torch
    from paper_2503_22562_amd.harness import to_device_bf16
    x = to_device_bf16(batch.x_in() if x_bits is None else x_bits)
    y = dl.run(_reqs(batch), x)
    torch.cuda.synchronize()
    return y.cpu().numpy().astype(np.float64)


def test_tiny_parity_all_rows_and_stages(hb):
    from paper_2503_22562_amd import hb as H
    from paper_2503_22562_amd.harness import bf16_bits
    b = tiny_batch()
    dl, w = _setup(hb, b)
    y = _run(dl, b)
    w64 = oracle.weights_to_f64(w)
    ref, st = oracle_for_batch(b, w64, stages=True)
    print("tiny y", errors(y, ref))
    assert_parity(y, ref)
    T = b.n_tokens
    q = oracle.bf16_bits_to_f64(bf16_bits(dl.stage(H.HB_STAGE_Q, T)))
    assert_stage(q, st["q"].reshape(T, -1), "q after RoPE")
    o = oracle.bf16_bits_to_f64(bf16_bits(dl.stage(H.HB_STAGE_ATTN, T)))
    assert_stage(o, st["o"], "attention output")
    h2 = dl.stage(H.HB_STAGE_H2, T).cpu().numpy()
    assert_parity(h2, st["h2"], "h2")
    m = oracle.bf16_bits_to_f64(bf16_bits(dl.stage(H.HB_STAGE_MLP, T)))
    assert_swiglu_stage(m, st, w64, b.shape.rms_eps)


# LDS-pipelined GEMM tile shapes of the library (hb_gemm_tile_count; a CPU test
# keeps the two equal)
GEMM_TILE_SHAPES = 15

SMALL_SHAPES = [
    LayerShape("g8-hd64", 512, 8, 1, 64, 256, weight_seed=11),
    LayerShape("g1-hd128", 512, 4, 4, 128, 336, weight_seed=12),
    LayerShape("g16-hd64", 1024, 16, 1, 64, 512, weight_seed=13),
    LayerShape("g4-hd128", 1024, 8, 2, 128, 688, weight_seed=14),
]


@pytest.mark.parametrize("splits", [(0, 0), (512, 256)], ids=["splits-auto", "item-512-tile-256"])
@pytest.mark.parametrize("shape", SMALL_SHAPES, ids=lambda s: s.name)
def test_small_shapes_parity(hb, monkeypatch, shape, splits):
    # short chunks (wave items), long chunks (workgroup tiles, split over a
    # long context), decodes on block edges and with long contexts, whose key
    # ranges run as the four waves of one workgroup combined in LDS or over
    # several such workgroups and a merge. Forced short splits: 520 keys leave
    # one wave of a workgroup an empty range, and the 300-token chunk's tiles
    # run in 256-key splits, the later ones past the first rows' positions
    split_item, split_tile = splits
    if split_item:
        monkeypatch.setenv("HB_ATTN_SPLIT_ITEM", str(split_item))
    if split_tile:
        monkeypatch.setenv("HB_ATTN_SPLIT_TILE", str(split_tile))
    lens = [(37, 21), (1, 0), (1, 15), (1, 16), (100, 0), (1, 300), (5, 3), (300, 1200), (1, 2000), (1, 519),
            (1, 3000), (1, 5000)]
    b = make_batch(shape, lens, seed=77, num_blocks=1024)
    dl, w = _setup(hb, b)
    y = _run(dl, b)
    ref = oracle_for_batch(b, oracle.weights_to_f64(w))
    print(shape.name, errors(y, ref))
    assert_parity(y, ref)




@pytest.mark.parametrize("shape", SMALL_SHAPES, ids=lambda s: s.name)
def test_item_only_batches_parity(hb, shape):
    """Batches without chunk tiles (decodes and chunks short enough to be wave
    items), whose attention launch runs one workgroup per CU: decodes at
    contexts from 0 to 5000, on block edges, one long enough to span several
    merged workgroups, and a few short chunks."""
    short = max(1, 64 // (shape.n_q_heads // shape.n_kv_heads) - 1)  # below the tile threshold
    lens = [(1, 0), (1, 15), (1, 16), (1, 300), (1, 519), (1, 2000), (1, 3000), (1, 5000), (short, 40),
            (short, 700), (2, 1), (1, 4097)]
    b = make_batch(shape, lens, seed=78, num_blocks=1024)
    dl, w = _setup(hb, b)
    y = _run(dl, b)
    ref = oracle_for_batch(b, oracle.weights_to_f64(w))
    print(shape.name, "short chunk", short, errors(y, ref))
    assert_parity(y, ref)

@pytest.mark.parametrize("case", range(6))
def test_random_batches_parity(hb, monkeypatch, case):
    """Seeded random batches on the small shapes: decodes, short and long
    chunks at random contexts, with the attention split lengths drawn too
    (automatic, or forced short so that ranges spread over merged
    workgroups, empty wave ranges and merge groups)."""
    rng = np.random.default_rng(9100 + case)
    shape = SMALL_SHAPES[case % len(SMALL_SHAPES)]
    split_item = int(rng.choice([0, 256, 512]))
    split_tile = int(rng.choice([0, 256, 1024]))
    if split_item:
        monkeypatch.setenv("HB_ATTN_SPLIT_ITEM", str(split_item))
    if split_tile:
        monkeypatch.setenv("HB_ATTN_SPLIT_TILE", str(split_tile))
    lens, T = [], 0
    for _ in range(int(rng.integers(4, 24))):
        kind = rng.integers(3)
        c = 1 if kind == 0 else int(rng.integers(2, 33)) if kind == 1 else int(rng.integers(33, 300))
        if T + c > 600:
            break
        lens.append((c, int(rng.integers(0, 3000))))
        T += c
    b = make_batch(shape, lens, seed=9200 + case, num_blocks=4096)
    print(f"case {case}: {shape.name} split_item={split_item} split_tile={split_tile} T={b.n_tokens} lens={lens}",
          flush=True)
    dl, w = _setup(hb, b)
    y = _run(dl, b)
    ref = oracle_for_batch(b, oracle.weights_to_f64(w))
    print(shape.name, errors(y, ref))
    assert_parity(y, ref)

def _expected_slots(batch, which):
    """{(block, kv_head, slot): bits[hd]} of the prior context (which = 0 K, 1 V)."""
    out = {}
    for r, req in enumerate(batch.requests):
        if not req.context_len:
            continue
        kv = batch.prior_kv(r)[which]
        for p in range(req.context_len):
            blk, s = oracle.kv_slot(req.block_table, p)
            for g in range(batch.shape.n_kv_heads):
                out[(blk, g, s)] = kv[p, g]
    return out


def _pool_bits(dl):
    """K and V pools as [block][kv head][slot][head_dim] bit patterns."""
    from paper_2503_22562_amd.harness import bf16_bits, k_by_slot, v_by_slot
    return k_by_slot(bf16_bits(dl.k_pool)), v_by_slot(bf16_bits(dl.v_pool))


def test_append_kv_placement_bit_exact(hb):
    lens = [(3, 45), (1, 16), (1, 1), (20, 31), (1, 0)]
    b = make_batch(TINY, lens, seed=5, num_blocks=64)
    dl, _ = _setup(hb, b)
    kp, vp = _pool_bits(dl)
    k_exp, v_exp = _expected_slots(b, 0), _expected_slots(b, 1)
    touched_k = np.zeros(kp.shape[:3], dtype=bool)
    for (blk, g, s), bits in k_exp.items():
        np.testing.assert_array_equal(kp[blk, g, s], bits)
        touched_k[blk, g, s] = True
    for (blk, g, s), bits in v_exp.items():
        np.testing.assert_array_equal(vp[blk, g, s], bits)
    assert np.all(kp[~touched_k] == 0xFFFF), "append_kv wrote K outside its slots"
    assert np.all(vp[~touched_k] == 0xFFFF), "append_kv wrote V outside its slots"


def test_run_writes_exactly_the_new_slots(hb):
    lens = [(23, 9), (1, 32), (1, 47), (16, 0)]
    b = make_batch(TINY, lens, seed=6, num_blocks=64)
    dl, w = _setup(hb, b)
    k0, v0 = _pool_bits(dl)
    _run(dl, b)
    k1, v1 = _pool_bits(dl)
    new = np.zeros(k0.shape[:3], dtype=bool)
    for req in b.requests:
        for p in range(req.context_len, req.kv_len):
            blk, s = oracle.kv_slot(req.block_table, p)
            new[blk, :, s] = True
    changed_k = np.any(k1 != k0, axis=-1)
    changed_v = np.any(v1 != v0, axis=-1)
    np.testing.assert_array_equal(changed_k, new)
    np.testing.assert_array_equal(changed_v, new)
    # the stored values are the rotated keys and the values of the new tokens
    _, st = oracle_for_batch(b, oracle.weights_to_f64(w), stages=True)
    starts = b.token_offsets()
    for r, req in enumerate(b.requests):
        for i in range(req.chunk_len):
            blk, s = oracle.kv_slot(req.block_table, req.context_len + i)
            t = starts[r] + i
            assert_stage(oracle.bf16_bits_to_f64(k1[blk, :, s]), st["k"][t], "stored K")
            assert_stage(oracle.bf16_bits_to_f64(v1[blk, :, s]), st["v"][t], "stored V")


def test_block_table_permutation_is_bit_exact(hb):
    lens = [(40, 50), (1, 70), (1, 3)]
    b1 = make_batch(TINY, lens, seed=8, num_blocks=64)
    b2 = make_batch(TINY, lens, seed=9, num_blocks=64)  # same data, other block ids
    b2.seed = b1.seed
    assert any(not np.array_equal(r1.block_table, r2.block_table) for r1, r2 in zip(b1.requests, b2.requests))
    w = make_weights(TINY)
    y1 = _run(_setup(hb, b1, w)[0], b1)
    y2 = _run(_setup(hb, b2, w)[0], b2)
    np.testing.assert_array_equal(y1, y2)


def test_request_order_permutes_rows_bit_exact(hb):
    lens = [(12, 30), (1, 40), (7, 0), (1, 18)]
    b = make_batch(TINY, lens, seed=10, num_blocks=64)
    dl, w = _setup(hb, b)
    x = b.x_in()
    y = _run(dl, b, x)
    order = [3, 0, 2, 1]
    starts = b.token_offsets()
    rows = np.concatenate([np.arange(starts[r], starts[r + 1]) for r in order])
    bp = make_batch(TINY, [lens[r] for r in order], seed=10, num_blocks=64)
    for i, r in enumerate(order):
        bp.requests[i].block_table = b.requests[r].block_table
    yp = _run(dl, bp, x[rows])
    np.testing.assert_array_equal(yp, y[rows])


def test_chunk_split_matches_unsplit(hb):
    w = make_weights(TINY)
    L = 70
    full = make_batch(TINY, [(L, 0), (1, 20)], seed=12, num_blocks=64)
    x_prompt = full.x_in()[:L]
    dl, _ = _setup(hb, full, w)
    x_full = full.x_in()
    y_full = _run(dl, full, x_full)[:L]
    ref = oracle_for_batch(full, oracle.weights_to_f64(w))[:L]
    assert_parity(y_full, ref, "unsplit")
    # same prompt, same blocks, as 4 chunks in successive iterations next to a decode
    dl2, _ = _setup(hb, full, w)
    bt = full.requests[0].block_table
    ys = []
    for s, e in [(0, 7), (7, 30), (30, 31), (31, 70)]:
        part = make_batch(TINY, [(e - s, s)], seed=12, num_blocks=64)
        part.requests[0].block_table = bt
        ys.append(_run(dl2, part, x_prompt[s:e]))
    y_split = np.concatenate(ys)
    assert_parity(y_split, ref, "split")
    assert_parity(y_split, y_full, "split vs unsplit", max_abs=1e-2, rel_l2=5e-3)


def test_edge_cases_positions_and_capacity(hb):
    # decode at position 0, decodes on block boundaries, a chunk that fills
    # the batch capacity exactly, block tables longer than needed
    lens = [(1, 0), (1, 15), (1, 16), (1, 31), (45, 17)]
    b = make_batch(TINY, lens, seed=13, num_blocks=64)
    b.requests[1].block_table = np.concatenate([b.requests[1].block_table, [63, 62]]).astype(np.int32)
    dl, w = _setup(hb, b, max_T=b.n_tokens, max_R=len(lens))
    y = _run(dl, b)
    ref = oracle_for_batch(b, oracle.weights_to_f64(w))
    assert_parity(y, ref)



def test_long_contexts_parity(hb):
    """Contexts of 64K-131K tokens: decodes whose key ranges spread over many
    merged workgroups and merge parts, and a chunk whose tiles are cut into
    ~25 key splits combined by the merge kernel."""
    lens = [(1, 131072), (64, 100000), (1, 65535), (1, 98304)]
    b = make_batch(TINY, lens, seed=14, num_blocks=26000)
    dl, w = _setup(hb, b)
    y = _run(dl, b)
    ref = oracle_for_batch(b, oracle.weights_to_f64(w))
    print("long contexts", errors(y, ref))
    assert_parity(y, ref)


def test_shared_prefix_blocks_parity(hb):
    """Requests that share read-only prefix blocks (prefix caching): three
    requests read the same two cached blocks (positions 0-31) and write their
    new tokens into blocks of their own; a fourth shares one block with the
    first and diverges after it. The cached values of a shared block are the
    last writer's on both sides (prior context is seeded in request order)."""
    lens = [(1, 40), (1, 40), (8, 32), (3, 20)]
    b = make_batch(TINY, lens, seed=15, num_blocks=64)
    b.requests[0].block_table = np.array([5, 9, 2], np.int32)
    b.requests[1].block_table = np.array([5, 9, 3], np.int32)
    b.requests[2].block_table = np.array([5, 9, 4], np.int32)
    b.requests[3].block_table = np.array([5, 7], np.int32)
    dl, w = _setup(hb, b)
    y = _run(dl, b)
    ref = oracle_for_batch(b, oracle.weights_to_f64(w))
    print("shared prefix", errors(y, ref))
    assert_parity(y, ref)


def test_many_requests_parity(hb):
    """400 decodes at contexts 0-600 and two chunks in one batch (metadata of
    hundreds of requests, hundreds of item groups, tiles beside them)."""
    rng = np.random.default_rng(16)
    lens = [(1, int(c)) for c in rng.integers(0, 600, 400)] + [(40, 300), (33, 0)]
    b = make_batch(TINY, lens, seed=16, num_blocks=16384)
    dl, w = _setup(hb, b)
    y = _run(dl, b)
    ref = oracle_for_batch(b, oracle.weights_to_f64(w))
    print("many requests", errors(y, ref))
    assert_parity(y, ref)


def test_layer_on_a_side_stream(hb):
    """A layer created while a non-default stream is current enqueues its work
    there: inputs written and outputs read on that stream give the oracle's
    result, for both entry points."""
    import torch
    from paper_2503_22562_amd import hb as H
    from paper_2503_22562_amd.harness import to_device_bf16
    b = tiny_batch()
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        dl, w = _setup(hb, b)
        x = to_device_bf16(b.x_in())
        y = dl.run(_reqs(b), x)
        y2 = torch.empty_like(y)
        H.hb_run_iteration_noalloc(dl.layer, _reqs(b), x, y2)
        side.synchronize()
        got, got2 = y.cpu().numpy().astype(np.float64), y2.cpu().numpy().astype(np.float64)
    ref = oracle_for_batch(b, oracle.weights_to_f64(w))
    assert_parity(got, ref)
    assert np.array_equal(got, got2)

def test_empty_batch_is_noop_and_errors_touch_nothing(hb):
    import torch
    from paper_2503_22562_amd import hb as H
    b = make_batch(TINY, [(5, 10), (1, 3)], seed=14, num_blocks=16)
    dl, _ = _setup(hb, b)
    k0, v0 = _pool_bits(dl)
    x = torch.zeros((8, TINY.hidden), dtype=torch.bfloat16, device="cuda")
    out = torch.full((8, TINY.hidden), 7.0, dtype=torch.float32, device="cuda")
    H.hb_run_iteration(dl.layer, [], x, out)
    bad = [
        [(0, 0, b.requests[0].block_table)],                        # chunk_len < 1
        [(5, 10, b.requests[0].block_table[:0])],                   # short table
        [(5, 10, np.array([99], dtype=np.int32))],                  # id out of range
        [(5, 10, b.requests[0].block_table), (5, 10, b.requests[0].block_table)],  # same slots
        [(9, 0, b.requests[0].block_table)],                        # T above capacity
    ]
    for reqs in bad:
        with pytest.raises(H.HBError):
            H.hb_run_iteration(dl.layer, reqs, x, out)
    torch.cuda.synchronize()
    k1, v1 = _pool_bits(dl)
    np.testing.assert_array_equal(k0, k1)
    np.testing.assert_array_equal(v0, v1)
    assert torch.all(out == 7.0)


def test_bf16_output_matches_fp32_output(hb):
    import torch
    from paper_2503_22562_amd import hb as H
    from paper_2503_22562_amd.harness import to_device_bf16
    b = tiny_batch(seed=3)
    dl, _ = _setup(hb, b)
    x = to_device_bf16(b.x_in())
    y32 = dl.run(_reqs(b), x, H.HB_OUT_F32)
    y16 = dl.run(_reqs(b), x, H.HB_OUT_BF16)
    torch.cuda.synchronize()
    ref = y32.to(torch.bfloat16)
    assert torch.equal(y16, ref)


@pytest.mark.parametrize("tile", list(range(GEMM_TILE_SHAPES)))
@pytest.mark.parametrize("ksplit", [1, 2, 3])
def test_every_gemm_tile_shape(hb, monkeypatch, tile, ksplit):
    """Each LDS-pipelined GEMM tile shape, whole K or split (the split-K
    reduce then applies RoPE + pool scatter, SwiGLU, or the residual add and,
    after the O projection, the pre-FFN RMSNorm),
    through whole-layer parity and the q / SwiGLU stages; all four GEMMs here
    have K % 64 == 0 and ragged M and N tails."""
    from paper_2503_22562_amd import hb as H
    from paper_2503_22562_amd.harness import bf16_bits
    monkeypatch.setenv("HB_GEMM_TILE", str(tile))
    monkeypatch.setenv("HB_GEMM_KSPLIT", str(ksplit))
    shape = LayerShape("gemm-tiles", 1024, 8, 2, 128, 1472, weight_seed=21)
    lens = [(200, 40), (1, 7), (1, 300), (90, 0), (1, 64)]
    b = make_batch(shape, lens, seed=31, num_blocks=64)
    dl, w = _setup(hb, b)
    y = _run(dl, b)
    w64 = oracle.weights_to_f64(w)
    ref, st = oracle_for_batch(b, w64, stages=True)
    print(f"tile {tile} ksplit {ksplit}", errors(y, ref))
    assert_parity(y, ref)
    T = b.n_tokens
    q = oracle.bf16_bits_to_f64(bf16_bits(dl.stage(H.HB_STAGE_Q, T)))
    assert_stage(q, st["q"].reshape(T, -1), "q after RoPE")
    h2 = dl.stage(H.HB_STAGE_H2, T).cpu().numpy()
    assert_parity(h2, st["h2"], "h2")
    m = oracle.bf16_bits_to_f64(bf16_bits(dl.stage(H.HB_STAGE_MLP, T)))
    assert_swiglu_stage(m, st, w64, b.shape.rms_eps)


def test_back_to_back_iterations_match_one_at_a_time(hb):
    """Iterations enqueued back to back, with no host synchronisation between
    them, through the ring of metadata slots (more iterations than slots,
    metadata of different sizes; two batches' metadata exceed a slot's first
    allocation, so its host and device buffers grow while earlier iterations
    are in flight) give bit-identical outputs to the same iterations run one
    at a time with a synchronisation after each."""
    import torch
    from paper_2503_22562_amd.harness import DeviceLayer, to_device_bf16
    shape = TINY
    nb = 70000
    lens_list = [
        [(64, 128)] + [(1, 256)] * 8,
        [(1, 7), (1, 300), (37, 21)],
        [(1, 16000)] * 64,            # ~100k int32 of metadata
        [(100, 0), (1, 15)],
        [(5, 3)],
        [(300, 1200), (1, 2000)],
        [(1, 9000)] * 96,             # again past the first allocation
        [(16, 16)],
        [(1, 0)],
        [(64, 128)] + [(1, 256)] * 8,
    ]
    batches = [make_batch(shape, lens, seed=900 + i, num_blocks=nb) for i, lens in enumerate(lens_list)]
    w = make_weights(shape)
    dl = DeviceLayer(shape, w, nb, max(b.n_tokens for b in batches), max(len(b.requests) for b in batches))
    xs = [to_device_bf16(b.x_in()) for b in batches]

    def reset_pool():
        dl.k_pool.view(torch.int16).fill_(0x3C00)  # bf16 2^-7
        dl.v_pool.view(torch.int16).fill_(0x3C00)

    reset_pool()
    ys = [dl.run(_reqs(b), x) for b, x in zip(batches, xs)]
    torch.cuda.synchronize()
    got = [y.cpu().numpy() for y in ys]
    reset_pool()
    for i, (b, x) in enumerate(zip(batches, xs)):
        y = dl.run(_reqs(b), x)
        torch.cuda.synchronize()
        ref = y.cpu().numpy()
        assert np.all(np.isfinite(ref)), f"batch {i}"
        assert np.array_equal(got[i].view(np.uint32), ref.view(np.uint32)), f"batch {i} differs when enqueued back to back"


def test_out_of_memory_is_reported_and_recoverable(hb, monkeypatch):
    """Device allocation failures, forced by a per-layer limit on the
    library's own device memory (HB_DEVICE_ALLOC_LIMIT, read at creation):
    creation fails with HB_ERR_OOM and leaves nothing behind; an iteration
    whose split-K partials do not fit fails with HB_ERR_OOM before anything is
    enqueued (pool and output untouched), and the layer then runs a batch
    that fits, matching the oracle."""
    import torch
    from gemmcover import COVER
    from paper_2503_22562_amd import hb as H
    from paper_2503_22562_amd.harness import DeviceLayer, bf16_bits, to_device_bf16
    w = make_weights(COVER)
    big = make_batch(COVER, [(2048, 0)], seed=71, num_blocks=256)
    monkeypatch.setenv("HB_DEVICE_ALLOC_LIMIT", "1000000")
    with pytest.raises(H.HBError) as e:
        DeviceLayer(COVER, w, big.num_blocks, big.n_tokens, 4)
    assert e.value.status == H.HB_ERR_OOM
    # workspace of about 100 MB fits, 8-way split-K partials of a 2048-token
    # batch (8 x 2048 x 5120 fp32 = 335 MB) do not
    monkeypatch.setenv("HB_DEVICE_ALLOC_LIMIT", str(200 << 20))
    monkeypatch.setenv("HB_GEMM_KSPLIT", "8")
    dl = DeviceLayer(COVER, w, big.num_blocks, big.n_tokens, 4)
    k0, v0 = bf16_bits(dl.k_pool), bf16_bits(dl.v_pool)
    x = to_device_bf16(big.x_in())
    y = torch.full((big.n_tokens, COVER.hidden), 7.0, dtype=torch.float32, device="cuda")
    with pytest.raises(H.HBError) as e:
        H.hb_run_iteration(dl.layer, _reqs(big), x, y)
    assert e.value.status == H.HB_ERR_OOM
    torch.cuda.synchronize()
    assert np.array_equal(bf16_bits(dl.k_pool), k0) and np.array_equal(bf16_bits(dl.v_pool), v0)
    assert torch.all(y == 7.0)
    small = make_batch(COVER, [(48, 20), (1, 100), (1, 0)], seed=72, num_blocks=256)
    for r, req in enumerate(small.requests):
        if req.context_len:
            k, v = small.prior_kv(r)
            dl.append_kv(req.block_table, 0, k, v)
    got = _run(dl, small)
    assert any(ks == 8 for _, ks in H.hb_layer_gemm_plans(dl.layer))
    assert_parity(got, oracle_for_batch(small, oracle.weights_to_f64(w)))


def test_profile_rejects_cells_beyond_the_pool(hb):
    """hb_profile validates every cell before touching the device: a cell
    that needs more blocks than the pool holds, or more tokens than the
    layer's capacity, is HB_ERR_INVALID and nothing runs."""
    from paper_2503_22562_amd import hb as H
    b = tiny_batch()
    dl, _ = _setup(hb, b)
    k0, v0 = _pool_bits(dl)
    with pytest.raises(H.HBError) as e:  # 256 blocks of 16: a 5000-token context does not fit
        H.hb_profile(dl.layer, [16], [([5000], 0)], warmup=0, iters=1)
    assert e.value.status == H.HB_ERR_INVALID
    with pytest.raises(H.HBError) as e:  # above max_batch_tokens
        H.hb_profile(dl.layer, [b.n_tokens + 1], [([], 0)], warmup=0, iters=1)
    assert e.value.status == H.HB_ERR_INVALID
    k1, v1 = _pool_bits(dl)
    assert np.array_equal(k0, k1) and np.array_equal(v0, v1)
