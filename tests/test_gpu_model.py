"""GPU parity of the whole-model iteration (embedding, stacked hybrid-batch
layers, final RMSNorm, LM head, greedy choice) against the fp64 model oracle.
Every call goes through the C ABI (libhb.so)."""
import numpy as np
import pytest

import oracle
from hb_workloads import TINY, LayerShape, make_batch, make_model_weights, tiny_batch
from hbref import MAX_ABS, assert_parity, assert_parity_bf16_out, errors

pytestmark = pytest.mark.gpu

VOCAB = 200  # a ragged last tile of the head GEMM


def check_model(dm, batch, mw, ids, run):
    """Per-layer parity of a model iteration. `run(hidden)` enqueues the
    iteration with every layer's output going to `hidden` and returns
    (next_tokens, logits). Layer l is checked against the oracle layer fed
    the GPU's own bf16 input to it (the embedding rows for layer 0), at the
    layer bar plus the bf16 storage rounding of the output; the logits against
    the oracle's final RMSNorm and LM head applied to the GPU's last hidden
    state, at the layer bar. Returns (next tokens, logits, oracle logits,
    logits max-abs)."""
    import torch
    from paper_2503_22562_amd.harness import bf16_bits
    shape = batch.shape
    n_layers = len(mw["layers"])
    T, H = batch.n_tokens, shape.hidden
    hidden = torch.empty((n_layers, T, H), dtype=torch.bfloat16, device="cuda")
    nxt, logits = run(hidden)
    torch.cuda.synchronize()
    hs = oracle.bf16_bits_to_f64(bf16_bits(hidden))
    lw, caches, embed, g_final, lm_head = _oracle_model(batch, mw)
    x = embed[np.clip(np.asarray(ids, dtype=np.int64), 0, embed.shape[0] - 1)]
    for l in range(n_layers):
        ref = oracle.layer_forward(lw[l], shape, caches[l], batch.requests, x)
        ma, rl = assert_parity_bf16_out(hs[l], ref, f"layer {l} output")
        print(f"layer {l}: max-abs {ma:.3e} rel-L2 {rl:.3e}")
        x = hs[l]
    last = np.cumsum([r.chunk_len for r in batch.requests]) - 1
    ref_logits = oracle.rmsnorm(x[last], g_final, shape.rms_eps) @ lm_head.T
    got = logits.cpu().numpy().astype(np.float64)
    ma, rl = assert_parity(got, ref_logits, "logits from the last hidden state")
    print(f"logits: max-abs {ma:.3e} rel-L2 {rl:.3e}")
    return nxt.cpu().numpy(), logits.cpu().numpy(), ref_logits, ma


def _reqs(batch):
    return [(r.chunk_len, r.context_len, r.block_table) for r in batch.requests]


def _device_model(batch, mw, max_T, max_R, seed_prior=True):
    from paper_2503_22562_amd.harness import DeviceModel
    dm = DeviceModel(batch.shape, mw, batch.num_blocks, max_T, max_R)
    if seed_prior:
        for l in range(len(mw["layers"])):
            for r, req in enumerate(batch.requests):
                if req.context_len:
                    k, v = batch.prior_kv(r, layer=l)
                    dm.append_kv(l, req.block_table, 0, k, v)
    return dm


def _oracle_model(batch, mw, seed_prior=True):
    shape = batch.shape
    lw = [oracle.weights_to_f64(w) for w in mw["layers"]]
    caches = []
    for l in range(len(lw)):
        cache = oracle.PagedKVCache(batch.num_blocks, shape.n_kv_heads, shape.head_dim)
        if seed_prior:
            for r, req in enumerate(batch.requests):
                if req.context_len:
                    k, v = batch.prior_kv(r, layer=l)
                    cache.write(req.block_table, 0, oracle.bf16_bits_to_f64(k), oracle.bf16_bits_to_f64(v))
        caches.append(cache)
    f = oracle.bf16_bits_to_f64
    return lw, caches, f(mw["embed"]), f(mw["g_final"]), f(mw["lm_head"])


def _check_choice(nxt, logits, ref_logits, tol):
    """next_tokens is the argmax of the device's own fp32 logits (lowest index
    on ties) exactly. Against the oracle: with every logit off by at most
    `tol` (the measured max-abs error), the device must pick the oracle's
    token wherever the oracle's top two logits are more than 2 tol apart, and
    otherwise one whose oracle logit is within 2 tol of the maximum."""
    assert np.array_equal(nxt, np.argmax(logits, axis=1)), "argmax kernel"
    for r in range(ref_logits.shape[0]):
        row = ref_logits[r]
        top = np.sort(row)[-2:]
        if top[1] - top[0] > 2 * tol:
            assert nxt[r] == int(np.argmax(row)), f"request {r}: next token {nxt[r]} vs oracle {np.argmax(row)}"
        else:
            assert row[nxt[r]] >= top[1] - 2 * tol, f"request {r}: next token {nxt[r]} not near the maximum"


def test_tiny_model_two_layers_parity(hb):
    import torch
    b = tiny_batch()
    mw = make_model_weights(TINY, 2, VOCAB)
    ids = b.token_ids(VOCAB)
    dm = _device_model(b, mw, b.n_tokens, len(b.requests))
    nxt, logits, ref, ma = check_model(dm, b, mw, ids, lambda hs: dm.run(_reqs(b), ids, hidden_states=hs))
    _check_choice(nxt, logits, ref, ma)


def test_model_without_logits_and_back_to_back(hb):
    """Three layers, chunks and decodes at various offsets; running the same
    iteration again with the logits kept internal (the new K/V rewritten with
    the same values) gives the same next tokens."""
    import torch
    shape = LayerShape("m-g4-hd128", 512, 8, 2, 128, 688, weight_seed=21)
    mw = make_model_weights(shape, 3, 512)
    lens = [(40, 17), (1, 33), (1, 0), (70, 0), (1, 150)]
    b = make_batch(shape, lens, seed=9, num_blocks=256)
    ids = b.token_ids(512)
    dm = _device_model(b, mw, 256, 16)
    n1, l1, ref, ma = check_model(dm, b, mw, ids, lambda hs: dm.run(_reqs(b), ids, hidden_states=hs))
    n2, _ = dm.run(_reqs(b), ids, keep_logits=False)
    n3, l3 = dm.run(_reqs(b), ids)
    torch.cuda.synchronize()
    assert np.array_equal(n1, n2.cpu().numpy())
    # the internal ping-pong buffers give the same result as per-layer slices
    assert np.array_equal(l1.view(np.uint32), l3.cpu().numpy().view(np.uint32))
    _check_choice(n1, l1, ref, ma)


def test_model_chunked_prompt_equals_unsplit(hb):
    """A 96-token prompt as one chunk, or as chunks of 40 + 56 in two
    iterations (decoding meanwhile next to another request), gives the same
    last-token logits within tolerance."""
    import torch
    shape = TINY
    mw = make_model_weights(shape, 2, VOCAB)
    whole = make_batch(shape, [(96, 0)], seed=13, num_blocks=64)
    ids = whole.token_ids(VOCAB)
    bt = whole.requests[0].block_table
    dm = _device_model(whole, mw, 128, 4, seed_prior=False)
    _, lw = dm.run([(96, 0, bt)], ids)
    torch.cuda.synchronize()
    ref_whole = lw.cpu().numpy().astype(np.float64)

    dm2 = _device_model(whole, mw, 128, 4, seed_prior=False)
    other = np.array(sorted(set(range(64)) - set(bt.tolist()))[:2], dtype=np.int32)  # blocks bt does not name
    _, _ = dm2.run([(40, 0, bt), (1, 0, other)], np.concatenate([ids[:40], [5]]).astype(np.int32))
    _, ls = dm2.run([(1, 1, other), (56, 40, bt)], np.concatenate([[7], ids[40:]]).astype(np.int32))
    torch.cuda.synchronize()
    split = ls.cpu().numpy().astype(np.float64)[1:2]
    print("chunked vs unsplit", errors(split, ref_whole))
    assert_parity(split, ref_whole, "last-token logits, chunked vs unsplit")
    # the unsplit run, layer by layer against the oracle
    dm3 = _device_model(whole, mw, 128, 4, seed_prior=False)
    check_model(dm3, whole, mw, ids, lambda hs: dm3.run([(96, 0, bt)], ids, hidden_states=hs))


def test_model_rejects_bad_batches(hb):
    from paper_2503_22562_amd import hb as H
    b = tiny_batch()
    mw = make_model_weights(TINY, 1, VOCAB)
    dm = _device_model(b, mw, b.n_tokens, len(b.requests), seed_prior=False)
    ids = b.token_ids(VOCAB)
    with pytest.raises(H.HBError) as e:
        dm.run([], ids[:0])
    assert e.value.status == H.HB_ERR_INVALID
    bad = [(1, 0, np.array([300], dtype=np.int32))]  # block id outside the pool
    with pytest.raises(H.HBError) as e:
        dm.run(bad, ids[:1])
    assert e.value.status == H.HB_ERR_RANGE


def test_llama8b_shaped_two_layer_model_full_vocab(hb):
    """Two Llama-3-8B-shaped layers and a 128256-row LM head on a hybrid batch
    (a 96-token chunk at context 200 plus 16 decodes): each layer's output and
    every request's logits against the fp64 oracle, at the layer bar."""
    import torch
    from hb_workloads import LLAMA3_8B
    vocab = 128256
    mw = make_model_weights(LLAMA3_8B, 2, vocab)
    rng = np.random.default_rng(11)
    lens = [(96, 200)] + [(1, int(c)) for c in rng.integers(1, 600, 16)]
    b = make_batch(LLAMA3_8B, lens, seed=21, num_blocks=2048)
    ids = b.token_ids(vocab)
    dm = _device_model(b, mw, b.n_tokens, len(b.requests))
    nxt, logits, ref, ma = check_model(dm, b, mw, ids, lambda hs: dm.run(_reqs(b), ids, hidden_states=hs))
    _check_choice(nxt, logits, ref, ma)


def test_model_token_ids_out_of_range_read_nearest_row(hb):
    """Token ids below 0 or at/above the vocabulary read the first or last
    embedding row (the documented clamp): the same logits as the clamped ids."""
    import torch
    b = tiny_batch()
    mw = make_model_weights(TINY, 1, VOCAB)
    ids = b.token_ids(VOCAB)
    bad = ids.copy()
    bad[::3] = -5
    bad[1::3] = VOCAB + 17
    clamped = np.clip(bad, 0, VOCAB - 1).astype(np.int32)
    dm = _device_model(b, mw, b.n_tokens, len(b.requests))
    _, l_bad = dm.run(_reqs(b), bad)
    torch.cuda.synchronize()
    got_bad = l_bad.cpu().numpy()
    _, l_ok = dm.run(_reqs(b), clamped)
    torch.cuda.synchronize()
    assert np.array_equal(got_bad, l_ok.cpu().numpy())


def test_model_out_of_memory_leaves_every_pool_untouched(hb, monkeypatch):
    """A model iteration whose split-K partials do not fit the per-layer
    device limit (HB_DEVICE_ALLOC_LIMIT, read at creation) fails with
    HB_ERR_OOM before anything is enqueued: every layer's pool is unchanged.
    The same model then runs a batch that fits."""
    import torch
    from paper_2503_22562_amd import hb as H
    from paper_2503_22562_amd.harness import bf16_bits
    shape = LayerShape("m-oom", 2048, 16, 4, 128, 2048, weight_seed=23)
    mw = make_model_weights(shape, 3, 256)
    big = make_batch(shape, [(1024, 0), (1, 40)], seed=31, num_blocks=128)
    # a layer's workspace and attention partials fit; its 8-way split-K
    # partials (8 x 1025 x 4096 fp32 gate/up partials: 134 MB) do not
    monkeypatch.setenv("HB_DEVICE_ALLOC_LIMIT", str(100 << 20))
    monkeypatch.setenv("HB_GEMM_KSPLIT", "8")
    dm = _device_model(big, mw, big.n_tokens, 4, seed_prior=False)
    before = [(bf16_bits(k), bf16_bits(v)) for k, v in dm.pools]
    with pytest.raises(H.HBError) as e:
        dm.run(_reqs(big), big.token_ids(256))
    assert e.value.status == H.HB_ERR_OOM
    torch.cuda.synchronize()
    for (k, v), (k0, v0) in zip(dm.pools, before):
        assert np.array_equal(bf16_bits(k), k0) and np.array_equal(bf16_bits(v), v0)
    small = make_batch(shape, [(8, 0), (1, 3)], seed=32, num_blocks=128)
    nxt, logits = dm.run(_reqs(small), small.token_ids(256))
    torch.cuda.synchronize()
    n = nxt.cpu().numpy()
    assert n.shape == (2,) and np.all((n >= 0) & (n < 256))
    assert np.all(np.isfinite(logits.cpu().numpy()))
