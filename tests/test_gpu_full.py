"""GPU parity at the full Llama-3 8B / 70B layer shapes and at one GPU's
share of them under tensor parallelism (8B at TP2, 70B at TP8), in the launch
configuration the benchmark times, against the fp64 oracle on sampled rows
(each chunk's first and last rows, random middle rows, random decodes): the
output y and every intermediate step (q after RoPE, the attention output,
h2, silu(gate)*up). Only the requests owning sampled rows get their cached
context seeded; the other requests read whatever finite values their blocks
hold, and their rows are checked for finiteness only. Plus the latency
profile properties dynamic chunking relies on."""
import numpy as np
import pytest

import oracle
from hb_workloads import (LLAMA3_8B, LLAMA3_8B_TP2, LLAMA3_70B, LLAMA3_70B_TP8, SWEEP_CHUNKS, SWEEP_DECODES,
                          llama70b_batch, llama8b_batch, make_weights, multi_batch, sweep_batch,
                          sweep_decode_contexts)
from hbref import (assert_parity, assert_stage, assert_swiglu_stage, check_attention_kernel, errors,
                    oracle_for_batch, sample_rows)

pytestmark = pytest.mark.gpu

_CACHE = {}


def _device_layer(shape, max_T, max_R):
    """One device layer per shape for the module (weights + 2M-token pool)."""
    from paper_2503_22562_amd.harness import DeviceLayer
    key = shape.name
    if key not in _CACHE:
        _CACHE.clear()
        import torch
        torch.cuda.empty_cache()
        w = make_weights(shape)
        from hb_workloads import POOL_TOKENS
        dl = DeviceLayer(shape, w, POOL_TOKENS // 16, max_T, max_R, pool_fill_bits=0)
        _CACHE[key] = (dl, w, oracle.weights_to_f64(w))
    return _CACHE[key]


def _check_batch(b, max_T=4096, max_R=512, seed=0, n_dec=16, stages=True):
    import torch
    from paper_2503_22562_amd import hb as H
    from paper_2503_22562_amd.harness import bf16_bits, to_device_bf16
    dl, w, w64 = _device_layer(b.shape, max_T, max_R)
    rows = sample_rows(b, seed=seed, n_dec=n_dec)
    starts = b.token_offsets()
    for r, req in enumerate(b.requests):
        owns = np.any((rows >= starts[r]) & (rows < starts[r + 1]))
        if req.context_len and owns:
            k, v = b.prior_kv(r)
            dl.append_kv(req.block_table, 0, k, v)
    x_bits = b.x_in()
    T = b.n_tokens
    y = dl.run([(q.chunk_len, q.context_len, q.block_table) for q in b.requests], to_device_bf16(x_bits))
    torch.cuda.synchronize()
    y = y.cpu().numpy()
    plans = H.hb_layer_gemm_plans(dl.layer)
    assert np.all(np.isfinite(y))
    ref, st = oracle_for_batch(b, w64, rows=rows, x_bits=x_bits, stages=True)
    ma, rl = errors(y[rows], ref)
    print(f"{b.label}: T={T} rows checked={len(rows)} max-abs={ma:.3e} rel-L2={rl:.3e} gemm plans {plans}")
    assert_parity(y[rows], ref, b.label)
    if not stages:
        return
    q_bits = bf16_bits(dl.stage(H.HB_STAGE_Q, T))[rows]
    assert_stage(oracle.bf16_bits_to_f64(q_bits), st["q"].reshape(len(rows), -1), b.label + ": q after RoPE")
    o_bits = bf16_bits(dl.stage(H.HB_STAGE_ATTN, T))[rows]
    # the attention output: the kernel against the oracle on the kernel's own
    # inputs (tight), and against the oracle's end-to-end value in rel-L2
    used = check_attention_kernel(dl, b, rows, q_bits, o_bits, b.label + ": attention kernel")
    ma_o, rl_o = errors(oracle.bf16_bits_to_f64(o_bits), st["o"])
    print(f"  attention: kernel error <= {used:.2f} of its bound; vs end-to-end oracle max-abs {ma_o:.3e} "
          f"rel-L2 {rl_o:.3e}")
    assert rl_o <= 1e-2, f"{b.label}: attention output rel-L2 {rl_o:.3e} against the oracle"
    h2 = dl.stage(H.HB_STAGE_H2, T).cpu().numpy()[rows]
    assert_parity(h2, st["h2"], b.label + ": h2")
    m = oracle.bf16_bits_to_f64(bf16_bits(dl.stage(H.HB_STAGE_MLP, T))[rows])
    assert_swiglu_stage(m, st, w64, b.shape.rms_eps, b.label + ": silu(gate)*up")


def test_llama8b_chunk512_plus_64_decodes(hb):
    _check_batch(llama8b_batch())


def test_llama8b_four_chunks_plus_256_decodes(hb):
    _check_batch(multi_batch())


@pytest.mark.parametrize("n_dec", SWEEP_DECODES)
@pytest.mark.parametrize("chunk", SWEEP_CHUNKS)
def test_llama8b_sweep_cells(hb, chunk, n_dec):
    """Every cell of the latency profile's grid (chunk 128..2048 x 0..256
    decodes), in the launch configuration the profile times."""
    _check_batch(sweep_batch(chunk, n_dec))


def test_latency_profile_monotone_in_chunk_size(hb):
    """Bigger chunks take longer per iteration and give more tokens/s (the
    chunk-size trade-off of the dynamic-chunking section). Criterion: for each
    decode count the median latency does not decrease with chunk size, except
    for ties within 1% on the weight-streaming plateau (chunks 128 and 256
    without decodes)."""
    from paper_2503_22562_amd import hb as H
    dl, _, _ = _device_layer(LLAMA3_8B, 4096, 512)
    mixes = [(sweep_decode_contexts(n), 0) for n in SWEEP_DECODES]
    prof = H.hb_profile(dl.layer, SWEEP_CHUNKS, mixes, warmup=3, iters=15, seed=1)
    med = prof["median_ms"]
    print("median ms\n", np.round(med, 4))
    print("tokens/s\n", np.round(prof["tokens_per_s"]))
    for i, n in enumerate(SWEEP_DECODES):
        for j in range(1, len(SWEEP_CHUNKS)):
            slack = 1.01 if (n == 0 and SWEEP_CHUNKS[j] <= 256) else 1.0
            assert med[i, j] * slack >= med[i, j - 1], f"n_dec={n}: latency drops from chunk {SWEEP_CHUNKS[j-1]} to {SWEEP_CHUNKS[j]}"
    assert np.all(prof["tokens_per_s"][:, -1] > prof["tokens_per_s"][:, 0])


@pytest.mark.timeout(900)
def test_llama70b_chunk2048_plus_32_decodes(hb):
    _check_batch(llama70b_batch(), max_T=2080, max_R=64, n_dec=4)


@pytest.mark.timeout(900)
def test_llama70b_tp8_shard_chunk2048_plus_32_decodes(hb):
    """One GPU's share of the 70B layer under tensor parallelism 8 (8 q heads
    over one kv head, F 3584, full hidden size) on the 70B request mix: the
    per-shard GEMM shapes (QKV N = 1280, O K = 1024, gate/up N = 7168, down
    K = 3584) and attention with eight query heads per kv head."""
    _check_batch(llama70b_batch(shape=LLAMA3_70B_TP8), max_T=2080, max_R=64, n_dec=4)


def test_llama8b_tp2_shard_chunk512_plus_64_decodes(hb):
    """One GPU's share of the 8B layer under tensor parallelism 2 (16 q / 4
    kv heads, F 7168) on the bench batch's request mix (its split chunk
    tiles are cut into even pieces: every work unit has a slot; the 70B TP8
    shard's keep full pieces)."""
    _check_batch(llama8b_batch(shape=LLAMA3_8B_TP2))


def _fill_pool_random(dl, seed=5):
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    for t in (dl.k_pool, dl.v_pool):
        flat = t.view(-1)
        for s in range(0, flat.numel(), 1 << 28):
            n = min(1 << 28, flat.numel() - s)
            flat[s:s + n].copy_(torch.randn(n, device="cuda", generator=g).to(torch.bfloat16))


def test_latency_model_predicts_off_grid_batches_and_selects_chunks(hb):
    """The latency model fitted to profile cells (the sweep grid plus chunks
    after a 4096-token context) predicts batches off that grid -- several
    chunks with 256 decodes, decode-only, long-context chunks -- within 15%
    on average and 25% at worst (kernel time, cold cache, both sides timed
    the same way); and a chunk the selector picks for a given slack, with
    the model's largest under-prediction on its fit cells as the safety
    margin, runs within that slack (no allowance)."""
    import torch
    from paper_2503_22562_amd import hb as H
    from paper_2503_22562_amd.harness import to_device_bf16
    from hb_workloads import make_batch
    dl, _, _ = _device_layer(LLAMA3_8B, 4096, 512)
    _fill_pool_random(dl)
    mixes = [(sweep_decode_contexts(n), 0) for n in SWEEP_DECODES] + [([], 4096), (sweep_decode_contexts(64), 4096)]
    prof = H.hb_profile(dl.layer, SWEEP_CHUNKS, mixes, warmup=3, iters=15, seed=1)
    model = H.hb_fit_latency_model(dl.cfg, SWEEP_CHUNKS, mixes, prof["median_ms"])
    print("coef", np.round(list(model.coef), 4), "fit rel rms", round(model.fit_rel_rms, 4),
          "fit max under", round(model.fit_max_under, 4))
    rng = np.random.default_rng(21)
    shape = LLAMA3_8B
    vals = [llama8b_batch(), multi_batch(), sweep_batch(384, 64),
            make_batch(shape, [(1, int(c)) for c in rng.integers(256, 8192, 200)], 41),
            make_batch(shape, [(768, 6000)] + [(1, int(c)) for c in rng.integers(512, 4096, 100)], 42),
            make_batch(shape, [(2048, 8192)], 43)]
    keep, batches = [], []
    for b in vals:
        x = to_device_bf16(b.x_in())
        y = torch.empty((b.n_tokens, shape.hidden), dtype=torch.float32, device="cuda")
        keep.append((x, y))
        batches.append(([(q.chunk_len, q.context_len, q.block_table) for q in b.requests], x, y))
    cells = H.hb_profile_batches(dl.layer, batches, warmup=3, iters=15)
    errs = []
    for b, cell in zip(vals, cells):
        pred = H.hb_predict_latency(model, dl.cfg, [(q.chunk_len, q.context_len) for q in b.requests])
        errs.append(pred / cell["median_ms"] - 1)
        print(f"T={b.n_tokens:5d} requests={len(b.requests):3d} measured {cell['median_ms']:.4f} "
              f"predicted {pred:.4f} ({100 * errs[-1]:+.1f}%)")
    errs = np.abs(errs)
    assert errs.mean() <= 0.15 and errs.max() <= 0.25, errs

    # dynamic chunking: 64 decodes, the chunk of a prompt at context 2048
    ctx = [int(c) for c in rng.integers(512, 4096, 64)]
    margin = model.fit_max_under
    for slack in (0.45, 0.6, 0.9):
        c, pred = H.hb_select_chunk(model, dl.cfg, ctx, [100.0 + slack] * 64, 100.0, 2048, 4096, 32, margin)
        assert c > 0, f"slack {slack} ms admits no chunk"
        b = make_batch(shape, [(c, 2048)] + [(1, x) for x in ctx], 50)
        x = to_device_bf16(b.x_in())
        y = torch.empty((b.n_tokens, shape.hidden), dtype=torch.float32, device="cuda")
        meas = H.hb_profile_batches(dl.layer, [([(q.chunk_len, q.context_len, q.block_table) for q in b.requests],
                                                 x, y)], warmup=3, iters=15)[0]["median_ms"]
        print(f"slack {slack} ms: chunk {c}, predicted {pred:.4f} (margin {margin:.3f}), measured {meas:.4f}")
        assert meas <= slack


def test_latency_profile_is_reproducible(hb):
    """Two hb_profile runs over the same cells (a decode-heavy, a balanced
    and a chunk-heavy one) agree within 3% on every median: the predictor is
    fitted to these numbers, so they must not depend on the run."""
    from paper_2503_22562_amd import hb as H
    dl, _, _ = _device_layer(LLAMA3_8B, 4096, 512)
    _fill_pool_random(dl)
    chunks = [128, 512, 2048]
    mixes = [(sweep_decode_contexts(n), 0) for n in (0, 256)]
    a = H.hb_profile(dl.layer, chunks, mixes, warmup=10, iters=40, seed=3)["median_ms"]
    b = H.hb_profile(dl.layer, chunks, mixes, warmup=10, iters=40, seed=3)["median_ms"]
    rel = np.abs(a / b - 1)
    print("run 1 ms\n", np.round(a, 4), "\nrun 2 ms\n", np.round(b, 4), "\nrelative difference\n", np.round(rel, 4))
    assert rel.max() <= 0.03
