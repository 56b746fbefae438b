"""The allocation-free entry point (hb_run_iteration_noalloc) against the
ordinary one (hb_run_iteration): same output on two calls in a row, the
second with a smaller batch, with split-K partials and split attention in
use; and a batch whose scratch exceeds the fixed device array is rejected
before anything is enqueued."""
import numpy as np
import pytest

import oracle
from gemmcover import COVER
from hbref import assert_parity, errors, oracle_for_batch

pytestmark = pytest.mark.gpu


def _layer(b, w, max_T, max_R):
    from paper_2503_22562_amd.harness import DeviceLayer
    dl = DeviceLayer(COVER, w, b.num_blocks, max_T, max_R)
    for i, q in enumerate(b.requests):
        if q.context_len:
            k, v = b.prior_kv(i)
            dl.append_kv(q.block_table, 0, k, v)
    return dl


def test_noalloc_matches_run_iteration_twice(hb):
    import torch
    from hb_workloads import make_batch, make_weights
    from paper_2503_22562_amd import hb as H
    from paper_2503_22562_amd.harness import to_device_bf16
    w = make_weights(COVER)
    w64 = oracle.weights_to_f64(w)
    nb = 1024
    big = make_batch(COVER, [(200, 1500), (1, 3000), (1, 700), (90, 0), (1, 64)], seed=61, num_blocks=nb)
    small = make_batch(COVER, [(40, 900), (1, 2000), (1, 5)], seed=62, num_blocks=nb)
    # the small batch takes blocks the big one does not use, so both keep their cached context
    used = set(np.concatenate([q.block_table for q in big.requests]).tolist())
    free = np.array(sorted(set(range(nb)) - used), dtype=np.int32)
    off = 0
    for q in small.requests:
        q.block_table = free[off:off + len(q.block_table)].copy()
        off += len(q.block_table)
    dl = _layer(big, w, big.n_tokens, len(big.requests))
    for i, q in enumerate(small.requests):
        if q.context_len:
            k, v = small.prior_kv(i)
            dl.append_kv(q.block_table, 0, k, v)
    for b in (big, small):
        reqs = [(q.chunk_len, q.context_len, q.block_table) for q in b.requests]
        x = to_device_bf16(b.x_in())
        y_na = torch.full((b.n_tokens, COVER.hidden), float("nan"), dtype=torch.float32, device="cuda")
        H.hb_run_iteration_noalloc(dl.layer, reqs, x, y_na)
        torch.cuda.synchronize()
        plans = H.hb_layer_gemm_plans(dl.layer)
        y_ref = torch.full_like(y_na, float("nan"))
        H.hb_run_iteration(dl.layer, reqs, x, y_ref)
        torch.cuda.synchronize()
        assert H.hb_layer_gemm_plans(dl.layer) == plans
        got, want = y_na.cpu().numpy(), y_ref.cpu().numpy()
        print(f"T={b.n_tokens} plans {plans}: noalloc vs run_iteration max-abs {np.max(np.abs(got - want)):.3e}")
        if b is big:
            assert any(ks > 1 for _, ks in plans), "the case must use split-K partials"
        # same kernels and plans: the same bits; and the oracle's bar
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
        ref = oracle_for_batch(b, w64)
        print("  vs oracle", errors(got, ref))
        assert_parity(got, ref)


def test_noalloc_rejects_batches_beyond_its_scratch(hb, monkeypatch):
    import torch
    from hb_workloads import make_batch, make_weights
    from paper_2503_22562_amd import hb as H
    from paper_2503_22562_amd.harness import bf16_bits, to_device_bf16
    monkeypatch.setenv("HB_GEMM_KSPLIT", "8")  # 8 x 2048 x 2 x 2560 fp32 gate/up partials: 335 MB
    w = make_weights(COVER)
    b = make_batch(COVER, [(2048, 0)], seed=63, num_blocks=256)
    dl = _layer(b, w, b.n_tokens, 1)
    k0, v0 = bf16_bits(dl.k_pool), bf16_bits(dl.v_pool)
    x = to_device_bf16(b.x_in())
    y = torch.full((b.n_tokens, COVER.hidden), 7.0, dtype=torch.float32, device="cuda")
    with pytest.raises(H.HBError) as e:
        H.hb_run_iteration_noalloc(dl.layer, [(q.chunk_len, q.context_len, q.block_table) for q in b.requests], x, y)
    assert e.value.status == H.HB_ERR_UNSUPPORTED and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert np.array_equal(bf16_bits(dl.k_pool), k0) and np.array_equal(bf16_bits(dl.v_pool), v0)
    assert torch.all(y == 7.0)
