"""Coverage of the GEMM launch grid: every (tile shape, K split) the planner
picks for the full-size configurations is one that the forced-grid GPU test
runs on the cover shape (host check), and that GPU test runs every pair of
the grid through whole-layer parity with per-step checks."""
import numpy as np
import pytest

import oracle
from gemmcover import COVER, COVER_LENS, COVER_T, CU_COUNT, MAX_KSPLIT, real_token_counts
from hbref import assert_parity, assert_stage, assert_swiglu_stage, errors, oracle_for_batch


@pytest.fixture(scope="module")
def H():
    from paper_2503_22562_amd import hb
    hb.load()
    return hb


def test_planner_picks_are_forced_on_the_cover_shape(H):
    """For each GEMM of each full-size configuration, forcing the planner's
    (tile, split) on the cover shape reproduces it, so the forced-grid GPU
    test launches exactly those kernel instantiations."""
    cover = H.make_config(COVER, COVER_T, 16)
    picks = set()
    for shape, T in real_token_counts():
        cfg = H.make_config(shape, 4096, 512)
        for g, (tile, ks) in enumerate(H.hb_plan_gemms(cfg, T, CU_COUNT)):
            picks.add((g, tile, ks))
    assert picks
    for g, tile, ks in sorted(picks):
        assert 1 <= ks <= MAX_KSPLIT
        assert H.hb_plan_gemms(cover, COVER_T, CU_COUNT, tile, ks)[g] == (tile, ks), (g, tile, ks)


_REF = {}


def _reference():
    if not _REF:
        from hb_workloads import make_batch, make_weights
        b = make_batch(COVER, COVER_LENS, seed=37, num_blocks=96)
        w = make_weights(COVER)
        w64 = oracle.weights_to_f64(w)
        ref, st = oracle_for_batch(b, w64, stages=True)
        _REF.update(batch=b, w=w, w64=w64, ref=ref, st=st)
    return _REF


@pytest.mark.gpu
@pytest.mark.parametrize("ksplit", list(range(1, MAX_KSPLIT + 1)))
def test_forced_grid_parity(H, monkeypatch, ksplit):
    """Every tile shape at this K split on all four GEMMs (QKV + RoPE + pool
    scatter, O + residual (+ fused pre-FFN RMSNorm when split), gate/up +
    SwiGLU, down + residual): the plan that ran is the forced one (relaxed
    only where the pair cannot run that GEMM, exactly as the host planner
    relaxes it), and y, q, the attention output, h2 and silu(gate)*up match
    the oracle."""
    import torch
    from paper_2503_22562_amd.harness import DeviceLayer, bf16_bits, to_device_bf16
    r = _reference()
    b, w, w64, ref, st = r["batch"], r["w"], r["w64"], r["ref"], r["st"]
    cover = H.make_config(COVER, COVER_T, 16)
    x = to_device_bf16(b.x_in())
    reqs = [(q.chunk_len, q.context_len, q.block_table) for q in b.requests]
    T = b.n_tokens
    for tile in range(H.hb_gemm_tile_count()):
        monkeypatch.setenv("HB_GEMM_TILE", str(tile))
        monkeypatch.setenv("HB_GEMM_KSPLIT", str(ksplit))
        dl = DeviceLayer(COVER, w, b.num_blocks, T, len(reqs))
        for i, q in enumerate(b.requests):
            if q.context_len:
                k, v = b.prior_kv(i)
                dl.append_kv(q.block_table, 0, k, v)
        y = dl.run(reqs, x)
        torch.cuda.synchronize()
        ran = H.hb_layer_gemm_plans(dl.layer)
        assert ran == H.hb_plan_gemms(cover, T, dl_cu(), tile, ksplit), (tile, ksplit, ran)
        what = f"tile {tile} ksplit {ksplit} plans {ran}"
        y = y.cpu().numpy().astype(np.float64)
        print(what, errors(y, ref))
        assert_parity(y, ref, what + " y")
        q = oracle.bf16_bits_to_f64(bf16_bits(dl.stage(H.HB_STAGE_Q, T)))
        assert_stage(q, st["q"].reshape(T, -1), what + " q after RoPE")
        o = oracle.bf16_bits_to_f64(bf16_bits(dl.stage(H.HB_STAGE_ATTN, T)))
        assert_stage(o, st["o"], what + " attention output")
        h2 = dl.stage(H.HB_STAGE_H2, T).cpu().numpy()
        assert_parity(h2, st["h2"], what + " h2")
        m = oracle.bf16_bits_to_f64(bf16_bits(dl.stage(H.HB_STAGE_MLP, T)))
        assert_swiglu_stage(m, st, w64, COVER.rms_eps, what + " silu(gate)*up")
        del dl


def dl_cu():
    import torch
    return torch.cuda.get_device_properties(0).multi_processor_count
