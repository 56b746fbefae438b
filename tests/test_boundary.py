"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every entry point include/hb.h declares, and rejects malformed batches with
the documented status before any device work (hb_validate_batch makes no HIP
call)."""
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def H():
    from paper_2503_22562_amd import hb
    try:
        hb.load()
    except RuntimeError as e:
        pytest.fail(str(e))
    return hb


def declared_functions():
    text = open(os.path.join(ROOT, "include", "hb.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hb_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("hb_create_layer", "hb_append_kv", "hb_run_iteration", "hb_profile", "hb_destroy_layer",
              "hb_validate_batch", "hb_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol(H):
    lib = H.load()
    for n in declared_functions():
        assert hasattr(lib, n), f"libhb.so does not export {n}"
    assert set(declared_functions()) == set(H.EXPORTED)


def test_kernel_names(H):
    names = [H.hb_kernel_name(k) for k in range(H.HB_K_COUNT)]
    assert len(set(names)) == H.HB_K_COUNT and "attention" in names
    assert H.hb_kernel_name(99) == "unknown"


class Shape:
    hidden, n_q_heads, n_kv_heads, head_dim, ffn_dim = 256, 4, 2, 64, 688
    rope_theta, rms_eps, kv_block = 5e5, 1e-5, 16


X_IN, X_OUT = 0x10000000, 0x20000000  # fake device addresses: never dereferenced


def _v(H, reqs, num_blocks=64, max_T=128, max_R=8, shape=Shape, x_in=X_IN, x_out=X_OUT, out_dtype=0):
    cfg = H.make_config(shape, max_T, max_R)
    return H.hb_validate_batch(cfg, num_blocks, reqs, x_in, x_out, out_dtype)


def bt(*ids):
    return np.array(ids, dtype=np.int32)


def test_valid_batches(H):
    assert _v(H, []) == H.HB_OK
    assert _v(H, [(64, 128, np.arange(12)), (1, 256, np.arange(20, 37))]) == H.HB_OK
    # shared read-only prefix blocks, distinct written slots
    assert _v(H, [(1, 16, bt(3, 4)), (1, 16, bt(3, 5))]) == H.HB_OK
    # two requests writing different slots of one block
    assert _v(H, [(1, 3, bt(7)), (1, 4, bt(7))]) == H.HB_OK


@pytest.mark.parametrize("reqs,status", [
    ([(0, 0, bt(1))], "INVALID"),                       # chunk_len < 1
    ([(1, -1, bt(1))], "INVALID"),                      # context_len < 0
    ([(17, 0, bt(1))], "INVALID"),                      # block table too short
    ([(1, 16, bt(1))], "INVALID"),                      # position 16 needs a second block
    ([(1, 0, bt(64))], "RANGE"),                        # block id == num_blocks
    ([(1, 0, bt(-1))], "RANGE"),                        # negative block id
    ([(1, 5, bt(2)), (1, 5, bt(2))], "INVALID"),        # two tokens, one slot
    ([(4, 0, bt(2)), (1, 3, bt(2))], "INVALID"),        # chunk overlaps a decode's slot
    ([(129, 0, np.arange(9))], "INVALID"),              # T above max_batch_tokens
    ([(1, 0, bt(i)) for i in range(9)], "INVALID"),     # above max_requests
])
def test_invalid_batches(H, reqs, status):
    assert _v(H, reqs) == getattr(H, "HB_ERR_" + status)
    assert H.hb_last_error()


def test_pointer_and_dtype_errors(H):
    r = [(2, 0, bt(1))]
    assert _v(H, r, x_in=0) == H.HB_ERR_INVALID
    assert _v(H, r, x_out=0) == H.HB_ERR_INVALID
    assert _v(H, r, out_dtype=7) == H.HB_ERR_INVALID
    # x_out overlapping x_in
    assert _v(H, r, x_out=X_IN + 256) == H.HB_ERR_INVALID
    assert _v(H, r, x_out=X_IN + 2 * 256 * 2) == H.HB_OK


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 96, "UNSUPPORTED"),
    ("kv_block", 32, "UNSUPPORTED"),
    ("n_kv_heads", 3, "UNSUPPORTED"),
    ("hidden", 200, "UNSUPPORTED"),
    ("ffn_dim", 100, "UNSUPPORTED"),
    ("hidden", 0, "INVALID"),
])
def test_config_errors(H, field, value, status):
    shape = type("S", (Shape,), {field: value})
    assert _v(H, [(1, 0, bt(1))], shape=shape) == getattr(H, "HB_ERR_" + status)


WINDOW = 0x7FFFFFF0  # bytes the GEMMs address in one operand


def _llama(H, max_T, **kw):
    """hb_validate_batch of a one-token batch under a Llama-shaped config."""
    base = dict(hidden=8192, n_q_heads=64, n_kv_heads=8, head_dim=128, ffn_dim=28672, rope_theta=5e5, rms_eps=1e-5,
                kv_block=16)
    base.update(kw)
    shape = type("S", (), base)
    return _v(H, [(1, 0, bt(1))], shape=shape, max_T=max_T)


def test_operand_window_limits(H):
    """Every GEMM operand must fit the 2^31 - 16-byte buffer window: the
    largest max_batch_tokens the 70B shape admits is the one whose SwiGLU
    activations ((max_T + 512) x 28672 bf16) still fit; one more token is
    rejected before any device work."""
    F = 28672
    limit = WINDOW // (2 * F) - 512
    assert _llama(H, limit) == H.HB_OK
    assert _llama(H, limit + 1) == H.HB_ERR_UNSUPPORTED
    assert "window" in H.hb_last_error()
    # the 8B shape: hidden 4096, ffn 14336
    lim8 = WINDOW // (2 * 14336) - 512
    assert _llama(H, lim8, hidden=4096, n_q_heads=32, ffn_dim=14336) == H.HB_OK
    assert _llama(H, lim8 + 1, hidden=4096, n_q_heads=32, ffn_dim=14336) == H.HB_ERR_UNSUPPORTED
    # weight matrices: gate/up (2F x H) and down (H x F) past the window
    assert _llama(H, 16, hidden=16384, ffn_dim=53248) == H.HB_ERR_UNSUPPORTED
    assert "w_gate_up" in H.hb_last_error()
    assert _llama(H, 16, hidden=16384, ffn_dim=32768 + 16) == H.HB_ERR_UNSUPPORTED  # down: 16384 x F * 2 B
    assert _llama(H, 16, hidden=16384, ffn_dim=32768 - 512) == H.HB_OK
    # QKV weights: (nq + 2 nkv) hd x H
    assert _llama(H, 16, hidden=16384, n_q_heads=512, n_kv_heads=32, ffn_dim=1024) == H.HB_ERR_UNSUPPORTED
    assert "w_qkv" in H.hb_last_error()


def test_gqa_group_must_divide_16(H):
    shape = type("S", (Shape,), {"n_q_heads": 32, "n_kv_heads": 1})
    assert _v(H, [(1, 0, bt(1))], shape=shape) == H.HB_ERR_UNSUPPORTED


def _create_model(H, n_layers=2, vocab=64, pool_blocks=(64, 64), null_embed=False):
    """hb_create_model with fake device addresses: every case here must be
    rejected before any HIP call."""
    import ctypes as C
    cfg = H.make_config(Shape, 128, 8)
    n = max(n_layers, 1)
    wa = (H.hb_layer_weights * n)()
    pa = (H.hb_kv_pool * n)()
    for i in range(n):
        wa[i] = H.hb_layer_weights(*[0x1000 * (j + 1) for j in range(6)])
        pa[i] = H.hb_kv_pool(0x30000000, 0x40000000, pool_blocks[i % len(pool_blocks)])
    d = H.hb_model_desc(n_layers, vocab, wa, pa, C.c_void_p(0 if null_embed else 0x50000000),
                        C.c_void_p(0x60000000), C.c_void_p(0x70000000))
    h = C.c_void_p()
    st = H.load().hb_create_model(C.byref(cfg), C.byref(d), None, C.byref(h))
    assert not h.value
    return st


@pytest.mark.parametrize("kw", [dict(n_layers=0), dict(vocab=60), dict(vocab=0), dict(pool_blocks=(64, 32)),
                                dict(null_embed=True)], ids=str)
def test_model_argument_errors(H, kw):
    assert _create_model(H, **kw) == H.HB_ERR_INVALID
    assert H.hb_last_error()


def test_model_lm_head_window(H):
    """The LM head (vocab x H bf16) is a GEMM operand: past the 2 GiB window
    the model is rejected before any HIP call."""
    vocab = (WINDOW // (2 * Shape.hidden) + 8) // 8 * 8
    assert _create_model(H, vocab=vocab) == H.HB_ERR_UNSUPPORTED
    assert "lm_head" in H.hb_last_error()


def test_gemm_plans_host_only(H):
    """The GEMM planner runs on the host: plans for the 8B shape are valid
    tile indices and K splits, and every (tile, split) is a launch the
    kernels implement."""
    from hb_workloads import LLAMA3_8B
    cfg = H.make_config(LLAMA3_8B, 4096, 512)
    n = H.hb_gemm_tile_count()
    from test_gpu_tiny import GEMM_TILE_SHAPES
    assert n == GEMM_TILE_SHAPES  # the forced-tile GPU test runs every shape
    for T in (1, 64, 128, 576, 2048, 4096):
        for tile, ks in H.hb_plan_gemms(cfg, T, 256):
            assert 0 <= tile < n and 1 <= ks <= 8
    with pytest.raises(H.HBError):
        H.hb_plan_gemms(cfg, 0, 256)


def test_model_layer_of_null_model(H):
    assert not H.load().hb_model_layer(None, 0)


@pytest.mark.parametrize("hd", [64, 128])
def test_pool_layout_views(hd):
    """The pool layouts hb.h documents, written out element by element, are
    what the harness's per-slot views undo: K of slot s, dimension d at
    [(s/4)%2][d/8][4(s/8) + s%4][d%8]; V at [s/8][d][s%8]."""
    from paper_2503_22562_amd.harness import k_by_slot, v_by_slot
    nb, nkv = 3, 2
    want = np.random.default_rng(hd).integers(0, 1 << 16, (nb, nkv, 16, hd)).astype(np.uint16)
    k = np.zeros((nb, nkv, 2, hd // 8, 8, 8), np.uint16)
    v = np.zeros((nb, nkv, 2, hd, 8), np.uint16)
    for s in range(16):
        for d in range(hd):
            k[:, :, (s // 4) % 2, d // 8, 4 * (s // 8) + s % 4, d % 8] = want[:, :, s, d]
            v[:, :, s // 8, d, s % 8] = want[:, :, s, d]
    assert np.array_equal(k_by_slot(k.reshape(nb, nkv, 16, hd)), want)
    assert np.array_equal(v_by_slot(v), want)


def test_device_rates_argument_errors(H):
    """hb_measure_device_rates rejects a null buffer or output and a buffer
    below 1 GiB before touching a device."""
    import ctypes as C
    out = H.hb_device_rates()
    lib = H.load()
    assert lib.hb_measure_device_rates(None, 1 << 30, None, C.byref(out)) == H.HB_ERR_INVALID
    assert lib.hb_measure_device_rates(C.c_void_p(4096), (1 << 30) - 1, None, C.byref(out)) == H.HB_ERR_INVALID
    assert lib.hb_measure_device_rates(C.c_void_p(4096), 1 << 30, None, None) == H.HB_ERR_INVALID
    assert "1 GiB" in H.hb_last_error()
