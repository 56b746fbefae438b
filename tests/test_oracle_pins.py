"""Pins of the CPU oracle against things other than itself: closed forms,
brute force on tiny inputs, special cases, a textbook library implementation
of the Llama decoder layer (HF transformers, fp64, dense causal attention) and
the invariants the method guarantees (chunking, paging and batching only
regroup the per-request computation)."""
import math

import numpy as np
import pytest
import torch

import oracle
from hb_workloads import TINY, f32_to_bf16_bits, make_batch, make_weights

RNG = np.random.default_rng(1234)


class Cfg:
    def __init__(self, hidden=64, nq=4, nkv=2, hd=16, ffn=96, theta=5e5, eps=1e-5, block=16):
        self.hidden, self.n_q_heads, self.n_kv_heads, self.head_dim = hidden, nq, nkv, hd
        self.ffn_dim, self.rope_theta, self.rms_eps, self.kv_block = ffn, theta, eps, block


def rand_weights(cfg, rng):
    h, hd, nq, nkv, f = cfg.hidden, cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads, cfg.ffn_dim
    return {
        "w_qkv": rng.standard_normal(((nq + 2 * nkv) * hd, h)) / math.sqrt(h),
        "w_o": rng.standard_normal((h, nq * hd)) / math.sqrt(nq * hd),
        "w_gate_up": rng.standard_normal((2 * f, h)) / math.sqrt(h),
        "w_down": rng.standard_normal((h, f)) / math.sqrt(f),
        "g_attn": 1 + 0.1 * rng.standard_normal(h),
        "g_ffn": 1 + 0.1 * rng.standard_normal(h),
    }


class Req:
    def __init__(self, chunk, ctx, bt):
        self.chunk_len, self.context_len, self.block_table = chunk, ctx, np.asarray(bt)


# ---------------------------------------------------------------- input decoding
def test_bf16_decode_known_patterns():
    bits = np.array([0x3F80, 0xC000, 0x3F81, 0x0000, 0x8000, 0x4049, 0x7F7F], dtype=np.uint16)
    want = [1.0, -2.0, 1.0 + 2 ** -7, 0.0, -0.0, 3.140625, 3.3895313892515355e38]
    got = oracle.bf16_bits_to_f64(bits)
    assert got.dtype == np.float64
    assert list(got) == want


def test_bf16_roundtrip_of_generator_is_exact():
    a = RNG.standard_normal(1000).astype(np.float32)
    bits = f32_to_bf16_bits(a)
    v = oracle.bf16_bits_to_f64(bits)
    # RNE: |v - a| <= half an ulp of bf16 (2^-8 relative)
    assert np.all(np.abs(v - a) <= np.abs(a) * 2.0 ** -8 + 1e-45)


# ---------------------------------------------------------------- RMSNorm
def test_rmsnorm_constant_vector_closed_form():
    for c in (3.0, -0.5, 1e-3):
        x = np.full((1, 32), c)
        g = np.linspace(0.5, 1.5, 32)
        eps = 1e-5
        want = g * c / math.sqrt(c * c + eps)
        np.testing.assert_allclose(oracle.rmsnorm(x, g, eps)[0], want, rtol=1e-14)


def test_rmsnorm_matches_library_routine():
    x = RNG.standard_normal((5, 48))
    g = RNG.standard_normal(48)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (48,), torch.from_numpy(g), eps=1e-5).numpy()
    np.testing.assert_allclose(oracle.rmsnorm(x, g, 1e-5), ref, rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------- linear
def test_linear_brute_force_nonsquare():
    a = RNG.standard_normal((3, 5))
    w = RNG.standard_normal((4, 5))  # [out][in]
    want = np.zeros((3, 4))
    for i in range(3):
        for o in range(4):
            want[i, o] = sum(a[i, k] * w[o, k] for k in range(5))
    np.testing.assert_allclose(oracle.linear(a, w), want, rtol=1e-13)


# ---------------------------------------------------------------- RoPE
def test_rope_position_zero_is_identity():
    z = RNG.standard_normal((1, 3, 8))
    np.testing.assert_array_equal(oracle.rope(z, np.array([0]), 5e5), z)


def test_rope_two_dim_closed_form():
    # hd = 2: a single pair with omega_0 = theta^0 = 1 -> rotation by p radians.
    for p in (1, 2, 7):
        out = oracle.rope(np.array([[[1.0, 0.0], [0.0, 1.0]]]), np.array([p]), 5e5)[0]
        np.testing.assert_allclose(out[0], [math.cos(p), math.sin(p)], atol=1e-15)
        np.testing.assert_allclose(out[1], [-math.sin(p), math.cos(p)], atol=1e-15)


def test_rope_equals_complex_rotation_and_keeps_pair_norms():
    hd, theta = 16, 10000.0
    z = RNG.standard_normal((4, 2, hd))
    pos = np.array([0, 3, 100, 4095])
    out = oracle.rope(z, pos, theta)
    half = hd // 2
    zc = z[..., :half] + 1j * z[..., half:]
    omega = np.array([theta ** (-2 * j / hd) for j in range(half)])
    rot = zc * np.exp(1j * pos[:, None, None] * omega[None, None, :])
    np.testing.assert_allclose(out[..., :half], rot.real, atol=1e-12)
    np.testing.assert_allclose(out[..., half:], rot.imag, atol=1e-12)
    np.testing.assert_allclose(np.abs(out[..., :half] + 1j * out[..., half:]), np.abs(zc), rtol=1e-13)


def test_rope_relative_position_property():
    hd = 32
    q = RNG.standard_normal((1, 1, hd))
    k = RNG.standard_normal((1, 1, hd))
    def dot(pq, pk):
        return float(np.sum(oracle.rope(q, np.array([pq]), 5e5) * oracle.rope(k, np.array([pk]), 5e5)))
    base = dot(10, 3)
    for shift in (1, 17, 1000):
        assert abs(dot(10 + shift, 3 + shift) - base) < 1e-10


def test_rope_matches_hf_llama():
    from transformers.models.llama.modeling_llama import apply_rotary_pos_emb
    hd, theta = 64, 5e5
    z = RNG.standard_normal((1, 3, 6, hd))  # [b, heads, seq, hd]
    pos = np.array([0, 1, 5, 17, 128, 300])
    phi = oracle.rope_angles(pos, hd, theta)
    emb = np.concatenate([phi, phi], axis=-1)[None]
    cos, sin = torch.from_numpy(np.cos(emb)), torch.from_numpy(np.sin(emb))
    qh, _ = apply_rotary_pos_emb(torch.from_numpy(z), torch.from_numpy(z), cos, sin)
    ours = oracle.rope(z[0].transpose(1, 0, 2), pos, theta).transpose(1, 0, 2)
    np.testing.assert_allclose(ours, qh.numpy()[0], rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------------- SiLU / MLP
def test_silu_closed_forms():
    assert oracle.silu(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(oracle.silu(np.array([40.0])), [40.0], rtol=1e-15)
    assert abs(oracle.silu(np.array([-40.0]))[0]) < 1e-15
    np.testing.assert_allclose(oracle.silu(np.array([1.0])), [1 / (1 + math.exp(-1))], rtol=1e-15)
    z = RNG.standard_normal(100) * 4
    np.testing.assert_allclose(oracle.silu(z), torch.nn.functional.silu(torch.from_numpy(z)).numpy(), rtol=1e-14)


def test_swiglu_gate_and_up_halves_not_swapped():
    f = RNG.standard_normal((2, 6))
    wg, wu = RNG.standard_normal((3, 6)), RNG.standard_normal((3, 6))
    wd = RNG.standard_normal((6, 3))
    want = (oracle.silu(f @ wg.T) * (f @ wu.T)) @ wd.T
    got = oracle.swiglu_mlp(f, np.concatenate([wg, wu]), wd)
    np.testing.assert_allclose(got, want, rtol=1e-13)
    swapped = oracle.swiglu_mlp(f, np.concatenate([wu, wg]), wd)
    assert np.max(np.abs(swapped - want)) > 1e-3


# ---------------------------------------------------------------- attention
def brute_attention(q, k, v, q_pos, nkv):
    rows, nq, hd = q.shape
    out = np.zeros_like(q)
    for i in range(rows):
        for h in range(nq):
            g = h // (nq // nkv)
            s = [sum(q[i, h, d] * k[j, g, d] for d in range(hd)) / math.sqrt(hd) for j in range(q_pos[i] + 1)]
            mx = max(s)
            e = [math.exp(x - mx) for x in s]
            z = sum(e)
            for d in range(hd):
                out[i, h, d] = sum(e[j] * v[j, g, d] for j in range(len(e))) / z
    return out


def test_attention_brute_force_gqa():
    nq, nkv, hd, n = 4, 2, 8, 11
    k = RNG.standard_normal((n, nkv, hd))
    v = RNG.standard_normal((n, nkv, hd))
    q_pos = np.array([0, 4, 9, 10])
    q = RNG.standard_normal((4, nq, hd))
    np.testing.assert_allclose(oracle.causal_attention(q, k, v, q_pos, nkv), brute_attention(q, k, v, q_pos, nkv), rtol=1e-12, atol=1e-13)


def test_attention_special_cases():
    nq, nkv, hd, n = 2, 1, 8, 9
    k = RNG.standard_normal((n, nkv, hd))
    v = RNG.standard_normal((n, nkv, hd))
    q = RNG.standard_normal((1, nq, hd))
    # first position sees only itself: output is v_0 exactly
    o = oracle.causal_attention(q, k, v, np.array([0]), nkv)
    np.testing.assert_array_equal(o[0, 0], v[0, 0])
    # all keys equal: output is the mean of the visible values
    keq = np.repeat(k[:1], n, axis=0)
    o = oracle.causal_attention(q, keq, v, np.array([5]), nkv)
    np.testing.assert_allclose(o[0, 1], v[:6, 0].mean(axis=0), rtol=1e-12)
    # one dominant key: output is that key's value
    kd = np.zeros_like(k)
    kd[3, 0] = 50.0 * q[0, 0] / np.linalg.norm(q[0, 0])
    o = oracle.causal_attention(q, kd, v, np.array([7]), nkv)
    np.testing.assert_allclose(o[0, 0], v[3, 0], atol=1e-12)
    # keys after the query position are invisible
    o1 = oracle.causal_attention(q, k, v, np.array([4]), nkv)
    k2, v2 = k.copy(), v.copy()
    k2[5:] = 100.0
    v2[5:] = -7.0
    np.testing.assert_array_equal(o1, oracle.causal_attention(q, k2, v2, np.array([4]), nkv))


# ---------------------------------------------------------------- paged cache
def test_kv_slot_brute_force():
    bt = [7, 2, 9, 0]
    for p in range(64):
        assert oracle.kv_slot(bt, p) == (bt[p // 16], p - 16 * (p // 16))


def test_cache_roundtrip_and_isolation():
    c = oracle.PagedKVCache(32, 2, 4)
    bt = [5, 9, 1]
    k = RNG.standard_normal((40, 2, 4))
    v = RNG.standard_normal((40, 2, 4))
    c.write(bt, 0, k[:23], v[:23])
    c.write(bt, 23, k[23:], v[23:])
    kk, vv = c.read(bt, 40)
    np.testing.assert_array_equal(kk, k)
    np.testing.assert_array_equal(vv, v)
    assert sorted(c.k) == [1, 5, 9]
    with pytest.raises(IndexError):
        c.write([40], 0, k[:1], v[:1])


# ---------------------------------------------------------------- whole layer vs textbook
def hf_layer(cfg, w):
    from transformers import LlamaConfig
    from transformers.models.llama.modeling_llama import LlamaDecoderLayer
    hc = LlamaConfig(hidden_size=cfg.hidden, num_attention_heads=cfg.n_q_heads,
                     num_key_value_heads=cfg.n_kv_heads, head_dim=cfg.head_dim,
                     intermediate_size=cfg.ffn_dim, rms_norm_eps=cfg.rms_eps,
                     attention_bias=False, mlp_bias=False, max_position_embeddings=8192)
    hc._attn_implementation = "eager"
    layer = LlamaDecoderLayer(hc, layer_idx=0).double()
    nq, nkv, hd, f = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.ffn_dim
    sd = {
        "self_attn.q_proj.weight": w["w_qkv"][: nq * hd],
        "self_attn.k_proj.weight": w["w_qkv"][nq * hd:(nq + nkv) * hd],
        "self_attn.v_proj.weight": w["w_qkv"][(nq + nkv) * hd:],
        "self_attn.o_proj.weight": w["w_o"],
        "mlp.gate_proj.weight": w["w_gate_up"][:f],
        "mlp.up_proj.weight": w["w_gate_up"][f:],
        "mlp.down_proj.weight": w["w_down"],
        "input_layernorm.weight": w["g_attn"],
        "post_attention_layernorm.weight": w["g_ffn"],
    }
    layer.load_state_dict({k: torch.from_numpy(np.ascontiguousarray(v)) for k, v in sd.items()})

    def run(x):
        L = x.shape[0]
        pos = np.arange(L)
        phi = oracle.rope_angles(pos, hd, cfg.rope_theta)
        emb = np.concatenate([phi, phi], axis=-1)[None]
        cos, sin = torch.from_numpy(np.cos(emb)), torch.from_numpy(np.sin(emb))
        mask = torch.full((L, L), float("-inf"), dtype=torch.float64).triu(1)[None, None]
        with torch.no_grad():
            y = layer(torch.from_numpy(x)[None], attention_mask=mask,
                      position_ids=torch.from_numpy(pos)[None], position_embeddings=(cos, sin))
        y = y[0] if isinstance(y, tuple) else y
        return y[0].numpy()
    return run


@pytest.mark.parametrize("nq,nkv,hd", [(4, 2, 16), (4, 1, 32), (2, 2, 8)])
def test_layer_matches_textbook_dense_layer(nq, nkv, hd):
    cfg = Cfg(hidden=64, nq=nq, nkv=nkv, hd=hd, ffn=96)
    rng = np.random.default_rng(nq * 100 + nkv * 10 + hd)
    w = rand_weights(cfg, rng)
    run_hf = hf_layer(cfg, w)
    # two prompts, processed as a sequence of hybrid iterations
    la, lb = 45, 20
    xa = rng.standard_normal((la, cfg.hidden))
    xb = rng.standard_normal((lb, cfg.hidden))
    ya_ref, yb_ref = run_hf(xa), run_hf(xb)
    cache = oracle.PagedKVCache(64, nkv, hd)
    bta, btb = [11, 3, 40], [7, 30]
    ya, yb = [], []
    # iteration 1: chunk A[0:13); iteration 2: A[13:29) + B[0:19); iteration 3: A[29:45) + decode B[19]
    for (ca, oa), (cb, ob) in [((13, 0), (0, 0)), ((16, 13), (19, 0)), ((16, 29), (1, 19))]:
        reqs, xs = [Req(ca, oa, bta)], [xa[oa:oa + ca]]
        if cb:
            reqs.append(Req(cb, ob, btb))
            xs.append(xb[ob:ob + cb])
        y = oracle.layer_forward(w, cfg, cache, reqs, np.concatenate(xs))
        ya.append(y[:ca])
        if cb:
            yb.append(y[ca:])
    np.testing.assert_allclose(np.concatenate(ya), ya_ref, rtol=1e-5, atol=2e-5)
    np.testing.assert_allclose(np.concatenate(yb), yb_ref, rtol=1e-5, atol=2e-5)


# ---------------------------------------------------------------- invariants
def _tiny_setup(seed=7):
    cfg = Cfg(hidden=64, nq=4, nkv=2, hd=16, ffn=96)
    rng = np.random.default_rng(seed)
    return cfg, rng, rand_weights(cfg, rng)


def test_chunk_split_equals_unsplit_including_mid_block():
    cfg, rng, w = _tiny_setup()
    x = rng.standard_normal((70, cfg.hidden))
    bt = [3, 17, 9, 22, 5]
    c1 = oracle.PagedKVCache(32, 2, 16)
    y_full = oracle.layer_forward(w, cfg, c1, [Req(70, 0, bt)], x)
    c2 = oracle.PagedKVCache(32, 2, 16)
    parts, y_parts = [(0, 7), (7, 30), (30, 31), (31, 70)], []
    for s, e in parts:
        y_parts.append(oracle.layer_forward(w, cfg, c2, [Req(e - s, s, bt)], x[s:e]))
    np.testing.assert_allclose(np.concatenate(y_parts), y_full, rtol=1e-12, atol=1e-12)
    k1, v1 = c1.read(bt, 70)
    k2, v2 = c2.read(bt, 70)
    np.testing.assert_allclose(k2, k1, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(v2, v1, rtol=1e-12, atol=1e-13)


def test_permuted_block_table_gives_same_output():
    cfg, rng, w = _tiny_setup(8)
    ctx, chunk = 37, 9
    kp = rng.standard_normal((ctx, 2, 16))
    vp = rng.standard_normal((ctx, 2, 16))
    x = rng.standard_normal((chunk, cfg.hidden))
    outs = []
    for bt in ([0, 1, 2], [29, 4, 11]):
        c = oracle.PagedKVCache(32, 2, 16)
        c.write(bt, 0, kp, vp)
        outs.append(oracle.layer_forward(w, cfg, c, [Req(chunk, ctx, bt)], x))
    np.testing.assert_array_equal(outs[0], outs[1])


def test_decode_equals_one_token_chunk_and_batch_independence():
    cfg, rng, w = _tiny_setup(9)
    ctxs = [20, 33, 5]
    bts = [[1, 2], [3, 4, 5], [6]]
    prior = [(rng.standard_normal((c, 2, 16)), rng.standard_normal((c, 2, 16))) for c in ctxs]
    xs = rng.standard_normal((3, cfg.hidden))

    def fresh():
        c = oracle.PagedKVCache(16, 2, 16)
        for bt, (k, v), n in zip(bts, prior, ctxs):
            c.write(bt, 0, k, v)
        return c
    y_batch = oracle.layer_forward(w, cfg, fresh(), [Req(1, c, bt) for c, bt in zip(ctxs, bts)], xs)
    for i in range(3):
        y_one = oracle.layer_forward(w, cfg, fresh(), [Req(1, ctxs[i], bts[i])], xs[i:i + 1])
        np.testing.assert_allclose(y_batch[i], y_one[0], rtol=1e-12, atol=1e-13)
    # reordering the requests permutes the output rows
    order = [2, 0, 1]
    y_perm = oracle.layer_forward(w, cfg, fresh(), [Req(1, ctxs[i], bts[i]) for i in order], xs[order])
    np.testing.assert_allclose(y_perm, y_batch[order], rtol=1e-12, atol=1e-13)


def test_row_sampling_equals_full_rows():
    cfg, rng, w = _tiny_setup(10)
    x = rng.standard_normal((12, cfg.hidden))
    reqs = [Req(8, 0, [0]), Req(1, 0, [1]), Req(3, 0, [2])]
    y = oracle.layer_forward(w, cfg, oracle.PagedKVCache(4, 2, 16), reqs, x)
    ys = oracle.layer_forward(w, cfg, oracle.PagedKVCache(4, 2, 16), reqs, x, rows=[2, 7, 8, 11])
    np.testing.assert_allclose(ys, y[[2, 7, 8, 11]], rtol=1e-12, atol=1e-13)


def test_tiny_workload_runs_through_oracle():
    from hb_workloads import tiny_batch
    b = tiny_batch()
    w = oracle.weights_to_f64(make_weights(TINY))
    cache = oracle.PagedKVCache(b.num_blocks, TINY.n_kv_heads, TINY.head_dim)
    oracle.seed_cache(cache, b.requests, lambda r: tuple(oracle.bf16_bits_to_f64(a) for a in b.prior_kv(r)))
    y = oracle.layer_forward(w, TINY, cache, b.requests, oracle.bf16_bits_to_f64(b.x_in()))
    assert y.shape == (72, 256) and np.all(np.isfinite(y))


def test_round_bf16_matches_torch_and_ties_to_even():
    """The model oracle's inter-layer rounding equals torch's bfloat16
    conversion (a library routine, RNE) on random and edge values."""
    import torch
    from oracle.model import round_bf16
    rng = np.random.default_rng(7)
    x = np.concatenate([rng.standard_normal(10000) * 10 ** rng.uniform(-6, 6, 10000),
                        [0.0, -0.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 65504.0, 1e-40]])
    want = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(round_bf16(x), want)


def test_model_chunk_split_equals_unsplit():
    """Whole-model invariant: a prompt processed in one chunk or in two gives
    the same last-token logits (every layer's cache holds the first chunk's
    K/V when the second runs)."""
    from hb_workloads import make_batch, make_model_weights
    from oracle.model import model_forward
    shape = TINY
    mw = make_model_weights(shape, 2, 64)
    lw = [oracle.weights_to_f64(w) for w in mw["layers"]]
    emb, head = oracle.bf16_bits_to_f64(mw["embed"]), oracle.bf16_bits_to_f64(mw["lm_head"])
    g = oracle.bf16_bits_to_f64(mw["g_final"])
    b = make_batch(shape, [(48, 0)], seed=5, num_blocks=64)
    ids = b.token_ids(64)
    req = b.requests[0]

    def caches():
        return [oracle.PagedKVCache(64, shape.n_kv_heads, shape.head_dim) for _ in lw]

    whole, _ = model_forward(shape, lw, caches(), emb, g, head, b.requests, ids)
    cs = caches()
    first = [type(req)(30, 0, req.block_table)]
    second = [type(req)(18, 30, req.block_table)]
    model_forward(shape, lw, cs, emb, g, head, first, ids[:30])
    split, _ = model_forward(shape, lw, cs, emb, g, head, second, ids[30:])
    assert np.allclose(whole, split, rtol=0, atol=1e-9)


def test_model_matches_textbook_causal_lm():
    """The model oracle with fp64 hidden states between layers equals HF
    transformers' LlamaForCausalLM (fp64, eager, untied head) on the last
    token's logits: one prompt as a single chunk, and the same prompt as two
    iterations (a chunk, then the rest beside a decode of another request)."""
    from transformers import LlamaConfig, LlamaForCausalLM
    from oracle.model import model_forward
    cfg = Cfg(hidden=64, nq=4, nkv=2, hd=16, ffn=96)
    vocab, n_layers = 48, 2
    rng = np.random.default_rng(1234)
    lw = [rand_weights(cfg, rng) for _ in range(n_layers)]
    embed = rng.standard_normal((vocab, cfg.hidden))
    head = rng.standard_normal((vocab, cfg.hidden)) / np.sqrt(cfg.hidden)
    g_final = 1.0 + 0.1 * rng.standard_normal(cfg.hidden)
    hc = LlamaConfig(vocab_size=vocab, hidden_size=cfg.hidden, num_hidden_layers=n_layers,
                     num_attention_heads=cfg.n_q_heads, num_key_value_heads=cfg.n_kv_heads, head_dim=cfg.head_dim,
                     intermediate_size=cfg.ffn_dim, rms_norm_eps=cfg.rms_eps, rope_theta=cfg.rope_theta,
                     attention_bias=False, mlp_bias=False, tie_word_embeddings=False, max_position_embeddings=256)
    hc._attn_implementation = "eager"
    m = LlamaForCausalLM(hc).double().eval()
    nq, nkv, hd, f = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.ffn_dim
    sd = {"model.embed_tokens.weight": embed, "model.norm.weight": g_final, "lm_head.weight": head}
    for i, w in enumerate(lw):
        p = f"model.layers.{i}."
        sd.update({p + "self_attn.q_proj.weight": w["w_qkv"][: nq * hd],
                   p + "self_attn.k_proj.weight": w["w_qkv"][nq * hd:(nq + nkv) * hd],
                   p + "self_attn.v_proj.weight": w["w_qkv"][(nq + nkv) * hd:],
                   p + "self_attn.o_proj.weight": w["w_o"], p + "mlp.gate_proj.weight": w["w_gate_up"][:f],
                   p + "mlp.up_proj.weight": w["w_gate_up"][f:], p + "mlp.down_proj.weight": w["w_down"],
                   p + "input_layernorm.weight": w["g_attn"], p + "post_attention_layernorm.weight": w["g_ffn"]})
    missing, unexpected = m.load_state_dict({k: torch.from_numpy(np.ascontiguousarray(v)) for k, v in sd.items()},
                                            strict=False)
    assert not unexpected and all("rotary" in k for k in missing)
    # fp64 RoPE frequencies (the library still forms the angles p * freq in
    # fp32, an error of ~1e-7 in the logits, hence the tolerance below)
    m.model.rotary_emb.inv_freq = torch.from_numpy(cfg.rope_theta ** (-np.arange(0, hd, 2, dtype=np.float64) / hd))
    ids = rng.integers(0, vocab, 37)
    with torch.no_grad():
        ref = m(torch.from_numpy(ids)[None]).logits[0, -1].numpy()

    def caches():
        return [oracle.PagedKVCache(32, nkv, hd) for _ in lw]

    bt = [5, 17, 2]
    got, nxt = model_forward(cfg, lw, caches(), embed, g_final, head, [Req(37, 0, bt)], ids, round_between=False)
    np.testing.assert_allclose(got[0], ref, rtol=1e-5, atol=1e-6)
    assert nxt[0] == int(np.argmax(ref))
    cs = caches()
    other = [9]
    model_forward(cfg, lw, cs, embed, g_final, head, [Req(20, 0, bt), Req(1, 0, other)],
                  np.concatenate([ids[:20], [3]]), round_between=False)
    got2, _ = model_forward(cfg, lw, cs, embed, g_final, head, [Req(1, 1, other), Req(17, 20, bt)],
                            np.concatenate([[4], ids[20:]]), round_between=False)
    np.testing.assert_allclose(got2[1], ref, rtol=1e-5, atol=1e-6)
