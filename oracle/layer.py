"""Plain fp64 CPU oracle of one hybrid-batch decoder-layer iteration.

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this module; the library never calls it, and it
shares no code with the HIP path (it does not import the library, and the
library does not read anything here).

What it computes. Section 3.1 (steps 5-6) and Section 3.3 of the paper
describe each scheduler iteration as ONE forward pass over a mixed batch:
every request in the decode queue contributes one token and a prefill request
contributes a chunk of its prompt; the linear layers run over all tokens of
the batch together (the fused prefill-decode MLP), while attention reads each
request's earlier tokens from the paged KV cache (Section 3.6: the engine is
vLLM with PagedAttention). The paper names its models (Llama3-8B, Qwen-7B,
evaluation setup) but never writes the layer out, so the oracle takes the
standard Llama-3 pre-norm decoder layer:

    a  = RMSNorm(x; g_attn)
    q, k, v = a W_q^T, a W_k^T, a W_v^T          (no biases)
    q, k  <- RoPE(position)                       (rotate-half pairs (j, j+hd/2))
    k, v  -> paged cache slot (block_table[p // 16], p % 16)
    o_h  = softmax_j(q_h . k_j / sqrt(hd)) v_j  over cached keys j = 0..p,
           kv head of q head h = h // (n_q / n_kv)
    h2 = x + o W_o^T
    f  = RMSNorm(h2; g_ffn)
    y  = h2 + (silu(f W_gate^T) * (f W_up^T)) W_down^T

Chunking, paging and batching only regroup this per-request computation, so
the batch result is each request's result, concatenated in request order.
Every step below is the plain definition in fp64; NumPy's matmul is used as a
library primitive, with no blocking, fusion or reordering of the definition.
"""
from __future__ import annotations

import math
from typing import Dict, Iterable, List, Optional, Sequence

import numpy as np


# ----------------------------------------------------------------------------
# input decoding
# ----------------------------------------------------------------------------
def bf16_bits_to_f64(bits) -> np.ndarray:
    """Exact value of bf16 bit patterns (uint16) as fp64."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def weights_to_f64(w: Dict[str, np.ndarray]) -> Dict[str, np.ndarray]:
    return {k: bf16_bits_to_f64(v) for k, v in w.items()}


# ----------------------------------------------------------------------------
# layer steps (each is the textbook definition)
# ----------------------------------------------------------------------------
def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps) * g."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def linear(a: np.ndarray, w: np.ndarray) -> np.ndarray:
    """y = a W^T with W stored [out][in] (no bias)."""
    return a @ w.T


def rope_angles(pos: np.ndarray, head_dim: int, theta: float) -> np.ndarray:
    """phi[t, j] = pos_t * theta^(-2j/head_dim), j < head_dim/2, in fp64."""
    j = np.arange(head_dim // 2, dtype=np.float64)
    omega = theta ** (-2.0 * j / head_dim)
    return np.asarray(pos, dtype=np.float64)[:, None] * omega[None, :]


def rope(z: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half RoPE of z[t, head, hd] at positions pos[t].

    Pair (z_j, z_{j+hd/2}) is rotated by angle phi[t, j]:
    (u, w) -> (u cos phi - w sin phi, w cos phi + u sin phi)."""
    hd = z.shape[-1]
    half = hd // 2
    phi = rope_angles(pos, hd, theta)[:, None, :]  # [t, 1, half]
    c, s = np.cos(phi), np.sin(phi)
    u, w = z[..., :half], z[..., half:]
    return np.concatenate([u * c - w * s, w * c + u * s], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    """silu(z) = z / (1 + exp(-z))."""
    return z / (1.0 + np.exp(-z))


def swiglu_mlp(f: np.ndarray, w_gate_up: np.ndarray, w_down: np.ndarray) -> np.ndarray:
    """(silu(f W_gate^T) * (f W_up^T)) W_down^T, W_gate_up rows = [gate | up]."""
    ffn = w_gate_up.shape[0] // 2
    gate = linear(f, w_gate_up[:ffn])
    up = linear(f, w_gate_up[ffn:])
    return linear(silu(gate) * up, w_down)


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, q_pos: np.ndarray,
                     n_kv_heads: int) -> np.ndarray:
    """Attention of query rows q[i, h, :] at absolute positions q_pos[i] over keys
    k[j], v[j] at positions j = 0..len(k)-1; row i sees keys j <= q_pos[i].

    GQA: q head h reads kv head h // (n_q / n_kv). Scale 1/sqrt(hd); softmax
    with the row maximum subtracted."""
    n_q, hd = q.shape[1], q.shape[2]
    group = n_q // n_kv_heads
    n_keys = k.shape[0]
    mask = np.arange(n_keys)[None, :] <= np.asarray(q_pos)[:, None]  # [rows, keys]
    out = np.empty_like(q)
    for h in range(n_q):
        g = h // group
        s = (q[:, h, :] @ k[:, g, :].T) / math.sqrt(hd)
        s = np.where(mask, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v[:, g, :]
    return out


# ----------------------------------------------------------------------------
# paged KV cache (logical slots; storage layout is the library's business)
# ----------------------------------------------------------------------------
def kv_slot(block_table: Sequence[int], pos: int, block: int = 16):
    """Physical slot of absolute position pos: (block_table[pos // B], pos % B)."""
    return int(block_table[pos // block]), pos % block


class PagedKVCache:
    """Blocks of `block` token slots per kv head, stored sparsely (only blocks
    written so far), values in fp64."""

    def __init__(self, num_blocks: int, n_kv_heads: int, head_dim: int, block: int = 16):
        self.num_blocks, self.n_kv, self.hd, self.block = num_blocks, n_kv_heads, head_dim, block
        self.k: Dict[int, np.ndarray] = {}
        self.v: Dict[int, np.ndarray] = {}

    def _blk(self, store, b: int) -> np.ndarray:
        if not 0 <= b < self.num_blocks:
            raise IndexError(f"block id {b} outside pool of {self.num_blocks}")
        if b not in store:
            store[b] = np.full((self.block, self.n_kv, self.hd), np.nan)
        return store[b]

    def write(self, block_table, start: int, k: np.ndarray, v: np.ndarray) -> None:
        """Store k[i], v[i] ([n][n_kv][hd]) at position start+i."""
        for i in range(k.shape[0]):
            b, o = kv_slot(block_table, start + i, self.block)
            self._blk(self.k, b)[o] = k[i]
            self._blk(self.v, b)[o] = v[i]

    def read(self, block_table, n: int):
        """Gather K, V [n][n_kv][hd] for positions 0..n-1 through the block table."""
        nb = -(-n // self.block)
        ks = [self.k[int(block_table[i])] for i in range(nb)]
        vs = [self.v[int(block_table[i])] for i in range(nb)]
        return np.concatenate(ks)[:n], np.concatenate(vs)[:n]


# ----------------------------------------------------------------------------
# one iteration over a hybrid batch
# ----------------------------------------------------------------------------
def layer_forward(w: Dict[str, np.ndarray], cfg, cache: PagedKVCache, requests,
                  x: np.ndarray, rows: Optional[Iterable[int]] = None,
                  stages: bool = False):
    """Run the decoder layer over a hybrid batch (tokens of all requests,
    concatenated in request order).

    w: fp64 weights (w_qkv, w_o, w_gate_up, w_down, g_attn, g_ffn).
    cfg: object with n_q_heads, n_kv_heads, head_dim, rope_theta, rms_eps, kv_block.
    requests: objects with chunk_len, context_len, block_table. Positions
      [0, context_len) must already be in `cache`.
    x: fp64 [T][hidden].
    rows: token rows whose output to compute (default: all). K/V of every token
      are always computed and stored, since later rows of a chunk read them.
    Returns y [len(rows)][hidden] (and a dict of per-step values if stages).
    """
    nq, nkv, hd = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    T = x.shape[0]
    chunk = [int(r.chunk_len) for r in requests]
    ctx = [int(r.context_len) for r in requests]
    if sum(chunk) != T:
        raise ValueError("x rows must equal the sum of chunk lengths")
    req_of = np.repeat(np.arange(len(requests)), chunk)
    starts = np.concatenate([[0], np.cumsum(chunk)])
    pos = np.array([ctx[r] + (t - starts[r]) for t, r in enumerate(req_of)], dtype=np.int64)
    rows = np.arange(T) if rows is None else np.asarray(sorted(set(int(i) for i in rows)), dtype=np.int64)

    wq = w["w_qkv"][: nq * hd]
    wk = w["w_qkv"][nq * hd:(nq + nkv) * hd]
    wv = w["w_qkv"][(nq + nkv) * hd:]

    a = rmsnorm(x, w["g_attn"], cfg.rms_eps)
    k_new = rope(linear(a, wk).reshape(T, nkv, hd), pos, cfg.rope_theta)
    v_new = linear(a, wv).reshape(T, nkv, hd)
    # all new K/V of the batch enter the cache before any attention
    for r, req in enumerate(requests):
        s, e = starts[r], starts[r + 1]
        cache.write(req.block_table, ctx[r], k_new[s:e], v_new[s:e])

    q = rope(linear(a[rows], wq).reshape(len(rows), nq, hd), pos[rows], cfg.rope_theta)
    o = np.empty_like(q)
    for r in np.unique(req_of[rows]):
        sel = np.nonzero(req_of[rows] == r)[0]
        kv_len = ctx[r] + chunk[r]
        kc, vc = cache.read(requests[r].block_table, kv_len)
        o[sel] = causal_attention(q[sel], kc, vc, pos[rows][sel], nkv)

    o_flat = o.reshape(len(rows), nq * hd)
    h2 = x[rows] + linear(o_flat, w["w_o"])
    f = rmsnorm(h2, w["g_ffn"], cfg.rms_eps)
    ffn = w["w_gate_up"].shape[0] // 2
    gate = linear(f, w["w_gate_up"][:ffn])
    up = linear(f, w["w_gate_up"][ffn:])
    m = silu(gate) * up
    y = h2 + linear(m, w["w_down"])
    if not stages:
        return y
    return y, {"rows": rows, "pos": pos, "a": a, "q": q, "k": k_new, "v": v_new,
               "o": o_flat, "h2": h2, "m": m, "y": y}


def seed_cache(cache: PagedKVCache, requests, prior_kv) -> None:
    """Place each request's cached context (K already rotated, V) at positions
    [0, context_len); prior_kv(r) returns (k, v) as fp64 [ctx][n_kv][hd]."""
    for r, req in enumerate(requests):
        if req.context_len:
            k, v = prior_kv(r)
            cache.write(req.block_table, 0, k, v)
