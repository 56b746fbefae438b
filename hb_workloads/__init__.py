"""Seeded synthetic inputs for the hybrid-batch decoder layer.

This module is shared by the tests, the benchmark and the smoke check. It
holds shapes, seeds and random draws only -- no step of the layer's
arithmetic -- so that the CPU oracle and the HIP library receive identical
inputs while sharing no code.

Everything is drawn with NumPy's PCG64 (``default_rng``) in fp32 and rounded
once to bf16 (round-to-nearest-even). Arrays of bf16 values are carried as
``uint16`` bit patterns; each consumer widens them itself.

Workloads stand in for the paper's traces (ShareGPT, Azure Conv, Azure Code,
Table "Datasets" of the evaluation section), which are not available: prompt
and context lengths are lognormal with sigma 1.0, whose p90/p50 ratio (3.6)
matches the prompt columns of that table.
"""
from __future__ import annotations

import dataclasses
import math
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

KV_BLOCK = 16
POOL_TOKENS = 1 << 21  # 2M-token paged pool -> 131072 blocks of 16


@dataclasses.dataclass(frozen=True)
class LayerShape:
    name: str
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    kv_block: int = KV_BLOCK
    rope_theta: float = 5e5
    rms_eps: float = 1e-5
    weight_seed: int = 0

    @property
    def qkv_dim(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def linear_params(self) -> int:
        h, hd = self.hidden, self.head_dim
        return (h * self.qkv_dim + self.n_q_heads * hd * h
                + 2 * h * self.ffn_dim + self.ffn_dim * h)


TINY = LayerShape("tiny", 256, 4, 2, 64, 688, weight_seed=101)
LLAMA3_8B = LayerShape("llama3-8b", 4096, 32, 8, 128, 14336, weight_seed=108)
LLAMA3_70B = LayerShape("llama3-70b", 8192, 64, 8, 128, 28672, weight_seed=170)


def tp_shard(shape: LayerShape, tp: int, weight_seed: int) -> LayerShape:
    """One GPU's share of a layer under tensor parallelism of degree tp,
    sharded by heads: n_q/tp query heads, n_kv/tp kv heads (at least one) and
    ffn_dim/tp FFN columns over the full hidden size. Its own weight seed: the
    shard's weights are a fresh random init, not a slice of the full layer's."""
    if shape.n_q_heads % tp or shape.ffn_dim % tp or (shape.n_kv_heads % tp and tp % shape.n_kv_heads):
        raise ValueError(f"{shape.name} does not shard {tp} ways by heads")
    return dataclasses.replace(shape, name=f"{shape.name}-tp{tp}-shard", n_q_heads=shape.n_q_heads // tp,
                               n_kv_heads=max(1, shape.n_kv_heads // tp), ffn_dim=shape.ffn_dim // tp,
                               weight_seed=weight_seed)


# the per-GPU shards of the 8B layer at TP2 and the 70B layer at TP8
LLAMA3_8B_TP2 = tp_shard(LLAMA3_8B, 2, weight_seed=182)
LLAMA3_70B_TP8 = tp_shard(LLAMA3_70B, 8, weight_seed=178)
SHAPES = {s.name: s for s in (TINY, LLAMA3_8B, LLAMA3_70B, LLAMA3_8B_TP2, LLAMA3_70B_TP8)}


# ----------------------------------------------------------------------------
# bf16 encoding of host fp32 draws (input preparation, shared by both sides)
# ----------------------------------------------------------------------------
def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16, nearest-even, returned as uint16 bit patterns."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32 (for host-side checks)."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


_CHUNK = 1 << 18  # values per independent PCG64 stream
_POOL = None


def _pool():
    global _POOL
    if _POOL is None:
        import concurrent.futures as cf
        _POOL = cf.ThreadPoolExecutor(max_workers=max(1, min(16, os.cpu_count() or 1)))
    return _POOL


def _round_bf16(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bits, nearest-even (torch's cast, multi-threaded; the same
    bits as f32_to_bf16_bits)."""
    import torch
    return torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def normal_bf16(key, shape, std: float = 1.0) -> np.ndarray:
    """N(0, std^2) draws as bf16 bits. Chunk i of 2^18 values comes from its
    own stream default_rng([*key, i]), so the values depend only on key and
    shape, not on the number of threads."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float32)
    key = list(key)

    def fill(i):
        s = i * _CHUNK
        e = min(n, s + _CHUNK)
        np.random.default_rng(key + [i]).standard_normal(size=e - s, dtype=np.float32, out=out[s:e])
        if std != 1.0:
            out[s:e] *= np.float32(std)

    list(_pool().map(fill, range((n + _CHUNK - 1) // _CHUNK)))
    return _round_bf16(out).reshape(shape)


# ----------------------------------------------------------------------------
# Weights
# ----------------------------------------------------------------------------
WEIGHT_NAMES = ("w_qkv", "w_o", "w_gate_up", "w_down", "g_attn", "g_ffn")


def make_weights(shape: LayerShape, seed: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Random-init layer weights as bf16 bit patterns, row-major [out][in].

    * each matrix ~ N(0, 1/fan_in) (std = 1/sqrt(fan_in)); fan_in = hidden for
      the QKV and gate/up projections, n_q_heads*head_dim for O, ffn_dim for down;
    * ``w_qkv`` rows are [q heads | k heads | v heads], each head head_dim rows;
    * ``w_gate_up`` rows are [gate (ffn_dim) | up (ffn_dim)];
    * RMSNorm gains g = 1 + 0.1*N(0,1).
    Every matrix has its own PCG64 stream keyed by (seed, index).
    """
    seed = shape.weight_seed if seed is None else seed
    h, f = shape.hidden, shape.ffn_dim
    qd = shape.n_q_heads * shape.head_dim
    specs = {
        "w_qkv": ((shape.qkv_dim, h), 1.0 / math.sqrt(h)),
        "w_o": ((h, qd), 1.0 / math.sqrt(qd)),
        "w_gate_up": ((2 * f, h), 1.0 / math.sqrt(h)),
        "w_down": ((h, f), 1.0 / math.sqrt(f)),
    }
    out: Dict[str, np.ndarray] = {}
    for i, (name, (shp, std)) in enumerate(specs.items()):
        out[name] = normal_bf16([seed, i], shp, std)
    for i, name in enumerate(("g_attn", "g_ffn")):
        rng = np.random.default_rng([seed, 10 + i])
        g = 1.0 + 0.1 * rng.standard_normal(size=(h,), dtype=np.float32)
        out[name] = f32_to_bf16_bits(g.astype(np.float32))
    return out


def make_model_weights(shape: LayerShape, n_layers: int, vocab: int, seed: Optional[int] = None) -> Dict:
    """Random-init weights of an n_layers model: per layer as make_weights
    (seed 1000 * seed + layer + 1), token embedding ~ N(0,1) (so hidden states
    start at the layer inputs' N(0,1) scale), LM head ~ N(0, 1/hidden), final
    RMSNorm gain 1 + 0.1 N(0,1); bf16 bits, rows [vocab][hidden]."""
    seed = shape.weight_seed if seed is None else seed
    h = shape.hidden
    rng = np.random.default_rng([seed, 22])
    return {"layers": [make_weights(shape, seed=1000 * seed + l + 1) for l in range(n_layers)],
            "embed": normal_bf16([seed, 20], (vocab, h), 1.0),
            "lm_head": normal_bf16([seed, 21], (vocab, h), 1.0 / math.sqrt(h)),
            "g_final": f32_to_bf16_bits((1.0 + 0.1 * rng.standard_normal(size=(h,), dtype=np.float32)))}


# ----------------------------------------------------------------------------
# Batches
# ----------------------------------------------------------------------------
@dataclasses.dataclass
class Request:
    chunk_len: int          # new tokens this iteration (1 = decode)
    context_len: int        # tokens already in the paged cache
    block_table: np.ndarray  # int32 physical block ids, ceil((ctx+chunk)/16) entries

    @property
    def kv_len(self) -> int:
        return self.context_len + self.chunk_len


@dataclasses.dataclass
class Batch:
    shape: LayerShape
    requests: List[Request]
    num_blocks: int
    seed: int
    label: str = ""

    @property
    def n_tokens(self) -> int:
        return int(sum(r.chunk_len for r in self.requests))

    @property
    def n_decode(self) -> int:
        return sum(1 for r in self.requests if r.chunk_len == 1)

    def token_offsets(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum([r.chunk_len for r in self.requests])]).astype(np.int64)

    def x_in(self) -> np.ndarray:
        """Token activations ~ N(0,1), bf16 bits [T][hidden]."""
        return normal_bf16([self.seed, 1], (self.n_tokens, self.shape.hidden))

    def prior_kv(self, r: int, layer: int = 0) -> Tuple[np.ndarray, np.ndarray]:
        """Synthetic cached K (already rotated) and V for positions [0, ctx) of
        request r in decoder layer `layer`, each ~ N(0,1), bf16 bits
        [ctx][n_kv][head_dim]."""
        req = self.requests[r]
        shp = (req.context_len, self.shape.n_kv_heads, self.shape.head_dim)
        key = [self.seed, 2, r] if layer == 0 else [self.seed, 2, r, 100 + layer]
        return normal_bf16(key + [0], shp), normal_bf16(key + [1], shp)

    def token_ids(self, vocab: int) -> np.ndarray:
        """Input token ids of the batch rows, uniform over [0, vocab), int32 [T]."""
        return np.random.default_rng([self.seed, 3]).integers(0, vocab, self.n_tokens).astype(np.int32)


def blocks_needed(kv_len: int, block: int = KV_BLOCK) -> int:
    return -(-kv_len // block)


def assign_blocks(lens: Sequence[Tuple[int, int]], num_blocks: int, seed: int,
                  block: int = KV_BLOCK) -> List[Request]:
    """Build requests from (chunk_len, context_len) pairs; block ids come from a
    seeded permutation of the pool, consumed in request order."""
    need = sum(blocks_needed(c + x, block) for c, x in lens)
    if need > num_blocks:
        raise ValueError(f"pool of {num_blocks} blocks cannot hold {need}")
    perm = np.random.default_rng([seed, 3]).permutation(num_blocks).astype(np.int32)
    out, off = [], 0
    for c, x in lens:
        n = blocks_needed(c + x, block)
        out.append(Request(int(c), int(x), perm[off:off + n].copy()))
        off += n
    return out


def make_batch(shape: LayerShape, lens: Sequence[Tuple[int, int]], seed: int,
               num_blocks: Optional[int] = None, label: str = "") -> Batch:
    if num_blocks is None:
        num_blocks = POOL_TOKENS // shape.kv_block
    return Batch(shape, assign_blocks(lens, num_blocks, seed, shape.kv_block), num_blocks, seed, label)


# --- the five workloads -------------------------------------------------------
def tiny_batch(seed: int = 1) -> Batch:
    """Tiny layer: one 64-token chunk at context 128 plus 8 decodes at context 256,
    in a shuffled 256-block pool."""
    lens = [(64, 128)] + [(1, 256)] * 8
    return make_batch(TINY, lens, seed, num_blocks=256, label="tiny")


def llama8b_batch(seed: int = 2, shape: LayerShape = LLAMA3_8B) -> Batch:
    """8B layer (or one of its shards): one 512-token chunk at offset
    U{0..4096} plus 64 decodes with contexts U{512..4096}."""
    rng = np.random.default_rng([seed, 0])
    off = int(rng.integers(0, 4096, endpoint=True))
    ctx = rng.integers(512, 4096, size=64, endpoint=True)
    lens = [(512, off)] + [(1, int(c)) for c in ctx]
    return make_batch(shape, lens, seed, label=f"{shape.name}: chunk 512 + 64 decodes")


SWEEP_CHUNKS = (128, 256, 512, 1024, 2048)
SWEEP_DECODES = (0, 32, 128, 256)


def sweep_decode_contexts(n_decode: int, lo: int = 256, hi: int = 8192) -> np.ndarray:
    """Decode contexts for one row of the chunk sweep: floor(exp(U(ln lo, ln hi))),
    seeded by the decode count so every chunk size sees the same decodes."""
    rng = np.random.default_rng([30000 + n_decode, 0])
    return np.floor(np.exp(rng.uniform(math.log(lo), math.log(hi), size=n_decode))).astype(np.int64)


def sweep_batch(chunk: int, n_decode: int) -> Batch:
    """8B layer, chunk-size sweep cell: chunk at offset 0 plus n_decode decodes."""
    ctx = sweep_decode_contexts(n_decode)
    lens = [(chunk, 0)] + [(1, int(c)) for c in ctx]
    return make_batch(LLAMA3_8B, lens, 31000 + chunk,
                      label=f"llama3-8b sweep: chunk {chunk} + {n_decode} decodes")


def multi_batch(seed: int = 4) -> Batch:
    """8B layer, 4 prefill chunks + 256 decodes, blocks shuffled in a 2M-token pool.

    Prompt P ~ floor(lognormal(ln 1024, 1.0)) capped at 16384; chunk c ~ U{256..1024},
    c_eff = min(c, P), offset ~ U{0..P-c_eff}. Decode contexts ~ lognormal(ln 1500, 1.0)
    capped at 16384."""
    rng = np.random.default_rng([seed, 0])
    lens = []
    for _ in range(4):
        p = int(min(16384, math.floor(rng.lognormal(math.log(1024), 1.0))))
        p = max(p, 1)
        c = int(rng.integers(256, 1024, endpoint=True))
        c_eff = min(c, p)
        off = int(rng.integers(0, max(0, p - c_eff), endpoint=True))
        lens.append((c_eff, off))
    ctx = np.minimum(16384, np.floor(rng.lognormal(math.log(1500), 1.0, size=256))).astype(np.int64)
    lens += [(1, int(max(c, 1))) for c in ctx]
    return make_batch(LLAMA3_8B, lens, seed, label="llama3-8b: 4 chunks + 256 decodes")


def llama70b_batch(seed: int = 5, shape: LayerShape = LLAMA3_70B) -> Batch:
    """70B layer (or one of its shards): one 2048-token chunk at offset 30720
    plus 32 decodes at context 32768."""
    lens = [(2048, 30720)] + [(1, 32768)] * 32
    return make_batch(shape, lens, seed, label=f"{shape.name}: chunk 2048 + 32 decodes")


WORKLOADS = {
    "tiny": tiny_batch,
    "llama3-8b": llama8b_batch,
    "llama3-8b-multi": multi_batch,
    "llama3-70b": llama70b_batch,
}


def scaled_shape(shape: LayerShape, **kw) -> LayerShape:
    return dataclasses.replace(shape, **kw)
