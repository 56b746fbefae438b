"""Plain fp64 oracle of one whole-model iteration (token embedding, a stack
of decoder layers, final RMSNorm, LM head, greedy choice).

TEST INFRASTRUCTURE ONLY. Only the tests may import this module; the library
never calls it, and it shares no code with the HIP path.

What it computes. Section 3.1 (steps 5-6): each scheduler iteration is one
forward pass of the model over the mixed batch; every request's last row
yields its next token. The paper runs whole models (Llama3-8B, Qwen-7B,
evaluation setup) without writing them out; the reading taken here is the
Llama-3 stack: x = embedding[token], then each decoder layer (oracle.layer,
with its own paged cache), then RMSNorm with the final gain and the LM head,
next token = the index of the largest logit (the lowest such index). Hidden
states pass between layers as bf16 (the model's activation dtype), rounded
to nearest-even here as on the device.
"""
from __future__ import annotations

from typing import Sequence

import numpy as np

from .layer import layer_forward, rmsnorm


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp64 values to the nearest bf16 (ties to even), returned as fp64."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    bits = f.view(np.uint32).astype(np.uint64)
    lower = bits & 0xFFFF
    keep = bits >> 16
    up = (lower > 0x8000) | ((lower == 0x8000) & ((keep & 1) == 1))
    keep = keep + up.astype(np.uint64)
    out = (keep << 16).astype(np.uint32).view(np.float32)
    nan = np.isnan(f)
    out = np.where(nan, f, out)
    return out.astype(np.float64)


def model_forward(cfg, layer_weights: Sequence[dict], caches, embed: np.ndarray, g_final: np.ndarray,
                  lm_head: np.ndarray, requests, token_ids: np.ndarray, round_between: bool = True):
    """Returns (logits [n_requests][vocab] of each request's last row, next
    token ids). layer_weights / caches: fp64 weights and a PagedKVCache per
    layer (prior contexts already stored); embed, lm_head: fp64 [vocab][H].
    round_between=False keeps the hidden states in fp64 between layers (the
    plain definition of the stack, used to pin it)."""
    x = embed[np.asarray(token_ids, dtype=np.int64)]
    for w, cache in zip(layer_weights, caches):
        x = layer_forward(w, cfg, cache, requests, x)
        if round_between:
            x = round_bf16(x)
    last = np.cumsum([int(r.chunk_len) for r in requests]) - 1
    h = rmsnorm(x[last], g_final, cfg.rms_eps)
    logits = h @ lm_head.T
    return logits, np.argmax(logits, axis=1)
