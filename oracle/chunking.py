"""Reference of the dynamic-chunking helpers: the iteration latency model and
the chunk selection.

TEST INFRASTRUCTURE ONLY. Only the tests and the benchmark may import this
module; the library never calls it, and it shares no code with the library's
host implementation (it does not import the library).

What it computes.
* Section 3.3 (dynamic chunking): each iteration takes the largest prefill
  chunk for which the batch -- that chunk next to every decode -- finishes
  before the earliest next-token deadline of the decodes; the slack of a
  decode is that deadline minus the current time (the TBT deadline equation
  of Section 3.2: D_n = t_arrival + SLO_TTFT + (n - 1) SLO_TBT).
* Section 3.1 (step 4) and 3.6: the batch latency comes from a lightweight
  predictor trained on offline profiles. The paper's predictor is a random
  forest on simulator profiles; the reading taken here is a linear model in
  five roofline terms of the batch (a constant, the token count that the
  linear layers scale with, the KV bytes that decode attention streams, and
  the attention flops of chunk rows against their cached context and within
  the chunk's causal triangle, whose rates differ), fitted by non-negative least squares on
  relative error to measured profile cells, so that the prediction cannot fall
  as the chunk grows.

The fit here enumerates every support set and solves each with NumPy's
least-squares routine (an SVD), keeping the best non-negative solution; the
selection scans every candidate chunk. Both are plain and slow by design.
"""
from __future__ import annotations

import itertools
import math
from typing import Sequence, Tuple

import numpy as np

N_FEATURES = 5


def latency_features(n_q_heads: int, n_kv_heads: int, head_dim: int,
                     requests: Sequence[Tuple[int, int]]) -> np.ndarray:
    """[1, T/1e3, KV GB read, attention TFLOP against cached context, attention
    TFLOP within the new tokens] of a batch of (chunk_len, context_len)."""
    T = kv = ctx_pairs = new_pairs = 0.0
    for chunk, ctx in requests:
        if chunk == 0:  # no new tokens: the request is not in the batch
            continue
        T += chunk
        kv += ctx + chunk
        ctx_pairs += chunk * ctx
        new_pairs += chunk * (chunk + 1) / 2
    per_pair = 4.0 * n_q_heads * head_dim
    return np.array([1.0, T / 1e3, kv * (2.0 * n_kv_heads * head_dim * 2.0) / 1e9,
                     ctx_pairs * per_pair / 1e12, new_pairs * per_pair / 1e12])


def profile_batches(chunk_sizes: Sequence[int], mixes: Sequence[Tuple[Sequence[int], int]]):
    """The batch of each profile cell, row-major [mix][chunk]: one chunk at the
    mix's chunk context, then the mix's decodes."""
    return [[[(c, cc)] + [(1, int(x)) for x in ctxs] for c in chunk_sizes] for ctxs, cc in mixes]


def fit_latency_model(n_q_heads: int, n_kv_heads: int, head_dim: int, chunk_sizes, mixes,
                      median_ms) -> Tuple[np.ndarray, float]:
    """Non-negative least squares of sum_i coef_i f_i / t = 1 over the cells;
    returns (coef, root mean square relative residual)."""
    rows, ys = [], []
    for mix_batches, mix_ms in zip(profile_batches(chunk_sizes, mixes), np.asarray(median_ms, float)):
        for batch, t in zip(mix_batches, mix_ms):
            rows.append(latency_features(n_q_heads, n_kv_heads, head_dim, batch) / t)
            ys.append(1.0)
    A, y = np.array(rows), np.array(ys)
    best, best_res = None, math.inf
    for k in range(1, N_FEATURES + 1):
        for support in itertools.combinations(range(N_FEATURES), k):
            sol, *_ = np.linalg.lstsq(A[:, support], y, rcond=None)
            if np.any(sol < 0):
                continue
            coef = np.zeros(N_FEATURES)
            coef[list(support)] = sol
            res = float(np.sum((A @ coef - y) ** 2))
            if res < best_res:
                best, best_res = coef, res
    return best, math.sqrt(best_res / len(y))


def predict_latency(coef, n_q_heads: int, n_kv_heads: int, head_dim: int, requests) -> float:
    f = latency_features(n_q_heads, n_kv_heads, head_dim, requests)
    s = 0.0
    for c, x in zip(coef, f):  # in feature order, as a dot product
        s += float(c) * float(x)
    return s


def select_chunk(coef, n_q_heads: int, n_kv_heads: int, head_dim: int, decode_contexts, deadlines_ms,
                 now_ms: float, chunk_context: int, max_chunk: int, granularity: int,
                 margin: float = 0.0) -> Tuple[int, float]:
    """Largest candidate chunk (multiples of granularity below max_chunk, or
    max_chunk) whose batch's predicted latency, scaled by (1 + margin), is
    within the slack; 0 if none. Section 3.3 asks for a chunk that violates no
    deadline; the predictor errs, so a caller covers its error with the
    margin (the relative under-prediction it is prepared to absorb)."""
    slack = min((d - now_ms for d in deadlines_ms), default=math.inf)
    decodes = [(1, int(x)) for x in decode_contexts]

    def pred(c):
        return predict_latency(coef, n_q_heads, n_kv_heads, head_dim, [(c, chunk_context)] + decodes)

    cands = sorted({c for c in range(granularity, max_chunk + 1, granularity)} | ({max_chunk} if max_chunk else set()))
    best = 0
    for c in cands:  # every candidate, no early exit
        if pred(c) * (1.0 + margin) <= slack:
            best = max(best, c)
    return best, pred(best)
