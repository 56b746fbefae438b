"""The GEMM launch grid and the configurations whose plans it must cover.

Every (tile shape, K split) pair is forced in turn on one layer shape, the
"cover" shape, on which all four GEMMs can take every split count (K / 64 is
32 or 40, so splits 1..8 each get work) and whose split-K reduce fused with
the pre-FFN RMSNorm takes the same instantiation as the 8B and 70B layers
(H / 8 in (256, 1024]). Token count and N are ragged against every tile.
The configurations below are the ones the benchmark and the full-size tests
run; the plans the library picks for them must be among the forced ones.
"""
from hb_workloads import (LLAMA3_70B, LLAMA3_8B, SWEEP_CHUNKS, SWEEP_DECODES, LayerShape, llama8b_batch,
                          multi_batch)

COVER = LayerShape("gemm-cover", 2560, 16, 4, 128, 2560, weight_seed=23)
COVER_LENS = [(200, 40), (1, 7), (1, 300), (90, 0), (1, 64)]  # T = 293
COVER_T = sum(c for c, _ in COVER_LENS)
MAX_KSPLIT = 8
CU_COUNT = 256  # MI355X


def real_token_counts():
    """(shape, T) of every timed or tested full-size batch."""
    out = [(LLAMA3_8B, c + n) for c in SWEEP_CHUNKS for n in SWEEP_DECODES]
    out.append((LLAMA3_8B, llama8b_batch().n_tokens))
    out.append((LLAMA3_8B, multi_batch().n_tokens))
    out.append((LLAMA3_70B, 2048 + 32))
    return out
