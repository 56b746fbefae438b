"""Python binding of libhb.so (include/hb.h): argument marshalling only.

Every step of the layer runs in the library's HIP kernels; PyTorch supplies
device memory and streams. Names and arguments follow the C ABI.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, Iterable, List, Optional, Sequence, Tuple

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhb.so")

HB_OK, HB_ERR_INVALID, HB_ERR_RANGE, HB_ERR_OOM, HB_ERR_HIP, HB_ERR_UNSUPPORTED = range(6)
HB_OUT_F32, HB_OUT_BF16 = 0, 1
(HB_K_RMSNORM_ATTN, HB_K_GEMM_QKV, HB_K_ATTENTION, HB_K_ATTN_MERGE, HB_K_GEMM_O,
 HB_K_RMSNORM_FFN, HB_K_GEMM_GATE_UP, HB_K_GEMM_DOWN, HB_K_COUNT) = range(9)
HB_STAGE_Q, HB_STAGE_ATTN, HB_STAGE_H2, HB_STAGE_MLP = range(4)
HB_GEMM_QKV, HB_GEMM_O, HB_GEMM_GATE_UP, HB_GEMM_DOWN, HB_GEMM_COUNT = range(5)
GEMM_NAMES = ("gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down")

EXPORTED = ("hb_create_layer", "hb_destroy_layer", "hb_append_kv", "hb_run_iteration", "hb_validate_batch",
            "hb_profile", "hb_profile_batches", "hb_latency_features", "hb_fit_latency_model", "hb_predict_latency", "hb_select_chunk",
            "hb_create_model", "hb_destroy_model", "hb_model_layer", "hb_run_model",
            "hb_set_kernel_timing", "hb_kernel_times", "hb_kernel_name", "hb_layer_stage", "hb_last_error",
            "hb_gemm_tile_count", "hb_plan_gemms", "hb_layer_gemm_plans", "hb_run_iteration_noalloc",
            "hb_measure_device_rates")
HB_LAT_FEATURES = 5


class hb_layer_config(C.Structure):
    _fields_ = [("hidden", C.c_int32), ("n_q_heads", C.c_int32), ("n_kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("ffn_dim", C.c_int32), ("kv_block_size", C.c_int32),
                ("rope_theta", C.c_float), ("rms_eps", C.c_float),
                ("max_batch_tokens", C.c_int32), ("max_requests", C.c_int32)]


class hb_layer_weights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("w_qkv", "w_o", "w_gate_up", "w_down", "g_attn", "g_ffn")]


class hb_kv_pool(C.Structure):
    _fields_ = [("k_pool", C.c_void_p), ("v_pool", C.c_void_p), ("num_blocks", C.c_int32)]


class hb_request(C.Structure):
    _fields_ = [("chunk_len", C.c_int32), ("context_len", C.c_int32),
                ("block_table", C.POINTER(C.c_int32)), ("n_blocks", C.c_int32)]


class hb_batch_desc(C.Structure):
    _fields_ = [("n_requests", C.c_int32), ("requests", C.POINTER(hb_request)),
                ("x_in", C.c_void_p), ("x_out", C.c_void_p), ("out_dtype", C.c_int32)]


class hb_device_rates(C.Structure):
    _fields_ = [("random_4kb_read_bytes_per_s", C.c_double), ("stream_read_bytes_per_s", C.c_double),
                ("mfma_bf16_flop_per_s", C.c_double)]


class hb_decode_mix(C.Structure):
    _fields_ = [("n_decode", C.c_int32), ("decode_contexts", C.POINTER(C.c_int32)), ("chunk_context", C.c_int32)]


class hb_profile_cell(C.Structure):
    _fields_ = [(n, C.c_float) for n in ("median_ms", "p10_ms", "p90_ms", "tokens_per_s", "hbm_frac", "mfma_frac")]


class hb_latency_model(C.Structure):
    _fields_ = [("coef", C.c_double * HB_LAT_FEATURES), ("fit_rel_rms", C.c_double), ("fit_max_under", C.c_double),
                ("n_cells", C.c_int32)]


class hb_model_desc(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("vocab", C.c_int32), ("layers", C.POINTER(hb_layer_weights)),
                ("pools", C.POINTER(hb_kv_pool)), ("embed", C.c_void_p), ("g_final", C.c_void_p),
                ("lm_head", C.c_void_p)]


class hb_model_batch(C.Structure):
    _fields_ = [("n_requests", C.c_int32), ("requests", C.POINTER(hb_request)), ("token_ids", C.c_void_p),
                ("logits", C.c_void_p), ("next_tokens", C.c_void_p), ("hidden_states", C.c_void_p)]


class HBError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"hb status {status}: {message}")
        self.status = status


_lib: Optional[C.CDLL] = None


def load() -> C.CDLL:
    """Load libhb.so; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2503_22562_amd.build`")
    # torch first: libhb then binds to the HIP runtime torch already loaded,
    # so torch's streams and allocations are valid handles for the library.
    import torch  # noqa: F401
    lib = C.CDLL(LIB_PATH)
    st = C.c_int
    lib.hb_create_layer.argtypes = [C.POINTER(hb_layer_config), C.POINTER(hb_layer_weights), C.POINTER(hb_kv_pool),
                                    C.c_void_p, C.POINTER(C.c_void_p)]
    lib.hb_create_layer.restype = st
    lib.hb_destroy_layer.argtypes = [C.c_void_p]
    lib.hb_destroy_layer.restype = None
    lib.hb_append_kv.argtypes = [C.c_void_p, C.POINTER(C.c_int32), C.c_int32, C.c_int32, C.c_int32, C.c_void_p,
                                 C.c_void_p]
    lib.hb_append_kv.restype = st
    lib.hb_run_iteration.argtypes = [C.c_void_p, C.POINTER(hb_batch_desc)]
    lib.hb_run_iteration.restype = st
    lib.hb_run_iteration_noalloc.argtypes = [C.c_void_p, C.POINTER(hb_batch_desc)]
    lib.hb_run_iteration_noalloc.restype = st
    lib.hb_validate_batch.argtypes = [C.POINTER(hb_layer_config), C.c_int32, C.POINTER(hb_batch_desc)]
    lib.hb_validate_batch.restype = st
    lib.hb_profile.argtypes = [C.c_void_p, C.POINTER(C.c_int32), C.c_int32, C.POINTER(hb_decode_mix), C.c_int32,
                               C.c_int32, C.c_int32, C.c_uint64, C.POINTER(hb_profile_cell)]
    lib.hb_profile.restype = st
    lib.hb_profile_batches.argtypes = [C.c_void_p, C.POINTER(hb_batch_desc), C.c_int32, C.c_int32, C.c_int32,
                                       C.POINTER(hb_profile_cell)]
    lib.hb_profile_batches.restype = st
    lib.hb_latency_features.argtypes = [C.POINTER(hb_layer_config), C.POINTER(hb_request), C.c_int32,
                                        C.POINTER(C.c_double)]
    lib.hb_latency_features.restype = st
    lib.hb_fit_latency_model.argtypes = [C.POINTER(hb_layer_config), C.POINTER(C.c_int32), C.c_int32,
                                         C.POINTER(hb_decode_mix), C.c_int32, C.POINTER(hb_profile_cell),
                                         C.POINTER(hb_latency_model)]
    lib.hb_fit_latency_model.restype = st
    lib.hb_predict_latency.argtypes = [C.POINTER(hb_latency_model), C.POINTER(hb_layer_config), C.POINTER(hb_request),
                                       C.c_int32, C.POINTER(C.c_double)]
    lib.hb_predict_latency.restype = st
    lib.hb_select_chunk.argtypes = [C.POINTER(hb_latency_model), C.POINTER(hb_layer_config), C.POINTER(C.c_int32),
                                    C.POINTER(C.c_double), C.c_int32, C.c_double, C.c_int32, C.c_int32, C.c_int32,
                                    C.c_double, C.POINTER(C.c_int32), C.POINTER(C.c_double)]
    lib.hb_select_chunk.restype = st
    lib.hb_create_model.argtypes = [C.POINTER(hb_layer_config), C.POINTER(hb_model_desc), C.c_void_p,
                                    C.POINTER(C.c_void_p)]
    lib.hb_create_model.restype = st
    lib.hb_destroy_model.argtypes = [C.c_void_p]
    lib.hb_destroy_model.restype = None
    lib.hb_model_layer.argtypes = [C.c_void_p, C.c_int32]
    lib.hb_model_layer.restype = C.c_void_p
    lib.hb_run_model.argtypes = [C.c_void_p, C.POINTER(hb_model_batch)]
    lib.hb_run_model.restype = st
    lib.hb_set_kernel_timing.argtypes = [C.c_void_p, C.c_uint32]
    lib.hb_set_kernel_timing.restype = st
    lib.hb_kernel_times.argtypes = [C.c_void_p, C.POINTER(C.c_double), C.POINTER(C.c_int64), C.c_int32]
    lib.hb_kernel_times.restype = st
    lib.hb_kernel_name.argtypes = [C.c_int32]
    lib.hb_kernel_name.restype = C.c_char_p
    lib.hb_layer_stage.argtypes = [C.c_void_p, C.c_int32, C.POINTER(C.c_void_p), C.POINTER(C.c_int64)]
    lib.hb_layer_stage.restype = st
    lib.hb_last_error.argtypes = []
    lib.hb_last_error.restype = C.c_char_p
    lib.hb_gemm_tile_count.argtypes = []
    lib.hb_gemm_tile_count.restype = C.c_int32
    lib.hb_plan_gemms.argtypes = [C.POINTER(hb_layer_config), C.c_int32, C.c_int32, C.c_int32, C.c_int32,
                                  C.POINTER(C.c_int32), C.POINTER(C.c_int32)]
    lib.hb_plan_gemms.restype = st
    lib.hb_layer_gemm_plans.argtypes = [C.c_void_p, C.POINTER(C.c_int32), C.POINTER(C.c_int32)]
    lib.hb_layer_gemm_plans.restype = st
    lib.hb_measure_device_rates.argtypes = [C.c_void_p, C.c_int64, C.c_void_p, C.POINTER(hb_device_rates)]
    lib.hb_measure_device_rates.restype = st
    _lib = lib
    return lib


def hb_last_error() -> str:
    return load().hb_last_error().decode()


def _check(status: int) -> None:
    if status != HB_OK:
        raise HBError(status, hb_last_error())


def make_config(shape, max_batch_tokens: int, max_requests: int) -> hb_layer_config:
    """hb_layer_config from any object with the layer-shape attributes."""
    return hb_layer_config(shape.hidden, shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.ffn_dim,
                           getattr(shape, "kv_block", 16), float(shape.rope_theta), float(shape.rms_eps),
                           int(max_batch_tokens), int(max_requests))


class Layer:
    """Owns an hb_layer handle (unless borrowed from a model) and keeps the
    tensors it points at alive."""

    borrowed = False

    def __init__(self, handle: C.c_void_p, cfg: hb_layer_config, keep: list):
        self.handle = handle
        self.cfg = cfg
        self._keep = keep

    def __del__(self):
        try:
            if not self.borrowed:
                hb_destroy_layer(self)
        except Exception:
            pass


class Model:
    """Owns an hb_model handle and keeps the tensors it points at alive."""

    def __init__(self, handle: C.c_void_p, cfg: hb_layer_config, n_layers: int, vocab: int, keep: list):
        self.handle = handle
        self.cfg = cfg
        self.n_layers = n_layers
        self.vocab = vocab
        self._keep = keep

    def layer(self, index: int) -> "Layer":
        """Borrowed handle of layer `index` (the model destroys it)."""
        h = load().hb_model_layer(self.handle, int(index))
        if not h:
            raise IndexError(index)
        lay = Layer(C.c_void_p(h), self.cfg, [self])
        lay.borrowed = True
        return lay

    def __del__(self):
        try:
            hb_destroy_model(self)
        except Exception:
            pass


def hb_create_model(cfg: hb_layer_config, layer_weights: Sequence[Dict[str, "torch.Tensor"]], pools,
                    num_blocks: int, embed, g_final, lm_head, stream: Optional[int] = None) -> Model:
    """pools: [(k_pool, v_pool)] per layer."""
    n = len(layer_weights)
    wa = (hb_layer_weights * n)()
    pa = (hb_kv_pool * n)()
    for i, (w, (kp, vp)) in enumerate(zip(layer_weights, pools)):
        wa[i] = hb_layer_weights(*(_ptr(w[k]) for k in ("w_qkv", "w_o", "w_gate_up", "w_down", "g_attn", "g_ffn")))
        pa[i] = hb_kv_pool(_ptr(kp), _ptr(vp), int(num_blocks))
    vocab = int(embed.shape[0])
    d = hb_model_desc(n, vocab, wa, pa, C.c_void_p(_ptr(embed)), C.c_void_p(_ptr(g_final)), C.c_void_p(_ptr(lm_head)))
    if stream is None:
        import torch
        stream = torch.cuda.current_stream().cuda_stream
    h = C.c_void_p()
    _check(load().hb_create_model(C.byref(cfg), C.byref(d), C.c_void_p(stream), C.byref(h)))
    return Model(h, cfg, n, vocab, [layer_weights, pools, embed, g_final, lm_head])


def hb_destroy_model(model: Model) -> None:
    if model.handle is not None and model.handle.value:
        load().hb_destroy_model(model.handle)
        model.handle = None


def hb_run_model(model: Model, requests: Sequence[Tuple[int, int, Iterable[int]]], token_ids, next_tokens,
                 logits=None, hidden_states=None) -> None:
    """token_ids: device int32 [T]; next_tokens: device int32 [n_requests];
    logits: device fp32 [n_requests][vocab] or None; hidden_states: device
    bf16 [n_layers][T][H] (every layer's output) or None."""
    d, keep = _desc(requests, 0, 0, HB_OUT_BF16)
    b = hb_model_batch(len(requests), d.requests, C.c_void_p(_ptr(token_ids)), C.c_void_p(_ptr(logits)),
                       C.c_void_p(_ptr(next_tokens)), C.c_void_p(_ptr(hidden_states)))
    _check(load().hb_run_model(model.handle, C.byref(b)))


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def hb_create_layer(cfg: hb_layer_config, weights: Dict[str, "torch.Tensor"], k_pool, v_pool,
                    num_blocks: int, stream: Optional[int] = None) -> Layer:
    lib = load()
    w = hb_layer_weights(*(_ptr(weights[n]) for n in ("w_qkv", "w_o", "w_gate_up", "w_down", "g_attn", "g_ffn")))
    pool = hb_kv_pool(_ptr(k_pool), _ptr(v_pool), int(num_blocks))
    if stream is None:
        import torch
        stream = torch.cuda.current_stream().cuda_stream
    h = C.c_void_p()
    _check(lib.hb_create_layer(C.byref(cfg), C.byref(w), C.byref(pool), C.c_void_p(stream), C.byref(h)))
    return Layer(h, cfg, [weights, k_pool, v_pool])


def hb_destroy_layer(layer: Layer) -> None:
    if layer.handle is not None and layer.handle.value:
        load().hb_destroy_layer(layer.handle)
        layer.handle = None


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def hb_append_kv(layer: Layer, block_table, context_len: int, k, v) -> None:
    bt = _i32(block_table)
    n = 0 if k is None else int(k.shape[0])
    _check(load().hb_append_kv(layer.handle, bt.ctypes.data_as(C.POINTER(C.c_int32)), len(bt), int(context_len), n,
                               C.c_void_p(_ptr(k)), C.c_void_p(_ptr(v))))


# hb_request as a NumPy record: the request array is filled with array
# operations instead of one ctypes object per request
_REQ_DTYPE = np.dtype({"names": ["chunk_len", "context_len", "block_table", "n_blocks"],
                       "formats": [np.int32, np.int32, np.uintp, np.int32],
                       "offsets": [hb_request.chunk_len.offset, hb_request.context_len.offset,
                                   hb_request.block_table.offset, hb_request.n_blocks.offset],
                       "itemsize": C.sizeof(hb_request)})


def _desc(requests: Sequence[Tuple[int, int, Iterable[int]]], x_in_ptr: int, x_out_ptr: int, out_dtype: int):
    n = len(requests)
    tables = [_i32(bt) for (_, _, bt) in requests]
    flat = np.concatenate(tables) if n else np.zeros(1, np.int32)
    lens = np.fromiter((len(bt) for bt in tables), dtype=np.int64, count=n)
    rec = np.zeros(max(1, n), dtype=_REQ_DTYPE)
    if n:
        cx = np.array([(r[0], r[1]) for r in requests], dtype=np.int64).reshape(n, 2)
        rec["chunk_len"][:n] = cx[:, 0]
        rec["context_len"][:n] = cx[:, 1]
        starts = np.concatenate([[0], np.cumsum(lens)[:-1]])
        rec["block_table"][:n] = flat.ctypes.data + 4 * starts
        rec["n_blocks"][:n] = lens
    arr = rec.ctypes.data_as(C.POINTER(hb_request))
    d = hb_batch_desc(n, arr, C.c_void_p(x_in_ptr), C.c_void_p(x_out_ptr), int(out_dtype))
    return d, (flat, rec, arr)


def hb_run_iteration(layer: Layer, requests: Sequence[Tuple[int, int, Iterable[int]]], x_in, x_out,
                     out_dtype: Optional[int] = None) -> None:
    """requests: (chunk_len, context_len, block_table) per request, in row order."""
    if out_dtype is None:
        import torch
        out_dtype = HB_OUT_F32 if x_out.dtype == torch.float32 else HB_OUT_BF16
    d, keep = _desc(requests, _ptr(x_in), _ptr(x_out), out_dtype)
    _check(load().hb_run_iteration(layer.handle, C.byref(d)))


def hb_run_iteration_noalloc(layer: Layer, requests: Sequence[Tuple[int, int, Iterable[int]]], x_in, x_out,
                             out_dtype: Optional[int] = None) -> None:
    """As hb_run_iteration, through the allocation-free entry point."""
    if out_dtype is None:
        import torch
        out_dtype = HB_OUT_F32 if x_out.dtype == torch.float32 else HB_OUT_BF16
    d, keep = _desc(requests, _ptr(x_in), _ptr(x_out), out_dtype)
    _check(load().hb_run_iteration_noalloc(layer.handle, C.byref(d)))


def hb_validate_batch(cfg: hb_layer_config, num_blocks: int, requests, x_in_ptr: int, x_out_ptr: int,
                      out_dtype: int = HB_OUT_F32) -> int:
    """Host-only check; returns the status code (no exception)."""
    d, keep = _desc(requests, x_in_ptr, x_out_ptr, out_dtype)
    return load().hb_validate_batch(C.byref(cfg), int(num_blocks), C.byref(d))


def hb_profile(layer: Layer, chunk_sizes: Sequence[int], mixes: Sequence[Tuple[Sequence[int], int]],
               warmup: int = 10, iters: int = 100, seed: int = 0) -> np.ndarray:
    """mixes: (decode_contexts, chunk_context) per row. Returns a structured array [n_mix][n_chunk]."""
    cs = _i32(chunk_sizes)
    ctxs = [_i32(m[0]) for m in mixes]
    marr = (hb_decode_mix * len(mixes))()
    for i, (c, (_, cc)) in enumerate(zip(ctxs, mixes)):
        marr[i] = hb_decode_mix(len(c), c.ctypes.data_as(C.POINTER(C.c_int32)), int(cc))
    out = (hb_profile_cell * (len(mixes) * len(cs)))()
    _check(load().hb_profile(layer.handle, cs.ctypes.data_as(C.POINTER(C.c_int32)), len(cs), marr, len(mixes),
                             int(warmup), int(iters), C.c_uint64(seed), out))
    names = [f[0] for f in hb_profile_cell._fields_]
    res = np.zeros((len(mixes), len(cs)), dtype=[(n, np.float64) for n in names])
    for i in range(len(mixes)):
        for j in range(len(cs)):
            cell = out[i * len(cs) + j]
            res[i, j] = tuple(getattr(cell, n) for n in names)
    return res


def hb_profile_batches(layer: Layer, batches, warmup: int = 3, iters: int = 15) -> np.ndarray:
    """batches: (requests, x_in, x_out) each, requests as for hb_run_iteration.
    Returns a structured array [n_batches] of profile cells."""
    descs = (hb_batch_desc * max(1, len(batches)))()
    keep = []
    for i, (reqs, x_in, x_out) in enumerate(batches):
        import torch
        out_dtype = HB_OUT_F32 if x_out.dtype == torch.float32 else HB_OUT_BF16
        d, k = _desc(reqs, _ptr(x_in), _ptr(x_out), out_dtype)
        descs[i] = d
        keep.append(k)
    out = (hb_profile_cell * max(1, len(batches)))()
    _check(load().hb_profile_batches(layer.handle, descs, len(batches), int(warmup), int(iters), out))
    names = [f[0] for f in hb_profile_cell._fields_]
    res = np.zeros(len(batches), dtype=[(n, np.float64) for n in names])
    for i in range(len(batches)):
        res[i] = tuple(getattr(out[i], n) for n in names)
    return res


def _requests_only(requests: Sequence[Tuple[int, int]]):
    """hb_request array of (chunk_len, context_len) pairs without block tables."""
    arr = (hb_request * max(1, len(requests)))()
    for i, r in enumerate(requests):
        arr[i] = hb_request(int(r[0]), int(r[1]), None, 0)
    return arr


def _mix_array(mixes: Sequence[Tuple[Sequence[int], int]]):
    ctxs = [_i32(m[0]) for m in mixes]
    marr = (hb_decode_mix * len(mixes))()
    for i, (c, (_, cc)) in enumerate(zip(ctxs, mixes)):
        marr[i] = hb_decode_mix(len(c), c.ctypes.data_as(C.POINTER(C.c_int32)), int(cc))
    return marr, ctxs


def hb_latency_features(cfg: hb_layer_config, requests: Sequence[Tuple[int, int]]) -> np.ndarray:
    """requests: (chunk_len, context_len) per request."""
    f = (C.c_double * HB_LAT_FEATURES)()
    _check(load().hb_latency_features(C.byref(cfg), _requests_only(requests), len(requests), f))
    return np.array(f[:], dtype=np.float64)


def hb_fit_latency_model(cfg: hb_layer_config, chunk_sizes: Sequence[int],
                         mixes: Sequence[Tuple[Sequence[int], int]], median_ms) -> hb_latency_model:
    """median_ms[n_mix][n_chunk]: the cells' medians (hb_profile's "median_ms")."""
    cs = _i32(chunk_sizes)
    marr, keep = _mix_array(mixes)
    med = np.asarray(median_ms, dtype=np.float64).reshape(len(mixes), len(cs))
    cells = (hb_profile_cell * med.size)()
    for i in range(len(mixes)):
        for j in range(len(cs)):
            cells[i * len(cs) + j].median_ms = float(med[i, j])
    model = hb_latency_model()
    _check(load().hb_fit_latency_model(C.byref(cfg), cs.ctypes.data_as(C.POINTER(C.c_int32)), len(cs), marr,
                                       len(mixes), cells, C.byref(model)))
    return model


def hb_predict_latency(model: hb_latency_model, cfg: hb_layer_config, requests: Sequence[Tuple[int, int]]) -> float:
    ms = C.c_double()
    _check(load().hb_predict_latency(C.byref(model), C.byref(cfg), _requests_only(requests), len(requests),
                                     C.byref(ms)))
    return ms.value


def hb_select_chunk(model: hb_latency_model, cfg: hb_layer_config, decode_contexts: Sequence[int],
                    decode_deadlines_ms: Sequence[float], now_ms: float, chunk_context: int, max_chunk: int,
                    granularity: int, margin: float = 0.0) -> Tuple[int, float]:
    ctx = _i32(decode_contexts)
    dl = np.ascontiguousarray(decode_deadlines_ms, dtype=np.float64)
    chunk, ms = C.c_int32(), C.c_double()
    _check(load().hb_select_chunk(C.byref(model), C.byref(cfg), ctx.ctypes.data_as(C.POINTER(C.c_int32)),
                                  dl.ctypes.data_as(C.POINTER(C.c_double)), len(ctx), float(now_ms),
                                  int(chunk_context), int(max_chunk), int(granularity), float(margin),
                                  C.byref(chunk), C.byref(ms)))
    return chunk.value, ms.value


def hb_set_kernel_timing(layer: Layer, kernels) -> None:
    """kernels: True (all), False (none) or an iterable of kernel names."""
    if kernels is True:
        mask = (1 << HB_K_COUNT) - 1
    elif kernels is False or kernels is None:
        mask = 0
    else:
        names = [hb_kernel_name(k) for k in range(HB_K_COUNT)]
        mask = 0
        for n in kernels:
            mask |= 1 << names.index(n)
    _check(load().hb_set_kernel_timing(layer.handle, mask))


def hb_kernel_times(layer: Layer, reset: bool = False) -> Dict[str, Tuple[float, int]]:
    ms = (C.c_double * HB_K_COUNT)()
    n = (C.c_int64 * HB_K_COUNT)()
    _check(load().hb_kernel_times(layer.handle, ms, n, 1 if reset else 0))
    return {hb_kernel_name(k): (ms[k], n[k]) for k in range(HB_K_COUNT)}


def hb_kernel_name(k: int) -> str:
    return load().hb_kernel_name(int(k)).decode()


def hb_gemm_tile_count() -> int:
    return int(load().hb_gemm_tile_count())


def hb_plan_gemms(cfg: hb_layer_config, n_tokens: int, cu_count: int, force_tile: int = -1,
                  force_ksplit: int = 0) -> List[Tuple[int, int]]:
    """(tile, ksplit) of the QKV, O, gate/up and down GEMMs for a batch of n_tokens."""
    t, k = (C.c_int32 * HB_GEMM_COUNT)(), (C.c_int32 * HB_GEMM_COUNT)()
    _check(load().hb_plan_gemms(C.byref(cfg), int(n_tokens), int(cu_count), int(force_tile), int(force_ksplit), t, k))
    return [(t[i], k[i]) for i in range(HB_GEMM_COUNT)]


def hb_layer_gemm_plans(layer: Layer) -> List[Tuple[int, int]]:
    """(tile, ksplit) of each GEMM of the layer's most recent iteration."""
    t, k = (C.c_int32 * HB_GEMM_COUNT)(), (C.c_int32 * HB_GEMM_COUNT)()
    _check(load().hb_layer_gemm_plans(layer.handle, t, k))
    return [(t[i], k[i]) for i in range(HB_GEMM_COUNT)]


def hb_layer_stage(layer: Layer, stage: int) -> Tuple[int, int]:
    p = C.c_void_p()
    s = C.c_int64()
    _check(load().hb_layer_stage(layer.handle, int(stage), C.byref(p), C.byref(s)))
    return int(p.value or 0), int(s.value)


def hb_measure_device_rates(buf, stream=None) -> Dict[str, float]:
    """Sustained random-4-KB read, streaming read and bf16 MFMA rates of the
    current device; buf: a device tensor of at least 1 GiB (scratch)."""
    r = hb_device_rates()
    s = 0 if stream is None else int(stream.cuda_stream)
    _check(load().hb_measure_device_rates(C.c_void_p(buf.data_ptr()), int(buf.numel() * buf.element_size()),
                                          C.c_void_p(s), C.byref(r)))
    return {f[0]: float(getattr(r, f[0])) for f in hb_device_rates._fields_}
