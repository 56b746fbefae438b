"""Device-memory plumbing around the binding: upload bf16 arrays, allocate a
paged pool, create a layer and read back intermediate buffers. PyTorch is
used for allocation and streams only; all layer arithmetic runs in libhb.
"""
from __future__ import annotations

import ctypes as C
from typing import Dict, Optional, Sequence, Tuple

import numpy as np

from . import hb

WEIGHT_NAMES = ("w_qkv", "w_o", "w_gate_up", "w_down", "g_attn", "g_ffn")
SENTINEL_BITS = 0xFFFF  # a NaN pattern no computed value takes


def _torch():
    import torch
    return torch


def to_device_bf16(bits: np.ndarray, device: str = "cuda"):
    torch = _torch()
    b = np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16)
    return torch.from_numpy(b).to(device).view(torch.bfloat16)


def k_by_slot(k_bits: np.ndarray) -> np.ndarray:
    """View a K pool [blocks][kv][16][hd] whose blocks are stored as
    [slot group 2][hd / 8][8 slots][8 dims] (group 0: slots 0-3 and 8-11,
    group 1: slots 4-7 and 12-15) as [blocks][kv][slot][hd]."""
    nb, nkv, _, hd = k_bits.shape
    x = k_bits.reshape(nb, nkv, 2, hd // 8, 8, 8).transpose(0, 1, 2, 4, 3, 5).reshape(nb, nkv, 2, 8, hd)
    s = np.arange(16)
    return x[:, :, (s >> 2) & 1, ((s >> 3) << 2) | (s & 3), :]


def v_by_slot(v_bits: np.ndarray) -> np.ndarray:
    """View a V pool [blocks][kv][2][hd][8] as [blocks][kv][slot][hd]."""
    nb, nkv, _, hd, _ = v_bits.shape
    return v_bits.transpose(0, 1, 2, 4, 3).reshape(nb, nkv, 16, hd)


def bf16_bits(t) -> np.ndarray:
    """uint16 bit patterns of a bf16 tensor (copied to host)."""
    torch = _torch()
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)


_hip = None


def _hip_memcpy_d2d(dst: int, src: int, nbytes: int) -> None:
    global _hip
    if _hip is None:
        hb.load()  # binds the HIP runtime torch loaded
        _hip = C.CDLL("libamdhip64.so.7")
        _hip.hipMemcpy.argtypes = [C.c_void_p, C.c_void_p, C.c_size_t, C.c_int]
        _hip.hipMemcpy.restype = C.c_int
    rc = _hip.hipMemcpy(C.c_void_p(dst), C.c_void_p(src), C.c_size_t(nbytes), 3)  # device to device
    if rc != 0:
        raise RuntimeError(f"hipMemcpy failed with {rc}")


class DeviceLayer:
    """A layer, its weights and its paged KV pool on the current GPU."""

    def __init__(self, shape, weights_bits: Dict[str, np.ndarray], num_blocks: int, max_batch_tokens: int,
                 max_requests: int, pool_fill_bits: Optional[int] = SENTINEL_BITS, device: str = "cuda"):
        torch = _torch()
        self.shape = shape
        self.device = device
        self.num_blocks = int(num_blocks)
        self.w = {n: to_device_bf16(weights_bits[n], device) for n in WEIGHT_NAMES}
        nkv, hd = shape.n_kv_heads, shape.head_dim
        self.k_pool = torch.empty((num_blocks, nkv, 16, hd), dtype=torch.bfloat16, device=device)
        self.v_pool = torch.empty((num_blocks, nkv, 2, hd, 8), dtype=torch.bfloat16, device=device)
        if pool_fill_bits is not None:
            fill = int(np.array([pool_fill_bits], dtype=np.uint16).view(np.int16)[0])
            self.k_pool.view(torch.int16).fill_(fill)
            self.v_pool.view(torch.int16).fill_(fill)
        self.cfg = hb.make_config(shape, max_batch_tokens, max_requests)
        self.layer = hb.hb_create_layer(self.cfg, self.w, self.k_pool, self.v_pool, num_blocks)

    def append_kv(self, block_table, context_len: int, k_bits: np.ndarray, v_bits: np.ndarray) -> None:
        if k_bits.shape[0] == 0:
            return
        k = to_device_bf16(k_bits, self.device)
        v = to_device_bf16(v_bits, self.device)
        hb.hb_append_kv(self.layer, block_table, context_len, k, v)
        _torch().cuda.current_stream().synchronize()  # k, v are freed on return

    def run(self, requests: Sequence[Tuple[int, int, np.ndarray]], x_in, out_dtype: int = hb.HB_OUT_F32,
            x_out=None):
        torch = _torch()
        T = int(sum(r[0] for r in requests))
        if x_out is None:
            dt = torch.float32 if out_dtype == hb.HB_OUT_F32 else torch.bfloat16
            x_out = torch.empty((T, self.shape.hidden), dtype=dt, device=self.device)
        hb.hb_run_iteration(self.layer, requests, x_in, x_out, out_dtype)
        return x_out

    def stage(self, which: int, T: int):
        """Copy of an intermediate buffer of the last iteration, [T][cols]."""
        torch = _torch()
        ptr, stride = hb.hb_layer_stage(self.layer, which)
        dt = torch.float32 if which == hb.HB_STAGE_H2 else torch.bfloat16
        out = torch.empty((T, stride), dtype=dt, device=self.device)
        torch.cuda.synchronize()
        _hip_memcpy_d2d(out.data_ptr(), ptr, out.numel() * out.element_size())
        return out


class DeviceModel:
    """A whole model (hb_model): per-layer weights and paged pools, token
    embedding, final gain and LM head on the current GPU."""

    def __init__(self, shape, model_bits: Dict, num_blocks: int, max_batch_tokens: int, max_requests: int,
                 pool_fill_bits: Optional[int] = 0, device: str = "cuda"):
        torch = _torch()
        self.shape = shape
        self.device = device
        self.num_blocks = int(num_blocks)
        self.w = [{n: to_device_bf16(lw[n], device) for n in WEIGHT_NAMES} for lw in model_bits["layers"]]
        nkv, hd = shape.n_kv_heads, shape.head_dim
        self.pools = []
        for _ in self.w:
            k = torch.empty((num_blocks, nkv, 16, hd), dtype=torch.bfloat16, device=device)
            v = torch.empty((num_blocks, nkv, 2, hd, 8), dtype=torch.bfloat16, device=device)
            if pool_fill_bits is not None:
                fill = int(np.array([pool_fill_bits], dtype=np.uint16).view(np.int16)[0])
                k.view(torch.int16).fill_(fill)
                v.view(torch.int16).fill_(fill)
            self.pools.append((k, v))
        self.embed = to_device_bf16(model_bits["embed"], device)
        self.lm_head = to_device_bf16(model_bits["lm_head"], device)
        self.g_final = to_device_bf16(model_bits["g_final"], device)
        self.vocab = int(self.embed.shape[0])
        self.cfg = hb.make_config(shape, max_batch_tokens, max_requests)
        self.model = hb.hb_create_model(self.cfg, self.w, self.pools, num_blocks, self.embed, self.g_final,
                                        self.lm_head)

    def append_kv(self, layer: int, block_table, context_len: int, k_bits: np.ndarray, v_bits: np.ndarray) -> None:
        if k_bits.shape[0] == 0:
            return
        k = to_device_bf16(k_bits, self.device)
        v = to_device_bf16(v_bits, self.device)
        hb.hb_append_kv(self.model.layer(layer), block_table, context_len, k, v)
        _torch().cuda.current_stream().synchronize()  # k, v are freed on return

    def run(self, requests: Sequence[Tuple[int, int, np.ndarray]], token_ids: np.ndarray, keep_logits: bool = True,
            hidden_states=None):
        """Enqueue one model iteration; returns (next_tokens int32 [R], logits fp32 [R][vocab] or None).
        hidden_states: None, or a device bf16 [n_layers][T][H] tensor that receives every layer's output."""
        torch = _torch()
        ids = torch.from_numpy(np.ascontiguousarray(token_ids, dtype=np.int32)).to(self.device)
        nxt = torch.empty(len(requests), dtype=torch.int32, device=self.device)
        logits = torch.empty((len(requests), self.vocab), dtype=torch.float32, device=self.device) if keep_logits else None
        hb.hb_run_model(self.model, requests, ids, nxt, logits, hidden_states)
        self._ids = ids  # alive until the caller synchronises
        return nxt, logits
