"""CPU oracle for the hybrid-batch decoder layer (test infrastructure only).

Imported by the tests, the smoke check and the benchmark's CPU-baseline leg;
never by the library.
"""
from .layer import (PagedKVCache, bf16_bits_to_f64, causal_attention, kv_slot,
                    layer_forward, linear, rmsnorm, rope, rope_angles, seed_cache,
                    silu, swiglu_mlp, weights_to_f64)

__all__ = ["PagedKVCache", "bf16_bits_to_f64", "causal_attention", "kv_slot",
           "layer_forward", "linear", "rmsnorm", "rope", "rope_angles", "seed_cache",
           "silu", "swiglu_mlp", "weights_to_f64"]
