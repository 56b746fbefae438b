"""The seeded workload module on the CPU: tensor-parallel shard shapes."""
import pytest

from hb_workloads import LLAMA3_8B, LLAMA3_8B_TP2, LLAMA3_70B, LLAMA3_70B_TP8, tp_shard


def test_shards_hold_one_tp_th_of_the_linear_weights():
    """Sharded by heads, every linear layer splits evenly when tp divides the
    kv heads: a shard holds exactly 1/tp of the layer's linear parameters at
    the full hidden size."""
    for full, shard, tp in ((LLAMA3_8B, LLAMA3_8B_TP2, 2), (LLAMA3_70B, LLAMA3_70B_TP8, 8)):
        assert shard.hidden == full.hidden and shard.head_dim == full.head_dim
        assert shard.n_q_heads * tp == full.n_q_heads and shard.n_kv_heads * tp == full.n_kv_heads
        assert shard.ffn_dim * tp == full.ffn_dim and shard.qkv_dim * tp == full.qkv_dim
        assert shard.linear_params * tp == full.linear_params
        assert shard.weight_seed != full.weight_seed


def test_shard_beyond_the_kv_heads_replicates_them():
    s = tp_shard(LLAMA3_70B, 16, weight_seed=1)
    assert (s.n_q_heads, s.n_kv_heads, s.ffn_dim) == (4, 1, 1792)


def test_uneven_shard_is_refused():
    with pytest.raises(ValueError):
        tp_shard(LLAMA3_8B, 3, weight_seed=1)
