"""Creating, running and destroying layers and models repeatedly gives their
device memory back: the device's free memory (hipMemGetInfo, which counts the
library's own allocations as well as torch's) after 20 more cycles is where
it was after the first one, within 8 MiB."""
import gc

import pytest

from hb_workloads import TINY, make_model_weights, make_weights, tiny_batch

pytestmark = pytest.mark.gpu


def _free_bytes(torch):
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return torch.cuda.mem_get_info()[0]


def test_layers_and_models_release_device_memory(hb):
    import torch
    from paper_2503_22562_amd.harness import DeviceLayer, DeviceModel, to_device_bf16
    b = tiny_batch()
    w = make_weights(b.shape)
    mw = make_model_weights(TINY, 2, 200)
    reqs = [(r.chunk_len, r.context_len, r.block_table) for r in b.requests]
    ids = b.token_ids(200)

    def cycle():
        dl = DeviceLayer(b.shape, w, b.num_blocks, b.n_tokens, len(b.requests))
        dl.run(reqs, to_device_bf16(b.x_in()))
        dm = DeviceModel(b.shape, mw, b.num_blocks, b.n_tokens, len(b.requests))
        dm.run(reqs, ids)
        torch.cuda.synchronize()
        del dl, dm

    cycle()
    base = _free_bytes(torch)
    for _ in range(20):
        cycle()
    after = _free_bytes(torch)
    print(f"free after one cycle {base >> 20} MiB, after 20 more {after >> 20} MiB")
    assert base - after <= 8 << 20
