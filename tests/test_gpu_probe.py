"""The device-rate probes (hb_measure_device_rates) on the GPU: every rate is
positive and no rate beats the published peak it is read against (HBM
8 TB/s, dense bf16 MFMA 2.5 PFLOP/s), with 2 % allowance for timer
resolution."""
import pytest

pytestmark = pytest.mark.gpu


def test_device_rates_within_published_peaks(hb):
    import torch
    buf = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    r = hb.hb_measure_device_rates(buf)
    print({k: f"{v:.4g}" for k, v in r.items()})
    assert 1e12 < r["random_4kb_read_bytes_per_s"] <= 8.0e12 * 1.02
    assert 1e12 < r["stream_read_bytes_per_s"] <= 8.0e12 * 1.02
    assert 2e14 < r["mfma_bf16_flop_per_s"] <= 2.5e15 * 1.02
    # the same stream, a second time: the result is a property of the device
    r2 = hb.hb_measure_device_rates(buf, torch.cuda.current_stream())
    for k in r:
        assert abs(r2[k] / r[k] - 1) < 0.25, (k, r[k], r2[k])
