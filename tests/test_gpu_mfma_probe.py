"""The fp32 matrix-core probe behind bench.py's measured ceiling: its counters
advance, the clock it implies is a plausible shader clock, and the rate it
sustains stays within what 256 CUs x 4 SIMDs x one 4096-flop MFMA per 64
cycles allow at that clock (157.3 TFLOP/s at 2.4 GHz)."""
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


def test_mfma_probe_rate_and_clock():
    import paper_2609_33591_amd as kia
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    wg, iters = 4 * cus, 512
    out = torch.zeros(4, dtype=torch.int64, device="cuda")
    kia.kia_mfma_peak_probe(out, wg, iters)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    kia.kia_mfma_peak_probe(out, wg, iters)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b)
    t0, t1, r0, r1 = out.cpu().tolist()
    assert t1 > t0 and r1 > r0
    clock_ghz = (t1 - t0) / (r1 - r0) * 0.1
    assert 0.5 < clock_ghz < 3.0
    tflops = wg * 4 * iters * 4 * 4096 / (ms * 1e-3) / 1e12
    per_clock = cus * 4 * 4096 / 64  # flops per shader cycle, whole chip
    assert 10.0 < tflops <= per_clock * 2.4e9 / 1e12 * 1.02


def test_mfma_probe_rejects_bad_sizes():
    import paper_2609_33591_amd as kia
    out = torch.zeros(4, dtype=torch.int64, device="cuda")
    with pytest.raises(kia.KiaError):
        kia.kia_mfma_peak_probe(out, 0, 16)
