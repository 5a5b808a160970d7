"""The measurement aids the benchmark reports next to the roofline: the
register-only MFMA rate (positive, below the chip's dense bf16 peak, no
slower on zero operands than on random ones), the MFMA rate under the
attention loop's instruction mix (no faster than the register-only loop, the
combined mix no faster than either part), and the global -> LDS request
stream rate (positive, below what 256 CUs can take in)."""
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

PEAK_BF16_TFLOPS = 2500.0


@pytest.mark.parametrize("shape", [0, 1], ids=["32x32x16", "16x16x32"])
def test_mfma_rate_is_plausible(shape):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_20289_amd import xcache as xcp
    stream = torch.cuda.current_stream().cuda_stream
    print(f"[mfma-rate] shape {shape}", flush=True)
    rnd = xcp.xc_mfma_rate(shape, True, stream)
    zero = xcp.xc_mfma_rate(shape, False, stream)
    print(f"[mfma-rate] random {rnd:.0f} TFLOP/s, zeros {zero:.0f} TFLOP/s", flush=True)
    assert 100.0 < rnd <= 1.05 * PEAK_BF16_TFLOPS
    assert 100.0 < zero <= 1.05 * PEAK_BF16_TFLOPS
    assert zero >= 0.9 * rnd


def test_attention_mix_rates_are_plausible():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_20289_amd import xcache as xcp
    stream = torch.cuda.current_stream().cuda_stream
    print("[mfma-mix] register-only 32x32x16, then + LDS reads, + softmax VALU, both", flush=True)
    base = xcp.xc_mfma_rate(0, True, stream)
    lds, valu, both = (xcp.xc_mfma_rate(s, True, stream) for s in (2, 3, 4))
    print(f"[mfma-mix] {base:.0f} / {lds:.0f} / {valu:.0f} / {both:.0f} TFLOP/s", flush=True)
    for r in (lds, valu, both):
        assert 100.0 < r <= 1.05 * base
    assert both <= 1.05 * min(lds, valu)


@pytest.mark.parametrize("row_bytes", [64, 128, 256])
def test_lds_dma_rate_is_plausible(row_bytes):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_20289_amd import xcache as xcp
    print(f"[lds-dma-rate] {row_bytes} B rows", flush=True)
    r = xcp.xc_lds_dma_rate(row_bytes, torch.cuda.current_stream().cuda_stream)
    print(f"[lds-dma-rate] {r:.2f} TB/s", flush=True)
    assert 0.5 < r < 100.0
