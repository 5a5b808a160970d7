"""The measurement aids the benchmark reports next to the roofline: the
register-only MFMA rate (positive, below the chip's dense bf16 peak, no
slower on zero operands than on random ones) and the global -> LDS request
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


@pytest.mark.parametrize("row_bytes", [64, 128, 256])
def test_lds_dma_rate_is_plausible(row_bytes):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_20289_amd import xcache as xcp
    print(f"[lds-dma-rate] {row_bytes} B rows", flush=True)
    r = xcp.xc_lds_dma_rate(row_bytes, torch.cuda.current_stream().cuda_stream)
    print(f"[lds-dma-rate] {r:.2f} TB/s", flush=True)
    assert 0.5 < r < 100.0
