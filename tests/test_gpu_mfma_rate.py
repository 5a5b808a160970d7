"""The register-only MFMA rate (a measurement aid the benchmark reports next
to the roofline): positive, below the chip's dense bf16 peak, and no slower
on zero operands than on random ones (zeros toggle no bits)."""
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
