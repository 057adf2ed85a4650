"""Device diagnostics on the GPU: compute-unit count and the measured MFMA ceilings."""
import pytest

pytestmark = pytest.mark.gpu


def test_device_info_and_mfma_ceilings():
    from paper_2206_08720_amd import _lib
    cu, clk = _lib.device_info()
    assert cu > 0 and clk > 0
    f32 = _lib.mfma_peak("fp32")
    f64 = _lib.mfma_peak("fp64")
    print(f"[diag] {cu} CUs, {clk / 1000:.0f} MHz, fp32 MFMA {f32:.1f} TFLOP/s, fp64 {f64:.1f}")
    # a chain of independent MFMAs must reach a sizeable part of the nominal rate
    # (256 FLOP/clk/CU fp32, 128 fp64) and cannot exceed it
    nominal32 = cu * 256 * clk * 1e3 / 1e12
    assert 0.3 * nominal32 < f32 <= 1.05 * nominal32
    assert 0.3 * nominal32 / 2 < f64 <= 1.05 * nominal32 / 2
