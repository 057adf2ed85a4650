"""MI355X (gfx950) structured-derivatives empirical NTK.

The compute lives in the HIP library `libntk.so` (C ABI in include/ntk.h);
`paper_2206_08720_amd.ntk` is the thin PyTorch-facing binding, and
`paper_2206_08720_amd.flops` the analytic operation counter.  Import the
submodules explicitly; this package module itself loads nothing.
"""
__all__ = ["ntk", "flops", "build"]
