"""GPU parity of the Jacobian-contraction baseline (NTK_METHOD_JACOBIAN) (needs an MI355X).

The baseline forms every weight tensor's per-sample Jacobian block explicitly and contracts
J(x1) J(x2)^T on the GPU; its Theta must match the fp64 oracle to the same bar as the
structured method, for every output/batch variant, and agree with the structured method.
"""
import numpy as np
import pytest

import oracle
import workloads as wl
from tests.gpu_helpers import (TOL, errors, gpu_ntk, report, scaled_errors, variant_of,
                               variant_scale)

pytestmark = pytest.mark.gpu
S = "fp32"
VARIANTS = [("full", "full"), ("trace", "full"), ("logit", "full"), ("full", "diagonal"),
            ("trace", "diagonal"), ("logit", "diagonal")]
VIDS = [f"{o}-{b}" for o, b in VARIANTS]


def _jc(spec, params, X1, X2, symmetric=True, variant=("full", "full", 0), handle=None):
    from paper_2206_08720_amd import _lib
    return gpu_ntk(spec, params, X1, X2, symmetric=symmetric, handle=handle, variant=variant,
                   options={_lib.NTK_OPT_METHOD: _lib.NTK_METHOD_JACOBIAN})


CASES = [
    ("tiny relu mlp with biases", wl.fcn_spec("j1", 16, [32, 32], 4, bias=True), 8, 8),
    ("relu 40-72-56-9, ragged", wl.fcn_spec("j2", 40, [72, 56], 9), 21, 21),
    ("readout only, bias", wl.fcn_spec("j3", 6, [], 4, bias=True), 5, 5),
    ("cnn 5x6, 2 conv layers", wl.cnn_spec("j4", (5, 6), 3, [8, 12], 5), 6, 6),
    ("cnn erf 4x4, O=3", wl.cnn_spec("j5", (4, 4), 2, [10], 3, act="erf"), 7, 7),
]


@pytest.mark.parametrize("variant", VARIANTS, ids=VIDS)
@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_jacobian_contraction_variants(case, variant):
    label, spec, n1, n2 = case
    params = wl.make_params(spec, 1700 + n1, "2/fan_in", bias_var=0.1)
    X1 = wl.make_inputs(spec, n1, 1800 + n1)
    X2 = wl.make_inputs(spec, n2, 1900 + n2)
    O = spec["layers"][-1]["out"]
    output, batch = variant
    logit = 1 if output == "logit" else 0
    for xa, xb, sym in ((X1, X2, True), (X1, X1, True), (X1, X1, False)):
        full, d1, d2 = oracle.ntk_jc_with_norms(spec, params, xa, xb, layer_storage=S)
        got = _jc(spec, params, xa, xb, symmetric=sym, variant=(output, batch, logit))
        ref = variant_of(full, output, batch, logit)
        cs, nw = scaled_errors(got, ref, variant_scale(d1, d2, output, batch, logit))
        report(f"JC {label} {output}/{batch} aliased={xb is xa} sym={sym}", cs, nw)
        assert got.shape == ref.shape
        assert cs <= TOL and nw <= TOL


@pytest.mark.parametrize("name", ["relu_mlp_d4_w512", "cnn4_c64_32x32"])
def test_jacobian_contraction_full_workloads_match_structured(name):
    spec, params, X1, X2 = wl.make_workload(name)
    sd = gpu_ntk(spec, params, X1, X2)
    jc = _jc(spec, params, X1, X2)
    if name == "cnn4_c64_32x32":
        ref, d1, d2 = oracle.ntk_jc_with_norms(spec, params, X1, X2, layer_storage=S)
    else:
        ref = oracle.ntk_structured_fp64(spec, params, X1, X2, layer_storage=S)
        d1 = d2 = oracle.ntk_structured_diag_fp64(spec, params, X1, layer_storage=S)
    for label, got in (("JC", jc), ("SD", sd)):
        cs, nw = errors(got, ref, d1, d2)
        report(f"{name} {label} vs fp64", cs, nw)
        assert cs <= TOL and nw <= TOL
    cs, nw = errors(jc, sd.astype(np.float64), d1, d2)
    report(f"{name} JC vs SD", cs, nw)
    assert cs <= 2 * TOL


def test_jacobian_contraction_subset_of_depth8_width2048():
    # 24 + 20 samples of the depth-8 width-2048 FCN: 2 N1 N2 O^2 P = 6.3e12 FLOPs
    spec, params, X1, X2 = wl.make_workload("relu_mlp_d8_w2048")
    X1, X2 = X1[:24], X2[:20]
    got = _jc(spec, params, X1, X2)
    ref = oracle.ntk_structured_fp64(spec, params, X1, X2, layer_storage=S)
    d1 = oracle.ntk_structured_diag_fp64(spec, params, X1, layer_storage=S)
    d2 = oracle.ntk_structured_diag_fp64(spec, params, X2, layer_storage=S)
    cs, nw = errors(got, ref, d1, d2)
    report("relu_mlp_d8_w2048[:24, :20] JC", cs, nw)
    assert cs <= TOL and nw <= TOL


def test_jacobian_contraction_handle_reuse_is_deterministic():
    from paper_2206_08720_amd.ntk import NTK
    spec = wl.fcn_spec("jr", 12, [20, 16], 3, bias=True)
    params = wl.make_params(spec, 3, bias_var=0.1)
    X1 = wl.make_inputs(spec, 9, 4)
    X2 = wl.make_inputs(spec, 7, 5)
    h = NTK(spec, 9, 9)
    try:
        a = _jc(spec, params, X1, X2, handle=h)
        b = _jc(spec, params, X1, X2, handle=h)
        assert np.array_equal(a, b)
        c = _jc(spec, params, X1[:4], X2[:3], handle=h)
        ref, d1, d2 = oracle.ntk_jc_with_norms(spec, params, X1[:4], X2[:3], layer_storage=S)
        cs, nw = errors(c, ref, d1, d2)
        assert cs <= TOL and nw <= TOL
    finally:
        h.close()
