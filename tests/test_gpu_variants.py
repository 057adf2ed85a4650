"""GPU parity of the output- and batch-axis variants against the fp64 oracle (needs an MI355X).

Variants (NTK_OPT_OUTPUT / NTK_OPT_BATCH): the trace over outputs, one logit, the batch
diagonal, and their combinations.  The references are the corresponding parts of the
oracle's full Theta (float32 layer storage, see tests/test_gpu_fcn.py), compared with the
per-entry Cauchy-Schwarz error scale of each variant.
"""
import numpy as np
import pytest

import oracle
import workloads as wl
from tests.gpu_helpers import TOL, gpu_ntk, report, scaled_errors, variant_of, variant_scale

pytestmark = pytest.mark.gpu
S = "fp32"
VARIANTS = [("trace", "full"), ("logit", "full"), ("full", "diagonal"), ("trace", "diagonal"),
            ("logit", "diagonal")]
VIDS = [f"{o}-{b}" for o, b in VARIANTS]


def _check(name, spec, params, X1, X2, ref_full, d1, d2, output, batch, symmetric=True,
           options=None):
    O = spec["layers"][-1]["out"]
    logit = O - 1 if output == "logit" else 0
    got = gpu_ntk(spec, params, X1, X2, symmetric=symmetric, options=options,
                  variant=(output, batch, logit))
    ref = variant_of(ref_full, output, batch, logit)
    scale = variant_scale(d1, d2, output, batch, logit)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    cs, nw = scaled_errors(got, ref, scale)
    report(f"{name} {output}/{batch} sym={symmetric}", cs, nw)
    assert cs <= TOL and nw <= TOL


# ---- fully-connected nets, Jacobian-contraction oracle ------------------------------------
FCN_CASES = [
    ("tiny relu mlp with biases", wl.fcn_spec("v1", 16, [32, 32], 4, bias=True), 8, 8),
    ("ragged relu 64-96-80-7, two split-K tiles", wl.fcn_spec("v2", 64, [96, 80], 7), 150, 150),
    ("readout only (no hidden layer), bias", wl.fcn_spec("v3", 6, [], 4, bias=True), 5, 5),
    ("erf 24-40-3", wl.fcn_spec("v4", 24, [40], 3, act="erf"), 33, 33),
]


@pytest.mark.parametrize("variant", VARIANTS, ids=VIDS)
@pytest.mark.parametrize("case", FCN_CASES, ids=[c[0] for c in FCN_CASES])
def test_fcn_variants(case, variant):
    label, spec, n1, n2 = case
    params = wl.make_params(spec, 1100 + n1, "2/fan_in", bias_var=0.1)
    X1 = wl.make_inputs(spec, n1, 1200 + n1)
    X2 = wl.make_inputs(spec, n2, 1300 + n2)
    full, d1, d2 = oracle.ntk_jc_with_norms(spec, params, X1, X2, layer_storage=S)
    _check(label, spec, params, X1, X2, full, d1, d2, *variant)
    fx, dx, _ = oracle.ntk_jc_with_norms(spec, params, X1, X1, layer_storage=S)
    for sym in (True, False):
        _check(label + " aliased", spec, params, X1, X1, fx, dx, dx, *variant, symmetric=sym)


@pytest.fixture(scope="module")
def c3_reference():
    spec, params, X1, X2 = wl.make_workload("relu_mlp_d8_w2048")
    ref = oracle.ntk_structured_fp64(spec, params, X1, X2, layer_storage=S)
    d1 = oracle.ntk_structured_diag_fp64(spec, params, X1, layer_storage=S)
    d2 = oracle.ntk_structured_diag_fp64(spec, params, X2, layer_storage=S)
    return spec, params, X1, X2, ref, d1, d2


@pytest.mark.parametrize("variant", VARIANTS, ids=VIDS)
def test_relu_mlp_d8_w2048_variants_full_size(c3_reference, variant):
    # against the fp64 structured reference (pinned to the Jacobian contraction)
    spec, params, X1, X2, ref, d1, d2 = c3_reference
    _check("relu_mlp_d8_w2048", spec, params, X1, X2, ref, d1, d2, *variant)


@pytest.mark.parametrize("variant", VARIANTS, ids=VIDS)
def test_relu_mlp_d4_w512_variants_aliased(variant):
    spec, params, X1, X2 = wl.make_workload("relu_mlp_d4_w512")
    ref = oracle.ntk_structured_fp64(spec, params, X1, X1, layer_storage=S)
    d = oracle.ntk_structured_diag_fp64(spec, params, X1, layer_storage=S)
    for sym in (True, False):
        _check("relu_mlp_d4_w512", spec, params, X1, X1, ref, d, d, *variant, symmetric=sym)


# ---- convolutional nets: both contraction orders --------------------------------------------
CNN_CASES = [
    ("outside-in 5x6", wl.cnn_spec("w1", (5, 6), 3, [8, 12], 5), "outside_in", 6, 6),
    ("inside-out D=16", wl.cnn_spec("w2", (4, 4), 3, [16, 16], 6), "inside_out", 7, 7),
    ("auto, mixed orders D=16", wl.cnn_spec("w3", (4, 4), 3, [64, 64, 64], 10), "auto", 5, 5),
    ("erf inside-out D=9, O=3", wl.cnn_spec("w4", (3, 3), 2, [10], 3, act="erf"), "inside_out", 4, 4),
    ("inside-out D=25, O=20 (two output blocks)", wl.cnn_spec("w5", (5, 5), 3, [12, 12], 20), "inside_out", 5, 5),
    ("inside-out D=64, O=18", wl.cnn_spec("w6", (8, 8), 4, [16], 18), "inside_out", 6, 6),
]


@pytest.mark.parametrize("variant", VARIANTS, ids=VIDS)
@pytest.mark.parametrize("case", CNN_CASES, ids=[c[0] for c in CNN_CASES])
def test_cnn_variants(case, variant):
    from paper_2206_08720_amd import _lib
    label, spec, order, n1, n2 = case
    code = {"outside_in": _lib.NTK_CONV_ORDER_OUTSIDE_IN, "inside_out": _lib.NTK_CONV_ORDER_INSIDE_OUT,
            "auto": _lib.NTK_CONV_ORDER_AUTO}[order]
    opts = {_lib.NTK_OPT_CONV_ORDER: code}
    params = wl.make_params(spec, 1400 + n1, "2/fan_in")
    X1 = wl.make_inputs(spec, n1, 1500 + n1)
    X2 = wl.make_inputs(spec, n2, 1600 + n2)
    full, d1, d2 = oracle.ntk_jc_with_norms(spec, params, X1, X2, layer_storage=S)
    _check(label, spec, params, X1, X2, full, d1, d2, *variant, options=opts)
    fx, dx, _ = oracle.ntk_jc_with_norms(spec, params, X1, X1, layer_storage=S)
    for sym in (True, False):
        _check(label + " aliased", spec, params, X1, X1, fx, dx, dx, *variant, symmetric=sym,
               options=opts)


@pytest.fixture(scope="module")
def c5_reference():
    spec, params, X1, X2 = wl.make_workload("cnn4_c64_32x32")
    ref, d1, d2 = oracle.ntk_jc_with_norms(spec, params, X1, X2, layer_storage=S)
    return spec, params, X1, X2, ref, d1, d2


@pytest.mark.parametrize("variant", VARIANTS, ids=VIDS)
def test_cnn4_c64_32x32_variants_full_size(c5_reference, variant):
    spec, params, X1, X2, ref, d1, d2 = c5_reference
    _check("cnn4_c64_32x32", spec, params, X1, X2, ref, d1, d2, *variant)


# ---- argument errors ------------------------------------------------------------------------
def test_variant_argument_errors_leave_output_untouched():
    import ctypes

    import torch
    from paper_2206_08720_amd import _lib
    from paper_2206_08720_amd.ntk import NTK
    from tests.gpu_helpers import to_dev
    spec = wl.fcn_spec("e", 8, [16], 3)
    params = to_dev(wl.make_params(spec, 1, "2/fan_in"))
    X1 = to_dev([wl.make_inputs(spec, 4, 2)])[0]
    X2 = to_dev([wl.make_inputs(spec, 3, 3)])[0]
    h = NTK(spec, 4, 4)
    try:
        with pytest.raises(_lib.NTKError) as ei:
            h.set_option(_lib.NTK_OPT_LOGIT, 3)          # O = 3
        assert ei.value.code == _lib.NTK_E_ARG
        with pytest.raises(_lib.NTKError):
            h.set_option(_lib.NTK_OPT_OUTPUT, 7)
        with pytest.raises(_lib.NTKError):
            h.set_option(_lib.NTK_OPT_BATCH, 2)
        h.set_variant("trace", "diagonal")
        bad = torch.full((4,), 5.0, device="cuda")
        ptrs = (ctypes.c_void_p * len(params))(*[p.data_ptr() for p in params])
        rc = h._lib.ntk_compute(h._h, ptrs, ctypes.c_void_p(X1.data_ptr()), 4,
                                ctypes.c_void_p(X2.data_ptr()), 3, ctypes.c_void_p(bad.data_ptr()))
        assert rc == _lib.NTK_E_ARG and "n1 == n2" in _lib.last_error(h._h)
        torch.cuda.synchronize()
        assert bool((bad == 5.0).all())
    finally:
        h.close()
