"""Pin the secondary fp64 structured reference to the Jacobian-contraction oracle (CPU only).

The structured reference (Section 4.1's per-layer formula, in float64) is used
for full-size coverage of the two large fully-connected workloads, where the
plain Jacobian contraction would take hours.  Here it must agree with the
definition on every small workload in full and on sample/output subsets of the
large ones (a sub-batch's NTK is exactly a sub-block).
"""
import numpy as np
import pytest

import oracle
import workloads as wl


def _close(a, b, tol=1e-11):
    scale = max(1.0, float(np.max(np.abs(b))))
    assert np.max(np.abs(a - b)) <= tol * scale, np.max(np.abs(a - b)) / scale


def test_structured_equals_jc_on_tiny_relu_mlp():
    spec, params, X1, X2 = wl.make_workload("tiny_relu_mlp")
    _close(oracle.ntk_structured_fp64(spec, params, X1, X2), oracle.ntk_jc(spec, params, X1, X2))


def test_structured_equals_jc_on_relu_mlp_d4_w512():
    spec, params, X1, X2 = wl.make_workload("relu_mlp_d4_w512", n1=24)
    _close(oracle.ntk_structured_fp64(spec, params, X1, X2), oracle.ntk_jc(spec, params, X1, X2))


@pytest.mark.parametrize("name,rows,outs", [
    ("relu_mlp_d8_w2048", [0, 511], [0, 9]),
    ("erf_mlp_d3_w4096", [0, 127], [0, 57, 99]),
])
def test_structured_equals_jc_on_subsets_of_large_workloads(name, rows, outs):
    spec, params, X1, X2 = wl.make_workload(name)
    a = oracle.ntk_structured_fp64(spec, params, X1[rows], X2[rows])
    b = oracle.ntk_jc(spec, params, X1[rows], X2[rows], outs, outs)
    _close(a[:, :, outs][:, :, :, outs], b)


@pytest.mark.parametrize("act,bias", [("relu", True), ("erf", False), ("none", True)])
def test_structured_equals_jc_on_random_ragged_mlps(act, bias):
    spec = wl.fcn_spec("ragged", 13, [37, 19, 41], 7, act=act, bias=bias)
    params = wl.make_params(spec, 7, bias_var=0.5)
    X1 = wl.make_inputs(spec, 9, 8)
    X2 = wl.make_inputs(spec, 5, 9)
    _close(oracle.ntk_structured_fp64(spec, params, X1, X2), oracle.ntk_jc(spec, params, X1, X2))


def test_structured_diag_equals_jc_row_norms():
    spec = wl.fcn_spec("ragged", 13, [37, 19], 7, act="erf", bias=True)
    params = wl.make_params(spec, 17, bias_var=0.5)
    X = wl.make_inputs(spec, 6, 18)
    _, sq, _ = oracle.ntk_jc_with_norms(spec, params, X, X[:1])
    _close(oracle.ntk_structured_diag_fp64(spec, params, X), sq)


@pytest.mark.parametrize("name,rows,outs", [
    ("tiny_relu_mlp", list(range(8)), None),
    ("relu_mlp_d8_w2048", [3, 400], [1, 8]),
])
def test_structured_equals_jc_with_fp32_layer_storage(name, rows, outs):
    spec, params, X1, X2 = wl.make_workload(name)
    a = oracle.ntk_structured_fp64(spec, params, X1[rows], X2[rows], layer_storage="fp32")
    b = oracle.ntk_jc(spec, params, X1[rows], X2[rows], outs, outs, layer_storage="fp32")
    if outs is not None:
        a = a[:, :, outs][:, :, :, outs]
    _close(a, b)
    d = oracle.ntk_structured_diag_fp64(spec, params, X1[rows], layer_storage="fp32")
    _, sq, _ = oracle.ntk_jc_with_norms(spec, params, X1[rows], X2[rows[:1]], outs, outs,
                                        layer_storage="fp32")
    _close(d if outs is None else d[:, outs], sq)
