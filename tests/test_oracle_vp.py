"""Pins of the oracle's NTK-vector product (CPU, fp64): against the full Theta contracted
with v, a closed form, linearity, and the identity columns giving Theta back."""
import numpy as np
import pytest

import oracle
import workloads as wl

NETS = [
    (wl.fcn_spec("vp_relu_bias", 5, [7, 6], 3, act="relu", bias=True), "1/fan_in"),
    (wl.fcn_spec("vp_erf", 4, [6, 5], 4, act="erf"), "1/fan_in"),
    (wl.cnn_spec("vp_cnn", (3, 4), 2, [3, 4], 3), "2/fan_in"),
]


@pytest.mark.parametrize("net", NETS, ids=[n[0]["name"] for n in NETS])
def test_vp_equals_full_theta_times_v(net):
    spec, wv = net
    params = wl.make_params(spec, 41, wv, bias_var=0.3)
    X1 = wl.make_inputs(spec, 4, 42)
    X2 = wl.make_inputs(spec, 6, 43)
    O = spec["layers"][-1]["out"]
    v = np.random.default_rng(44).standard_normal((6, O))
    got, scale = oracle.ntk_vp(spec, params, X1, X2, v)
    full = oracle.ntk_jc(spec, params, X1, X2)
    ref = np.einsum("abij,bj->ai", full, v)
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-12 * np.abs(ref).max())
    assert np.all(np.abs(got) <= scale * (1 + 1e-12))


def test_vp_with_identity_columns_is_theta():
    spec = wl.fcn_spec("vpi", 4, [5], 3, act="erf", bias=True)
    params = wl.make_params(spec, 7, bias_var=0.2)
    X1 = wl.make_inputs(spec, 2, 8)
    X2 = wl.make_inputs(spec, 3, 9)
    full = oracle.ntk_jc(spec, params, X1, X2)
    for n2 in range(3):
        for o2 in range(3):
            v = np.zeros((3, 3))
            v[n2, o2] = 1.0
            got, _ = oracle.ntk_vp(spec, params, X1, X2, v)
            np.testing.assert_allclose(got, full[:, n2, :, o2], rtol=1e-12, atol=1e-14)


def test_vp_of_one_linear_layer_closed_form():
    # Theta = (x1 . x2 + 1) I_O  =>  (Theta v)[n1] = sum_n2 (x1 . x2 + 1) v[n2]
    spec = wl.fcn_spec("lin", 6, [], 4, bias=True)
    params = wl.make_params(spec, 5, bias_var=1.0)
    X1 = wl.make_inputs(spec, 3, 6)
    X2 = wl.make_inputs(spec, 5, 7)
    v = np.random.default_rng(8).standard_normal((5, 4))
    k = X1.astype(np.float64) @ X2.astype(np.float64).T + 1.0
    got, _ = oracle.ntk_vp(spec, params, X1, X2, v)
    np.testing.assert_allclose(got, k @ v, rtol=1e-13)


def test_vp_is_linear_in_v():
    spec = wl.fcn_spec("lin2", 5, [8], 3, act="relu")
    params = wl.make_params(spec, 11)
    X1 = wl.make_inputs(spec, 3, 12)
    X2 = wl.make_inputs(spec, 4, 13)
    rng = np.random.default_rng(14)
    a, b = rng.standard_normal((4, 3)), rng.standard_normal((4, 3))
    fa, _ = oracle.ntk_vp(spec, params, X1, X2, a)
    fb, _ = oracle.ntk_vp(spec, params, X1, X2, b)
    fab, _ = oracle.ntk_vp(spec, params, X1, X2, 2.0 * a - 3.0 * b)
    np.testing.assert_allclose(fab, 2.0 * fa - 3.0 * fb, rtol=1e-12, atol=1e-13)
