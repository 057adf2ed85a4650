"""Pins of the oracle's output- and batch-axis variants (CPU, fp64).

`oracle.ntk_jc_variant` contracts only the Jacobian rows a variant keeps; here it is checked
against slices and sums of the full Theta of `oracle.ntk_jc` (a different contraction of the
same definition), against closed forms, and against the trace identity."""
import numpy as np
import pytest

import oracle
import workloads as wl

NETS = [
    (wl.fcn_spec("v_relu_bias", 5, [7, 6], 3, act="relu", bias=True), "1/fan_in"),
    (wl.fcn_spec("v_erf", 4, [6, 5], 4, act="erf"), "1/fan_in"),
    (wl.cnn_spec("v_cnn", (3, 4), 2, [3, 4], 3), "2/fan_in"),
]
COMBOS = [(o, b) for o in ("full", "trace", "logit") for b in ("full", "diagonal")]


def _reference(full, output, batch, logit):
    """The variant read off the full Theta [N1, N2, O, O]."""
    if batch == "diagonal":
        n = np.arange(full.shape[0])
        full = full[n, n]                                   # [N, O, O]
    if output == "trace":
        return np.trace(full, axis1=-2, axis2=-1)
    if output == "logit":
        return full[..., logit, logit]
    return full


@pytest.mark.parametrize("combo", COMBOS, ids=[f"{o}-{b}" for o, b in COMBOS])
@pytest.mark.parametrize("net", NETS, ids=[n[0]["name"] for n in NETS])
def test_variant_equals_the_part_of_full_theta(net, combo):
    spec, wv = net
    output, batch = combo
    params = wl.make_params(spec, 901, wv, bias_var=0.3)
    X1 = wl.make_inputs(spec, 5, 902)
    X2 = wl.make_inputs(spec, 5, 903)
    O = spec["layers"][-1]["out"]
    full = oracle.ntk_jc(spec, params, X1, X2)
    for logit in (range(O) if output == "logit" else [0]):
        got, scale = oracle.ntk_jc_variant(spec, params, X1, X2, output, batch, logit)
        ref = _reference(full, output, batch, logit)
        assert got.shape == ref.shape == scale.shape
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12 * np.abs(full).max())
        assert np.all(np.abs(got) <= scale * (1 + 1e-12) + 1e-300)


@pytest.mark.parametrize("bias", [False, True])
def test_variants_of_one_linear_layer_closed_form(bias):
    # Theta = (x1 . x2 [+1]) I_O, so the trace is O (x1 . x2 [+1]) and each logit x1 . x2 [+1]
    spec = wl.fcn_spec("lin", 6, [], 4, bias=bias)
    params = wl.make_params(spec, 5, bias_var=1.0)
    X1 = wl.make_inputs(spec, 3, 6)
    X2 = wl.make_inputs(spec, 3, 7)
    k = X1.astype(np.float64) @ X2.astype(np.float64).T + (1.0 if bias else 0.0)
    tr, _ = oracle.ntk_jc_variant(spec, params, X1, X2, "trace")
    np.testing.assert_allclose(tr, 4 * k, rtol=1e-13)
    lg, _ = oracle.ntk_jc_variant(spec, params, X1, X2, "logit", logit=3)
    np.testing.assert_allclose(lg, k, rtol=1e-13)
    dg, _ = oracle.ntk_jc_variant(spec, params, X1, X2, "full", "diagonal")
    np.testing.assert_allclose(dg, np.diag(k)[:, None, None] * np.eye(4), rtol=1e-13, atol=1e-15)
    td, _ = oracle.ntk_jc_variant(spec, params, X1, X2, "trace", "diagonal")
    np.testing.assert_allclose(td, 4 * np.diag(k), rtol=1e-13)


def test_traced_diagonal_is_the_squared_jacobian_norm():
    # sum_o Theta(x, x)[o, o] = ||df(x)/dtheta||_F^2
    spec = wl.fcn_spec("tr", 5, [8, 6], 3, act="erf", bias=True)
    params = wl.make_params(spec, 17, bias_var=0.2)
    X = wl.make_inputs(spec, 4, 18)
    J = oracle.jacobian(spec, params, X)                     # [N, O, P]
    td, _ = oracle.ntk_jc_variant(spec, params, X, X, "trace", "diagonal")
    np.testing.assert_allclose(td, (J ** 2).sum(axis=(1, 2)), rtol=1e-12)


def test_variant_arguments_are_checked():
    spec = wl.fcn_spec("a", 3, [4], 2)
    params = wl.make_params(spec, 1)
    X = wl.make_inputs(spec, 3, 2)
    with pytest.raises(ValueError):
        oracle.ntk_jc_variant(spec, params, X, X[:2], batch="diagonal")
    with pytest.raises(ValueError):
        oracle.ntk_jc_variant(spec, params, X, X, output="diag")
