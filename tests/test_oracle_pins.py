"""Pins of the fp64 oracle against things other than itself (CPU only).

* torch's own layer routines and autograd Jacobian (an independent library);
* central finite differences of the network function;
* closed forms (one and two linear layers);
* hand-worked examples under tests/golden/;
* symmetry, positive semi-definiteness, ReLU homogeneity, the 1x1-image CNN
  reducing to an MLP, the trace identity, the Gram-spectrum identity, and the
  exactness of sample / output subsets.
"""
import json
import os

import numpy as np
import pytest

import oracle
import workloads as wl
from tests.torch_reference_net import torch_forward, torch_jacobian

torch = pytest.importorskip("torch")


def _tiny_specs():
    return [
        (wl.fcn_spec("fcn_relu_bias", 5, [7, 6], 3, act="relu", bias=True), "1/fan_in"),
        (wl.fcn_spec("fcn_erf", 4, [6, 5, 7], 3, act="erf"), "1/fan_in"),
        (wl.fcn_spec("fcn_linear", 4, [5], 2, act="none", bias=True), "1/fan_in"),
        (wl.cnn_spec("cnn_relu", (4, 3), 2, [3, 4], 3, act="relu"), "2/fan_in"),
        (wl.cnn_spec("cnn_erf_bias", (3, 3), 2, [3], 2, act="erf", bias=True), "2/fan_in"),
        # the further layer kinds: depthwise conv, per-channel scale, 2x2 average pool
        (wl.cnn_layers_spec("cnn_struct_erf", (4, 6), 2,
                            [("conv3x3", 3, "erf", True), ("dwconv3x3", "erf", True),
                             ("avgpool2",), ("scale", "erf", True), ("conv3x3", 2, "erf", False)],
                            3), "2/fan_in"),
        (wl.cnn_layers_spec("cnn_struct_relu", (4, 4), 3,
                            [("dwconv3x3", "relu", False), ("conv3x3", 4, "none", True),
                             ("scale", "relu", False), ("avgpool2",), ("dwconv3x3", "none", True)],
                            2), "2/fan_in"),
        # depthwise-separable blocks: depthwise 3x3 then pointwise 1x1
        (wl.cnn_layers_spec("cnn_separable_erf", (4, 6), 3,
                            [("conv1x1", 4, "erf", True), ("dwconv3x3", "erf", False),
                             ("conv1x1", 5, "erf", True), ("avgpool2",), ("conv1x1", 3, "none", False)],
                            2), "2/fan_in"),
    ]


@pytest.mark.parametrize("idx", range(8))
def test_forward_matches_torch_layers(idx):
    spec, wv = _tiny_specs()[idx]
    params = wl.make_params(spec, 11 + idx, wv, bias_var=0.3)
    X = wl.make_inputs(spec, 4, 21 + idx)
    ref = torch_forward(spec, [torch.tensor(p, dtype=torch.float64) for p in params],
                        torch.tensor(X, dtype=torch.float64)).numpy()
    got = oracle.forward(spec, params, X)
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("idx", range(8))
def test_jacobian_matches_torch_autograd(idx):
    spec, wv = _tiny_specs()[idx]
    params = wl.make_params(spec, 31 + idx, wv, bias_var=0.3)
    X = wl.make_inputs(spec, 3, 41 + idx)
    Jt = torch_jacobian(spec, params, X)
    Jo = oracle.jacobian(spec, params, X)
    assert Jo.shape == Jt.shape
    np.testing.assert_allclose(Jo, Jt, rtol=1e-12, atol=1e-12)


def _relu_margin_ok(spec, params, X, margin=1e-3):
    """True when no ReLU pre-activation is within `margin` of the kink (FD is then valid)."""
    from oracle.ntk_jc import _forward_record
    rec, _ = _forward_record(spec, params, X)
    for L, r in zip(spec["layers"], rec):
        if L.get("act") == "relu" and np.min(np.abs(r["z"])) < margin:
            return False
    return True


@pytest.mark.parametrize("idx", [0, 1, 3, 4, 5, 7])
def test_jacobian_central_finite_differences(idx):
    spec, wv = _tiny_specs()[idx]
    params = wl.make_params(spec, 51 + idx, wv, bias_var=0.3)
    X = wl.make_inputs(spec, 2, 61 + idx)
    if not _relu_margin_ok(spec, params, X):
        pytest.skip("a ReLU pre-activation sits too close to 0 for finite differences")
    J = oracle.jacobian(spec, params, X)                       # [N, O, P]
    flat = np.concatenate([p.astype(np.float64).ravel() for p in params])
    sizes = [p.size for p in params]
    shapes = [p.shape for p in params]

    def f(theta):
        ps, off = [], 0
        for s, sh in zip(sizes, shapes):
            ps.append(theta[off:off + s].reshape(sh))
            off += s
        return oracle.forward(spec, ps, X)

    eps = 1e-6
    Jfd = np.zeros_like(J)
    for p in range(flat.size):
        e = np.zeros_like(flat)
        e[p] = eps
        Jfd[:, :, p] = (f(flat + e) - f(flat - e)) / (2 * eps)
    np.testing.assert_allclose(J, Jfd, rtol=1e-6, atol=1e-8)


def test_closed_form_single_linear_layer():
    # f = W x (+ b): dtheta f_o = e_o (x) x^T (+ e_o), so Theta = (x1.x2 [+1]) I_O
    for bias in (False, True):
        spec = wl.fcn_spec("lin", 6, [], 4, bias=bias)
        params = wl.make_params(spec, 5, bias_var=1.0)
        X1 = wl.make_inputs(spec, 3, 6)
        X2 = wl.make_inputs(spec, 5, 7)
        th = oracle.ntk_jc(spec, params, X1, X2)
        gram = X1.astype(np.float64) @ X2.astype(np.float64).T + (1.0 if bias else 0.0)
        exp = gram[:, :, None, None] * np.eye(4)
        np.testing.assert_allclose(th, exp, rtol=1e-14, atol=1e-14)


def test_closed_form_two_linear_layers():
    # f = W2 W1 x: Theta = (x1.x2) W2 W2^T + (W1 x1 . W1 x2) I_O
    spec = wl.fcn_spec("lin2", 5, [7], 3, act="none")
    params = wl.make_params(spec, 8)
    W1, W2 = (p.astype(np.float64) for p in params)
    X1 = wl.make_inputs(spec, 4, 9).astype(np.float64)
    X2 = wl.make_inputs(spec, 2, 10).astype(np.float64)
    th = oracle.ntk_jc(spec, params, X1, X2)
    exp = (X1 @ X2.T)[:, :, None, None] * (W2 @ W2.T) \
        + ((X1 @ W1.T) @ (X2 @ W1.T).T)[:, :, None, None] * np.eye(3)
    np.testing.assert_allclose(th, exp, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("fname", ["fcn_hand_relu.json", "fcn_hand_relu_bias.json",
                                   "cnn_hand_1x2.json", "cnn_hand_struct.json"])
def test_hand_worked_golden(golden_dir, fname):
    d = json.load(open(os.path.join(golden_dir, fname)))
    spec = d["spec"]
    params = [np.array(p, dtype=np.float32) for p in d["params"]]
    X = np.array(d["X"], dtype=np.float32)
    th = oracle.ntk_jc(spec, params, X, X)
    np.testing.assert_allclose(th, np.array(d["theta"]), rtol=0, atol=1e-12)


@pytest.mark.parametrize("idx", [0, 1, 3, 5, 6, 7])
def test_symmetry_and_psd(idx):
    spec, wv = _tiny_specs()[idx]
    params = wl.make_params(spec, 71 + idx, wv, bias_var=0.3)
    X1 = wl.make_inputs(spec, 4, 81 + idx)
    X2 = wl.make_inputs(spec, 3, 91 + idx)
    a = oracle.ntk_jc(spec, params, X1, X2)
    b = oracle.ntk_jc(spec, params, X2, X1)
    # Theta(X1,X2)[n1,n2,o1,o2] = Theta(X2,X1)[n2,n1,o2,o1] (also catches o1<->o2 mix-ups)
    np.testing.assert_allclose(a, b.transpose(1, 0, 3, 2), rtol=1e-14, atol=1e-14)
    K = oracle.ntk_jc(spec, params, X1, X1)
    N, O = K.shape[0], K.shape[2]
    M = K.transpose(0, 2, 1, 3).reshape(N * O, N * O)
    np.testing.assert_allclose(M, M.T, rtol=1e-14, atol=1e-14)
    ev = np.linalg.eigvalsh(M)
    assert ev.min() >= -1e-12 * ev.max()


@pytest.mark.parametrize("idx", [0, 3])
def test_relu_homogeneity(idx):
    # bias-free ReLU nets: h_l(a x) = a h_l(x), masks unchanged => Theta(a X1, X2) = a Theta(X1, X2)
    spec, wv = _tiny_specs()[idx]
    spec = dict(spec, layers=[dict(L, bias=False) if "bias" in L else L for L in spec["layers"]])
    params = wl.make_params(spec, 101 + idx, wv)
    X1 = wl.make_inputs(spec, 3, 111 + idx)
    X2 = wl.make_inputs(spec, 2, 121 + idx)
    a = 2.5
    np.testing.assert_allclose(oracle.ntk_jc(spec, params, (a * X1.astype(np.float64)), X2),
                               a * oracle.ntk_jc(spec, params, X1, X2), rtol=1e-13, atol=1e-13)


def test_cnn_on_1x1_images_equals_mlp_of_centre_taps():
    spec = wl.cnn_spec("cnn1x1", (1, 1), 3, [5, 4], 2, act="erf")
    params = wl.make_params(spec, 131, "2/fan_in")
    X1 = wl.make_inputs(spec, 3, 132)
    X2 = wl.make_inputs(spec, 2, 133)
    mlp = wl.fcn_spec("centre", 3, [5, 4], 2, act="erf")
    mparams = [params[0][:, 1, 1, :], params[1][:, 1, 1, :], params[2]]
    a = oracle.ntk_jc(spec, params, X1, X2)
    b = oracle.ntk_jc(mlp, mparams, X1.reshape(3, 3), X2.reshape(2, 3))
    np.testing.assert_allclose(a, b, rtol=1e-13, atol=1e-14)


def test_trace_and_gram_spectrum():
    spec, wv = _tiny_specs()[3]
    params = wl.make_params(spec, 141, wv)
    X = wl.make_inputs(spec, 3, 142)
    J = oracle.jacobian(spec, params, X)          # [N, O, P]
    K = oracle.ntk_jc(spec, params, X, X)
    N, O, P = J.shape
    # sum_o Theta(x, x)[o, o] = ||J(x)||_F^2
    for n in range(N):
        np.testing.assert_allclose(np.trace(K[n, n]), np.sum(J[n] ** 2), rtol=1e-13)
    # eigenvalues of Theta(X, X) = the nonzero eigenvalues of J^T J (Appendix "NTK vs Hessian")
    Jm = J.reshape(N * O, P)
    ev_ntk = np.sort(np.linalg.eigvalsh(K.transpose(0, 2, 1, 3).reshape(N * O, N * O)))
    ev_jtj = np.sort(np.linalg.eigvalsh(Jm.T @ Jm))[-N * O:]
    np.testing.assert_allclose(ev_ntk, ev_jtj, rtol=1e-9, atol=1e-9 * ev_ntk.max())


def test_sample_and_output_subsets_are_exact_blocks():
    spec = wl.fcn_spec("sub", 6, [9, 8], 5, act="erf", bias=True)
    params = wl.make_params(spec, 151)
    X1 = wl.make_inputs(spec, 6, 152)
    X2 = wl.make_inputs(spec, 5, 153)
    full, n1, n2 = oracle.ntk_jc_with_norms(spec, params, X1, X2)
    r1, r2, o1, o2 = [0, 3, 5], [1, 4], [4, 0], [2, 3, 1]
    sub, s1, s2 = oracle.ntk_jc_with_norms(spec, params, X1[r1], X2[r2], o1, o2)
    np.testing.assert_allclose(sub, full[np.ix_(r1, r2, o1, o2)], rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(s1, n1[np.ix_(r1, o1)], rtol=1e-14)
    # the squared row norms are the diagonal of Theta(X, X)
    d = oracle.ntk_jc(spec, params, X1, X1)
    np.testing.assert_allclose(n1, np.einsum("nnoo->no", d), rtol=1e-13)


def test_block_chunking_does_not_change_the_result():
    spec = wl.cnn_spec("chunk", (3, 4), 2, [5, 3], 3, act="relu", bias=True)
    params = wl.make_params(spec, 161, "2/fan_in", bias_var=0.2)
    X1 = wl.make_inputs(spec, 3, 162)
    X2 = wl.make_inputs(spec, 2, 163)
    a = oracle.ntk_jc(spec, params, X1, X2)
    b = oracle.ntk_jc(spec, params, X1, X2, max_block_bytes=600)   # forces many column chunks
    np.testing.assert_allclose(a, b, rtol=1e-14, atol=1e-14)


# ---- float32 layer storage (the mode GPU parity uses) --------------------------------------
@pytest.mark.parametrize("fname", ["fcn_hand_relu.json", "fcn_hand_relu_bias.json",
                                   "cnn_hand_1x2.json", "cnn_hand_struct.json"])
def test_fp32_storage_reproduces_the_hand_worked_values(golden_dir, fname):
    # every intermediate value of these examples is exactly representable in float32
    d = json.load(open(os.path.join(golden_dir, fname)))
    params = [np.array(p, dtype=np.float32) for p in d["params"]]
    X = np.array(d["X"], dtype=np.float32)
    th = oracle.ntk_jc(d["spec"], params, X, X, layer_storage="fp32")
    np.testing.assert_allclose(th, np.array(d["theta"]), rtol=0, atol=1e-12)


@pytest.mark.parametrize("idx", [1, 4])
def test_fp32_storage_is_a_float32_perturbation_on_smooth_nets(idx):
    # erf nets: rounding the stored layer outputs to float32 moves Theta by ~1e-7 relative
    spec, wv = _tiny_specs()[idx]
    params = wl.make_params(spec, 171 + idx, wv, bias_var=0.3)
    X1 = wl.make_inputs(spec, 4, 181 + idx)
    X2 = wl.make_inputs(spec, 3, 191 + idx)
    a = oracle.ntk_jc(spec, params, X1, X2)
    b = oracle.ntk_jc(spec, params, X1, X2, layer_storage="fp32")
    assert not np.array_equal(a, b)
    assert np.max(np.abs(a - b)) <= 1e-6 * np.max(np.abs(a))


def test_fp32_storage_rounds_every_stored_layer_output():
    from oracle.ntk_jc import _forward_record
    spec, wv = _tiny_specs()[3]
    params = wl.make_params(spec, 201, wv)
    X = wl.make_inputs(spec, 3, 202)
    rec, _ = _forward_record(spec, params, X, layer_storage="fp32")
    for r in rec[1:]:
        h = r["h"]
        assert np.array_equal(h, h.astype(np.float32).astype(np.float64))
    with pytest.raises(ValueError):
        _forward_record(spec, params, X, layer_storage="fp16")


# ---- the further layer kinds: closed forms and reductions to pinned layers ------------------
def _readout_net(blocks, hw=(4, 6), c=3, O=3):
    return wl.cnn_layers_spec("closed", hw, c, blocks, O)


def test_closed_form_scale_with_bias():
    # f_o = sum_c Wd[o,c] (w[c] xbar[c] + b[c]) with xbar the pixel mean of x: by linearity
    # df_o/dw[c] = Wd[o,c] xbar[c], df_o/db[c] = Wd[o,c], df_o/dWd[o',c] = delta (w xbar + b)[c]
    spec = _readout_net([("scale", "none", True)])
    params = wl.make_params(spec, 211, bias_var=0.5)
    w, b, Wd = (p.astype(np.float64) for p in params)
    X1 = wl.make_inputs(spec, 3, 212).astype(np.float64)
    X2 = wl.make_inputs(spec, 2, 213).astype(np.float64)
    m1, m2 = X1.mean(axis=(1, 2)), X2.mean(axis=(1, 2))            # [N, C]
    g1, g2 = m1 * w + b, m2 * w + b
    exp = np.einsum("oc,qc,nc,mc->nmoq", Wd, Wd, m1, m2) + np.einsum("oc,qc->oq", Wd, Wd) \
        + (g1 @ g2.T)[:, :, None, None] * np.eye(3)
    np.testing.assert_allclose(oracle.ntk_jc(spec, params, X1, X2), exp, rtol=1e-13, atol=1e-13)


def test_closed_form_depthwise_with_bias():
    # f_o = sum_c Wd[o,c] (sum_t w[t,c] s_t[c] + b[c]), s_t[c] = mean over output pixels of the
    # input pixel at tap offset t (zero outside the image)
    spec = _readout_net([("dwconv3x3", "none", True)])
    params = wl.make_params(spec, 221, "2/fan_in", bias_var=0.5)
    w, b, Wd = (p.astype(np.float64) for p in params)
    H, W = 4, 6

    def shifted_means(X):
        N, _, _, C = X.shape
        s = np.zeros((N, 3, 3, C))
        for kh in range(3):
            for kw in range(3):
                for y in range(H):
                    for x in range(W):
                        yy, xx = y + kh - 1, x + kw - 1
                        if 0 <= yy < H and 0 <= xx < W:
                            s[:, kh, kw] += X[:, yy, xx]
        return s / (H * W)

    X1 = wl.make_inputs(spec, 3, 222).astype(np.float64)
    X2 = wl.make_inputs(spec, 2, 223).astype(np.float64)
    s1, s2 = shifted_means(X1), shifted_means(X2)                  # [N, 3, 3, C]
    g1 = np.einsum("nijc,ijc->nc", s1, w) + b
    g2 = np.einsum("nijc,ijc->nc", s2, w) + b
    exp = np.einsum("oc,qc,nijc,mijc->nmoq", Wd, Wd, s1, s2) + np.einsum("oc,qc->oq", Wd, Wd) \
        + (g1 @ g2.T)[:, :, None, None] * np.eye(3)
    np.testing.assert_allclose(oracle.ntk_jc(spec, params, X1, X2), exp, rtol=1e-13, atol=1e-13)


def test_closed_form_conv_bias_summand():
    # a conv bias is broadcast over the pixels (output block-tiled): with no activation its
    # Jacobian rows are Wd[o, :] for every input, so it adds Wd Wd^T to every O x O block
    blocks_b = [("conv3x3", 4, "none", True)]
    blocks_n = [("conv3x3", 4, "none", False)]
    sb, sn = _readout_net(blocks_b), _readout_net(blocks_n)
    params = wl.make_params(sb, 231, "2/fan_in", bias_var=0.5)
    pn = [params[0], params[2]]
    X1 = wl.make_inputs(sb, 3, 232)
    X2 = wl.make_inputs(sb, 2, 233)
    Wd = params[2].astype(np.float64)
    # the readout summand changes with the bias (g moves by b); compare the parameter blocks
    a = oracle.ntk_jc(sb, params, X1, X2)
    Jb = oracle.jacobian(sb, params, X1)
    np.testing.assert_allclose(Jb[:, :, 4 * 27:4 * 27 + 4], np.broadcast_to(Wd, (3, 3, 4)),
                               rtol=1e-14, atol=1e-15)
    Jn = oracle.jacobian(sn, pn, X1)
    np.testing.assert_allclose(Jb[:, :, :4 * 27], Jn[:, :, :4 * 27], rtol=1e-14, atol=1e-15)
    assert a.shape == (3, 2, 3, 3)


def test_avgpool_before_gap_is_invisible():
    # the mean of the 2x2-window means is the mean over all pixels
    with_pool = _readout_net([("conv3x3", 4, "erf", True), ("avgpool2",)])
    without = _readout_net([("conv3x3", 4, "erf", True)])
    params = wl.make_params(with_pool, 241, "2/fan_in", bias_var=0.3)
    X1 = wl.make_inputs(with_pool, 3, 242)
    X2 = wl.make_inputs(with_pool, 2, 243)
    np.testing.assert_allclose(oracle.ntk_jc(with_pool, params, X1, X2),
                               oracle.ntk_jc(without, params, X1, X2), rtol=1e-13, atol=1e-14)


def test_avgpool_between_convs_matches_strided_means():
    # the pooled image is the mean of each 2x2 block; pin the pooling layer's forward map
    # through a net whose first layer is an identity scale (w = 1, b = 0, no activation)
    spec = _readout_net([("scale", "none", False), ("avgpool2",), ("conv3x3", 2, "none", False)],
                        hw=(4, 6), c=2, O=2)
    params = wl.make_params(spec, 251, "2/fan_in")
    params[0] = np.ones_like(params[0])
    X = wl.make_inputs(spec, 2, 252).astype(np.float64)
    pooled = np.zeros((2, 2, 3, 2))
    for y in range(2):
        for x in range(3):
            pooled[:, y, x] = X[:, 2 * y:2 * y + 2, 2 * x:2 * x + 2].sum(axis=(1, 2)) / 4
    ref = wl.cnn_spec("ref", (2, 3), 2, [2], 2, act="none")
    np.testing.assert_allclose(oracle.forward(spec, params, X),
                               oracle.forward(ref, params[1:], pooled), rtol=1e-13, atol=1e-14)


def test_depthwise_with_one_channel_is_a_3x3_conv():
    dw = _readout_net([("dwconv3x3", "erf", True)], c=1, O=2)
    cv = _readout_net([("conv3x3", 1, "erf", True)], c=1, O=2)
    params = wl.make_params(dw, 261, "2/fan_in", bias_var=0.3)
    cparams = [params[0].reshape(1, 3, 3, 1), params[1], params[2]]
    X1 = wl.make_inputs(dw, 3, 262)
    X2 = wl.make_inputs(dw, 2, 263)
    np.testing.assert_allclose(oracle.ntk_jc(dw, params, X1, X2),
                               oracle.ntk_jc(cv, cparams, X1, X2), rtol=1e-13, atol=1e-14)


def test_pointwise_layers_on_1x1_images_are_the_mlp():
    # on 1x1 images a pointwise convolution is a dense layer and the pool over one pixel is the
    # identity, so the CNN's NTK is the MLP's
    spec = wl.cnn_layers_spec("pw1x1", (1, 1), 5, [("conv1x1", 7, "erf", True), ("conv1x1", 6, "relu", True)], 3)
    params = wl.make_params(spec, 271, "2/fan_in", bias_var=0.3)
    X1 = wl.make_inputs(spec, 3, 272)
    X2 = wl.make_inputs(spec, 4, 273)
    mlp = {"name": "mlp", "input_shape": (5,),
           "layers": [{"kind": "dense", "in": 5, "out": 7, "act": "erf", "bias": True},
                      {"kind": "dense", "in": 7, "out": 6, "act": "relu", "bias": True},
                      {"kind": "dense", "in": 6, "out": 3, "act": "none", "bias": False}]}
    a = oracle.ntk_jc(spec, params, X1, X2)
    b = oracle.ntk_jc(mlp, params, X1.reshape(3, 5), X2.reshape(4, 5))
    np.testing.assert_allclose(a, b, rtol=1e-13, atol=1e-14)


def test_pointwise_is_the_centre_tap_of_a_3x3_conv():
    # a 3x3 convolution whose only nonzero tap is the centre acts as a pointwise one
    pw = wl.cnn_layers_spec("pw", (3, 4), 3, [("conv1x1", 5, "erf", True)], 2)
    cv = wl.cnn_layers_spec("cv", (3, 4), 3, [("conv3x3", 5, "erf", True)], 2)
    params = wl.make_params(pw, 281, "2/fan_in", bias_var=0.3)
    K = np.zeros((5, 3, 3, 3), dtype=np.float32)
    K[:, 1, 1, :] = params[0]
    X = wl.make_inputs(pw, 3, 282)
    np.testing.assert_allclose(oracle.forward(pw, params, X), oracle.forward(cv, [K] + params[1:], X),
                               rtol=1e-13, atol=1e-14)
    # the Jacobian blocks: the pointwise block is the 3x3 block's centre-tap columns
    Jp = oracle.jacobian(pw, params, X)
    Jc = oracle.jacobian(cv, [K] + params[1:], X)
    centre = np.zeros((5, 3, 3, 3), dtype=bool)
    centre[:, 1, 1, :] = True
    np.testing.assert_allclose(Jp[:, :, :15], Jc[:, :, :135][:, :, centre.ravel()], rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(Jp[:, :, 15:], Jc[:, :, 135:], rtol=1e-13, atol=1e-14)
