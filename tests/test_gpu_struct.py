"""GPU parity of the further structure rules against the fp64 oracle (needs an MI355X).

Convolutional models with depthwise 3x3 convolutions (block-diagonal weight-space Jacobian),
per-channel scale layers (block-diagonal over channels, output block-tiled over pixels),
biases broadcast over the pixels (output block-tiled) and 2x2 average pools.  References are
the Jacobian-contraction oracle with float32 layer storage (see tests/test_gpu_fcn.py).
"""
import numpy as np
import pytest

import oracle
import workloads as wl
from tests.gpu_helpers import (TOL, errors, gpu_ntk, report, scaled_errors, variant_of,
                               variant_scale)

pytestmark = pytest.mark.gpu
S = "fp32"


def _spec(label, hw, c, blocks, O):
    return wl.cnn_layers_spec(label, hw, c, blocks, O)


def _data(spec, n1, n2, seed):
    params = wl.make_params(spec, seed, "2/fan_in", bias_var=0.1)
    X1 = wl.make_inputs(spec, n1, seed + 1)
    X2 = wl.make_inputs(spec, n2, seed + 2)
    return params, X1, X2


def _vs_jc(name, spec, params, X1, X2, symmetric=True, options=None):
    print(f"[parity] {name}: start", flush=True)
    got = gpu_ntk(spec, params, X1, X2, symmetric=symmetric, options=options)
    ref, d1, d2 = oracle.ntk_jc_with_norms(spec, params, X1, X2, layer_storage=S)
    cs, nw = errors(got, ref, d1, d2)
    report(name, cs, nw)
    assert got.shape == ref.shape
    assert cs <= TOL and nw <= TOL
    return got


@pytest.mark.timeout(600)
def test_cnn_struct_c64_32x32_full():
    spec, params, X1, X2 = wl.make_workload("cnn_struct_c64_32x32")
    _vs_jc("cnn_struct_c64_32x32", spec, params, X1, X2)


CASES = [
    # label, spec, n1, n2
    ("depthwise, 3 channels (scalar lanes), ragged 5x7, bias, erf",
     _spec("s1", (5, 7), 3, [("dwconv3x3", "erf", True)], 4), 5, 6),
    ("scale with bias then conv, 8 channels",
     _spec("s2", (4, 4), 8, [("scale", "relu", True), ("conv3x3", 8, "relu", False)], 3), 7, 4),
    ("pool first, then conv with bias",
     _spec("s3", (6, 4), 3, [("avgpool2",), ("conv3x3", 16, "relu", True)], 10), 4, 9),
    ("conv, pool, depthwise, pool, scale: 8x8 down to 2x2",
     _spec("s4", (8, 8), 3, [("conv3x3", 16, "relu", True), ("avgpool2",), ("dwconv3x3", "relu", True),
                             ("avgpool2",), ("scale", "erf", True)], 5), 6, 6),
    ("last spatial layer a pool (seed without act')",
     _spec("s5", (4, 6), 4, [("conv3x3", 8, "erf", True), ("dwconv3x3", "none", False), ("avgpool2",)], 3),
     3, 5),
    ("O = 1, one image each",
     _spec("s6", (6, 6), 4, [("dwconv3x3", "relu", True), ("conv3x3", 8, "relu", True)], 1), 1, 1),
    ("1x1 images, depthwise sees only its centre tap",
     _spec("s7", (1, 1), 8, [("dwconv3x3", "erf", True), ("scale", "relu", False)], 3), 4, 3),
    ("6 channels (scalar lanes) through pool and scale",
     _spec("s8", (4, 8), 6, [("scale", "erf", False), ("avgpool2",), ("dwconv3x3", "relu", True),
                             ("conv3x3", 5, "erf", True)], 4), 5, 4),
    ("1028 channels: two channel passes of the pixel sums",
     _spec("s9", (2, 2), 1028, [("scale", "relu", True), ("dwconv3x3", "erf", True)], 2), 3, 2),
    ("258 channels (scalar lanes): two channel passes",
     _spec("s10", (2, 2), 258, [("dwconv3x3", "relu", True), ("scale", "none", True)], 2), 2, 3),
    ("32 channels (direct-to-LDS conv loads) with biases, ragged rows",
     _spec("s11", (6, 6), 3, [("conv3x3", 32, "relu", True), ("dwconv3x3", "relu", True),
                              ("avgpool2",), ("conv3x3", 32, "relu", True)], 10), 23, 17),
    # pointwise (1x1) convolutions: depthwise-separable blocks
    ("separable block, 32 channels (direct-to-LDS pointwise product)",
     _spec("s12", (8, 8), 3, [("conv3x3", 32, "relu", True), ("dwconv3x3", "relu", True),
                              ("conv1x1", 64, "relu", True), ("avgpool2",), ("dwconv3x3", "erf", False),
                              ("conv1x1", 32, "erf", True)], 10), 9, 7),
    ("pointwise first, 3 and 6 channels (register-staged loaders)",
     _spec("s13", (5, 7), 3, [("conv1x1", 6, "erf", True), ("dwconv3x3", "relu", False),
                              ("conv1x1", 5, "relu", True)], 4), 5, 6),
    ("pointwise on 1x1 images (an MLP with biases)",
     _spec("s14", (1, 1), 12, [("conv1x1", 40, "erf", True), ("scale", "relu", True),
                               ("conv1x1", 24, "relu", True)], 5), 13, 11),
    ("pointwise first on 3 channels padded to 4, 16x16 images",
     _spec("s16", (16, 16), 3, [("conv1x1", 8, "relu", True), ("conv3x3", 8, "erf", False)], 3), 3, 2),
    ("pointwise after a pool, last layer without activation",
     _spec("s15", (4, 4), 8, [("dwconv3x3", "relu", True), ("avgpool2",), ("conv1x1", 16, "none", True)], 3),
     4, 3),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_struct_edge_shapes(case):
    label, spec, n1, n2 = case
    params, X1, X2 = _data(spec, n1, n2, 500 + n1 + 7 * n2)
    _vs_jc(label, spec, params, X1, X2)


# conv orders: the 3x3 convolutions of a model with pools (per-layer image sizes) contracted
# inside-out, outside-in and by the cost model; the Jacobian-contraction method
ORDER_SPEC = _spec("ord", (8, 8), 4, [("conv3x3", 16, "relu", True), ("avgpool2",),
                                     ("dwconv3x3", "relu", True), ("conv3x3", 8, "erf", True)], 6)


@pytest.mark.parametrize("order", ["auto", "outside_in", "inside_out", "jacobian"])
def test_struct_conv_orders_and_method(order):
    from paper_2206_08720_amd import _lib
    params, X1, X2 = _data(ORDER_SPEC, 9, 7, 611)
    opts = {"auto": {_lib.NTK_OPT_CONV_ORDER: _lib.NTK_CONV_ORDER_AUTO},
            "outside_in": {_lib.NTK_OPT_CONV_ORDER: _lib.NTK_CONV_ORDER_OUTSIDE_IN},
            "inside_out": {_lib.NTK_OPT_CONV_ORDER: _lib.NTK_CONV_ORDER_INSIDE_OUT},
            "jacobian": {_lib.NTK_OPT_METHOD: _lib.NTK_METHOD_JACOBIAN}}[order]
    _vs_jc(f"struct model, {order}", ORDER_SPEC, params, X1, X2, options=opts)


SEP_SPEC = _spec("sep", (8, 8), 4, [("conv1x1", 16, "relu", True), ("dwconv3x3", "relu", True),
                                   ("avgpool2",), ("conv1x1", 12, "erf", True), ("conv3x3", 8, "relu", False)], 5)


@pytest.mark.parametrize("mode", ["jacobian", "inside_out", "outside_in", "trace", "logit-diagonal", "aliased"])
def test_pointwise_model_modes(mode):
    from paper_2206_08720_amd import _lib
    params, X1, X2 = _data(SEP_SPEC, 7, 6, 661)
    if mode in ("jacobian", "inside_out", "outside_in"):
        opts = {"jacobian": {_lib.NTK_OPT_METHOD: _lib.NTK_METHOD_JACOBIAN},
                "inside_out": {_lib.NTK_OPT_CONV_ORDER: _lib.NTK_CONV_ORDER_INSIDE_OUT},
                "outside_in": {_lib.NTK_OPT_CONV_ORDER: _lib.NTK_CONV_ORDER_OUTSIDE_IN}}[mode]
        _vs_jc(f"separable, {mode}", SEP_SPEC, params, X1, X2, options=opts)
        return
    if mode == "aliased":
        got = _vs_jc("separable, aliased", SEP_SPEC, params, X1, X1)
        N, O = got.shape[0], got.shape[2]
        M = got.transpose(0, 2, 1, 3).reshape(N * O, N * O)
        np.testing.assert_allclose(M, M.T, rtol=0, atol=1e-5 * np.abs(M).max())
        return
    output, batch = ("trace", "full") if mode == "trace" else ("logit", "diagonal")
    X2 = X2 if batch == "full" else wl.make_inputs(SEP_SPEC, 7, 662)
    full, d1, d2 = oracle.ntk_jc_with_norms(SEP_SPEC, params, X1, X2, layer_storage=S)
    got = gpu_ntk(SEP_SPEC, params, X1, X2, variant=(output, batch, 3))
    ref = variant_of(full, output, batch, 3)
    scale = variant_scale(d1, d2, output, batch, 3)
    assert got.shape == ref.shape
    cs, nw = scaled_errors(got, ref, scale)
    report(f"separable {output}/{batch}", cs, nw)
    assert cs <= TOL and nw <= TOL


@pytest.mark.parametrize("symmetric", [True, False])
def test_struct_aliased_inputs(symmetric):
    params, X, _ = _data(ORDER_SPEC, 11, 1, 621)
    got = _vs_jc(f"struct aliased sym={symmetric}", ORDER_SPEC, params, X, X, symmetric=symmetric)
    N, O = got.shape[0], got.shape[2]
    M = got.transpose(0, 2, 1, 3).reshape(N * O, N * O)
    np.testing.assert_allclose(M, M.T, rtol=0, atol=1e-5 * np.abs(M).max())


VARIANTS = [("trace", "full"), ("logit", "full"), ("full", "diagonal"), ("trace", "diagonal"),
            ("logit", "diagonal")]


@pytest.mark.parametrize("order", ["outside_in", "inside_out"])
@pytest.mark.parametrize("variant", VARIANTS, ids=[f"{o}-{b}" for o, b in VARIANTS])
def test_struct_variants(variant, order):
    from paper_2206_08720_amd import _lib
    output, batch = variant
    params, X1, X2 = _data(ORDER_SPEC, 8, 8, 631)
    full, d1, d2 = oracle.ntk_jc_with_norms(ORDER_SPEC, params, X1, X2, layer_storage=S)
    O = ORDER_SPEC["layers"][-1]["out"]
    logit = O - 2 if output == "logit" else 0
    opt = {_lib.NTK_OPT_CONV_ORDER: _lib.NTK_CONV_ORDER_OUTSIDE_IN if order == "outside_in"
           else _lib.NTK_CONV_ORDER_INSIDE_OUT}
    got = gpu_ntk(ORDER_SPEC, params, X1, X2, options=opt, variant=(output, batch, logit))
    ref = variant_of(full, output, batch, logit)
    scale = variant_scale(d1, d2, output, batch, logit)
    assert got.shape == ref.shape
    cs, nw = scaled_errors(got, ref, scale)
    report(f"struct {output}/{batch} {order}", cs, nw)
    assert cs <= TOL and nw <= TOL


def test_struct_graph_replays_and_determinism():
    import torch
    from paper_2206_08720_amd import _lib
    from paper_2206_08720_amd.ntk import NTK
    from tests.gpu_helpers import to_dev
    params, X1, X2 = _data(ORDER_SPEC, 10, 6, 641)
    ps, (x1, x2) = to_dev(params), to_dev([X1, X2])
    h = NTK(ORDER_SPEC, 10, 6)
    try:
        eager = h.compute(ps, x1, x2).clone()
        again = h.compute(ps, x1, x2).clone()
        torch.cuda.synchronize()
        assert torch.equal(eager, again)
        h.set_option(_lib.NTK_OPT_GRAPH, 1)
        for _ in range(3):
            out = h.compute(ps, x1, x2)
            torch.cuda.synchronize()
            assert torch.equal(out, eager)
    finally:
        h.close()


@pytest.mark.parametrize("symmetric", [True, False])
def test_hand_worked_struct_golden_on_gpu(golden_dir, symmetric):
    import json
    import os
    d = json.load(open(os.path.join(golden_dir, "cnn_hand_struct.json")))
    params = [np.array(p, dtype=np.float32) for p in d["params"]]
    X = np.array(d["X"], dtype=np.float32)
    got = gpu_ntk(d["spec"], params, X, X, symmetric=symmetric)
    np.testing.assert_allclose(got, np.array(d["theta"]), rtol=1e-6, atol=1e-5)


LARGE_CASES = [
    ("128x128 images, 16384-pixel planes",
     _spec("l1", (128, 128), 4, [("conv3x3", 8, "relu", True), ("dwconv3x3", "erf", True), ("avgpool2",),
                                 ("conv1x1", 4, "relu", True), ("scale", "erf", True)], 3), 2, 3),
    ("2048 channels: 32 channel groups of 64 in the depthwise columns, wide pointwise columns",
     _spec("l2", (2, 2), 2048, [("dwconv3x3", "relu", True), ("scale", "erf", True), ("conv1x1", 8, "relu", True)], 3),
     3, 2),
]


@pytest.mark.parametrize("case", LARGE_CASES, ids=[c[0] for c in LARGE_CASES])
def test_struct_large_sizes(case):
    label, spec, n1, n2 = case
    params, X1, X2 = _data(spec, n1, n2, 700 + n1 * 5 + n2)
    _vs_jc(label, spec, params, X1, X2)
