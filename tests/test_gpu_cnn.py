"""GPU parity of the convolutional path against the fp64 oracle (needs an MI355X).

The references are the Jacobian-contraction oracle with float32 layer storage
(see tests/test_gpu_fcn.py); the 4-layer 64-channel CNN on 32x32x3 inputs is
compared in full.
"""
import json
import os

import numpy as np
import pytest

import oracle
import workloads as wl
from tests.gpu_helpers import TOL, errors, gpu_ntk, report

pytestmark = pytest.mark.gpu
S = "fp32"


def _vs_jc(name, spec, params, X1, X2, symmetric=True):
    got = gpu_ntk(spec, params, X1, X2, symmetric=symmetric)
    print(f"[parity] {name}: GPU done", flush=True)
    ref, d1, d2 = oracle.ntk_jc_with_norms(spec, params, X1, X2, layer_storage=S)
    cs, nw = errors(got, ref, d1, d2)
    report(name, cs, nw)
    assert got.shape == ref.shape
    assert cs <= TOL and nw <= TOL
    return got


@pytest.mark.parametrize("symmetric", [True, False])
def test_hand_worked_cnn_golden_on_gpu(golden_dir, symmetric):
    d = json.load(open(os.path.join(golden_dir, "cnn_hand_1x2.json")))
    params = [np.array(p, dtype=np.float32) for p in d["params"]]
    X = np.array(d["X"], dtype=np.float32)
    got = gpu_ntk(d["spec"], params, X, X, symmetric=symmetric)
    np.testing.assert_allclose(got, np.array(d["theta"]), rtol=1e-6, atol=1e-5)


def test_cnn4_c64_32x32_full():
    spec, params, X1, X2 = wl.make_workload("cnn4_c64_32x32")
    _vs_jc("cnn4_c64_32x32", spec, params, X1, X2)


@pytest.fixture(scope="module")
def c4x4_reference():
    spec, params, X1, X2 = wl.make_workload("cnn4_c64_4x4")
    ref, d1, d2 = oracle.ntk_jc_with_norms(spec, params, X1, X2, layer_storage=S)
    return spec, params, X1, X2, ref, d1, d2


@pytest.mark.parametrize("order", ["auto", "outside_in", "inside_out"])
def test_cnn4_c64_4x4_full(c4x4_reference, order):
    """The 4-layer CNN on 4x4 images in full, in the cost model's mixed orders (the three
    64->64 convolutions inside-out, the 3-channel one outside-in: both the pair-sum and the
    split-K kernels run) and forced all-outside-in and all-inside-out."""
    from paper_2206_08720_amd import _lib
    spec, params, X1, X2, ref, d1, d2 = c4x4_reference
    opt = {"auto": _lib.NTK_CONV_ORDER_AUTO, "outside_in": _lib.NTK_CONV_ORDER_OUTSIDE_IN,
           "inside_out": _lib.NTK_CONV_ORDER_INSIDE_OUT}[order]
    print(f"[parity] cnn4_c64_4x4 order={order}", flush=True)
    prof = {}
    got = gpu_ntk(spec, params, X1, X2, options={_lib.NTK_OPT_CONV_ORDER: opt}, profile=prof)
    cs, nw = errors(got, ref, d1, d2)
    report(f"cnn4_c64_4x4 {order}", cs, nw)
    assert got.shape == ref.shape and cs <= TOL and nw <= TOL
    assert ("conv_pairsum" in prof) == (order != "outside_in")
    assert ("ntk_splitk" in prof) == (order != "inside_out")


CASES = [
    # label, spec, n1, n2
    ("one conv layer, 1x1 images", wl.cnn_spec("c1", (1, 1), 3, [8], 4), 5, 6),
    ("channels not multiple of 4, erf", wl.cnn_spec("c2", (5, 3), 5, [6, 10], 3, act="erf"), 5, 7),
    ("ragged 7x9, 3 layers", wl.cnn_spec("c3", (7, 9), 3, [16, 12, 20], 10), 9, 4),
    ("O=1, n1=n2=1", wl.cnn_spec("c4", (6, 6), 4, [8, 8], 1), 1, 1),
    ("tile-spanning rows, 8x8", wl.cnn_spec("c5", (8, 8), 3, [32, 32], 10), 23, 17),
    # 32-channel layers take the direct-to-LDS patch loads; 5 x 7 images leave ragged row
    # tiles and padding taps on every border
    ("direct-to-LDS patches, ragged 5x7", wl.cnn_spec("c6", (5, 7), 3, [32, 32, 32], 3), 5, 4),
    ("direct-to-LDS patches, 1x1 images", wl.cnn_spec("c7", (1, 1), 4, [32, 64], 2), 3, 7),
    # image width a multiple of 32: each 32-pixel K tile of the weight-space product is one run
    # of an image row (tiles at x = 0 and x = 32 of each of the 3 rows)
    ("aligned pixel rows, 3x64 images", wl.cnn_spec("c8", (3, 64), 3, [32, 32], 3), 4, 3),
    # 3 input channels on 16x20 images: the weight-space product of the first layer on the
    # direct-to-LDS path through a copy padded to 4 channels (the pad columns not stored)
    ("3 input channels padded to 4, 16x20", wl.cnn_spec("c9", (16, 20), 3, [16, 12], 4), 3, 4),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_cnn_edge_shapes(case):
    label, spec, n1, n2 = case
    params = wl.make_params(spec, 300 + n1, "2/fan_in")
    X1 = wl.make_inputs(spec, n1, 310 + n1)
    X2 = wl.make_inputs(spec, n2, 320 + n2)
    _vs_jc(label, spec, params, X1, X2)


FOLD_CASES = [
    # label, spec, n1, n2, folded: the last convolution's summand through per-channel Grams of
    # its O-free rows (its cotangent is the readout's through the global pool)
    ("3x3 last, ragged 6x7", wl.cnn_layers_spec("f1", (6, 7), 3, [("conv3x3", 16, "relu", True),
                                                                 ("conv3x3", 24, "erf", False)], 5), 7, 5, True),
    ("pointwise last, 32 channels", wl.cnn_layers_spec("f2", (4, 8), 4, [("conv3x3", 32, "relu", False),
                                                                        ("conv1x1", 32, "relu", True)], 3), 6, 9, True),
    # a single convolution without bias: no other weight-space column, so no fold
    ("single convolution", wl.cnn_layers_spec("f3", (5, 5), 3, [("conv3x3", 8, "relu", False)], 4), 4, 3, False),
]


@pytest.mark.parametrize("variant", [("full", "full"), ("trace", "full"), ("full", "diagonal"),
                                     ("trace", "diagonal")], ids=lambda v: f"{v[0]}-{v[1]}")
@pytest.mark.parametrize("symmetric", [True, False])
@pytest.mark.parametrize("case", FOLD_CASES, ids=[c[0] for c in FOLD_CASES])
def test_folded_last_convolution(case, symmetric, variant):
    """The last convolution's O outputs factor out of its weight-space product: A[n, c, k] from
    act'(z) alone, Theta += sum_c Wr[o1, c] Wr[o2, c] (A1 A2^T)_c / D^2 (the trace: weights
    sum_o Wr[o, c]^2; the batch diagonal: the Grams' diagonals).  Parity against the oracle,
    forced outside-in, with X2 = X1 on the symmetric schedule and distinct batches otherwise; the
    fold's Grams are a second launch of the Gram class."""
    from paper_2206_08720_amd import _lib
    from tests.gpu_helpers import scaled_errors, variant_of, variant_scale
    label, spec, n1, n2, folded = case
    output, batch = variant
    if batch == "diagonal":
        n2 = n1
    params = wl.make_params(spec, 600 + n1, "2/fan_in")
    X1 = wl.make_inputs(spec, n1, 610 + n1)
    X2 = X1 if symmetric else wl.make_inputs(spec, n2, 620 + n2)
    prof = {}
    got = gpu_ntk(spec, params, X1, X2, symmetric=symmetric,
                  options={_lib.NTK_OPT_CONV_ORDER: _lib.NTK_CONV_ORDER_OUTSIDE_IN}, profile=prof,
                  variant=(output, batch, 0))
    ref, d1, d2 = oracle.ntk_jc_with_norms(spec, params, X1, X2, layer_storage=S)
    if variant == ("full", "full"):
        cs, nw = errors(got, ref, d1, d2)
    else:
        ref = variant_of(ref, output, batch, 0)
        cs, nw = scaled_errors(got, ref, variant_scale(d1, d2, output, batch, 0))
    report(f"fold {label} {output}/{batch} sym={symmetric}", cs, nw)
    assert got.shape == ref.shape and cs <= TOL and nw <= TOL
    assert prof["gram"][1] == (2 if folded else 1)


@pytest.mark.parametrize("symmetric", [True, False])
def test_cnn_aliased_inputs(symmetric):
    spec = wl.cnn_spec("alias", (6, 5), 3, [16, 16], 10)
    params = wl.make_params(spec, 401, "2/fan_in")
    X = wl.make_inputs(spec, 30, 402)
    got = _vs_jc(f"cnn aliased sym={symmetric}", spec, params, X, X, symmetric=symmetric)
    N, O = got.shape[0], got.shape[2]
    M = got.transpose(0, 2, 1, 3).reshape(N * O, N * O)
    np.testing.assert_allclose(M, M.T, rtol=0, atol=1e-5 * np.abs(M).max())


def test_cnn_determinism_and_reuse():
    from paper_2206_08720_amd.ntk import NTK
    spec = wl.cnn_spec("det", (8, 8), 3, [16, 16], 5)
    params = wl.make_params(spec, 501, "2/fan_in")
    X1 = wl.make_inputs(spec, 12, 502)
    X2 = wl.make_inputs(spec, 9, 503)
    h = NTK(spec, 16, 16)
    try:
        a = gpu_ntk(spec, params, X1, X2, handle=h)
        b = gpu_ntk(spec, params, X1, X2, handle=h)
        assert np.array_equal(a, b), "two calls must be bit-identical"
        c = gpu_ntk(spec, params, X1[:3], X2[:2], handle=h)
        ref, d1, d2 = oracle.ntk_jc_with_norms(spec, params, X1[:3], X2[:2], layer_storage=S)
        cs, nw = errors(c, ref, d1, d2)
        assert cs <= TOL and nw <= TOL
    finally:
        h.close()


# ---- contraction order: outside-in vs inside-out (appendix "CNN NTK Complexity") ----------
ORDER_CASES = [
    ("D=1", wl.cnn_spec("o1", (1, 1), 3, [16, 16], 10), 6, 5),
    ("D=4", wl.cnn_spec("o4", (2, 2), 3, [16, 16], 10), 6, 5),
    ("D=16", wl.cnn_spec("o16", (4, 4), 3, [64, 64, 64], 10), 8, 7),
    ("D=16 erf, C=20, O=7", wl.cnn_spec("o16e", (4, 4), 5, [20, 20], 7, act="erf"), 5, 9),
    # the matrix-core pair kernel's other pixel blocks (Dp = 32, 48, 64), ragged images, odd
    # channel counts and several blocks of 16 outputs (O = 20: 2 x 2 output blocks, O = 33: 3 x 3)
    ("D=36 (6x6), C=24", wl.cnn_spec("o36", (6, 6), 3, [24, 24], 10), 7, 6),
    ("D=64 (8x8), C=32, O=5", wl.cnn_spec("o64", (8, 8), 3, [32, 32], 5), 5, 6),
    ("D=49 (7x7), O=20", wl.cnn_spec("o49", (7, 7), 3, [16, 16], 20), 5, 4),
    ("D=9 (3x3), odd channels, O=33", wl.cnn_spec("o9", (3, 3), 5, [7, 9], 33, act="erf"), 4, 5),
    ("D=30 (5x6), 3 layers, O=17", wl.cnn_spec("o30", (5, 6), 2, [12, 20, 16], 17), 3, 7),
]


@pytest.mark.parametrize("order", ["outside_in", "inside_out", "auto"])
@pytest.mark.parametrize("case", ORDER_CASES, ids=[c[0] for c in ORDER_CASES])
def test_conv_contraction_orders(case, order):
    from paper_2206_08720_amd import _lib
    label, spec, n1, n2 = case
    code = {"outside_in": _lib.NTK_CONV_ORDER_OUTSIDE_IN, "inside_out": _lib.NTK_CONV_ORDER_INSIDE_OUT,
            "auto": _lib.NTK_CONV_ORDER_AUTO}[order]
    params = wl.make_params(spec, 700 + n1, "2/fan_in")
    X1 = wl.make_inputs(spec, n1, 710 + n1)
    X2 = wl.make_inputs(spec, n2, 720 + n2)
    prof = {}
    got = gpu_ntk(spec, params, X1, X2, options={_lib.NTK_OPT_CONV_ORDER: code}, profile=prof)
    ref, d1, d2 = oracle.ntk_jc_with_norms(spec, params, X1, X2, layer_storage=S)
    cs, nw = errors(got, ref, d1, d2)
    report(f"{label} order={order} kernels={sorted(prof)}", cs, nw)
    assert cs <= TOL and nw <= TOL
    if order == "inside_out":
        assert "conv_pairsum" in prof and "ntk_splitk" not in prof
    if order == "outside_in":
        assert "conv_pairsum" not in prof and "ntk_splitk" in prof
    if order == "auto" and label == "D=16":
        # the first layer (Cin = 3) is cheaper outside-in, the 64-channel layers inside-out
        assert "conv_pairsum" in prof and "ntk_splitk" in prof


def test_inside_out_symmetric():
    from paper_2206_08720_amd import _lib
    spec = wl.cnn_spec("ios", (3, 3), 4, [12, 12], 6)
    params = wl.make_params(spec, 801, "2/fan_in")
    X = wl.make_inputs(spec, 11, 802)
    got = gpu_ntk(spec, params, X, X, options={_lib.NTK_OPT_CONV_ORDER: _lib.NTK_CONV_ORDER_INSIDE_OUT})
    ref, d1, d2 = oracle.ntk_jc_with_norms(spec, params, X, X, layer_storage=S)
    cs, nw = errors(got, ref, d1, d2)
    report("inside-out symmetric", cs, nw)
    assert cs <= TOL and nw <= TOL


def test_inside_out_rejects_large_images_without_enqueuing():
    import torch
    from paper_2206_08720_amd import _lib
    from paper_2206_08720_amd.ntk import NTK
    from tests.gpu_helpers import to_dev
    spec = wl.cnn_spec("big", (9, 9), 3, [8], 2)         # D = 81 > 64 pixels
    params = to_dev(wl.make_params(spec, 1, "2/fan_in"))
    X = to_dev([wl.make_inputs(spec, 2, 2)])[0]
    h = NTK(spec, 2, 2)
    try:
        h.set_option(_lib.NTK_OPT_CONV_ORDER, _lib.NTK_CONV_ORDER_INSIDE_OUT)
        out = torch.full((2, 2, 2, 2), 3.0, device="cuda")
        with pytest.raises(_lib.NTKError) as ei:
            h.compute(params, X, X, out=out)
        assert ei.value.code == _lib.NTK_E_UNSUPPORTED
        torch.cuda.synchronize()
        assert bool((out == 3.0).all())
    finally:
        h.close()
