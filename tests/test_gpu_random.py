"""Seeded random architectures against the fp64 oracle (needs an MI355X).

Each case draws a network from a fixed seed: for CNNs a sequence of the spatial layer kinds
(3x3, pointwise and depthwise convolutions, scale layers, 2x2 pools where the image allows),
random channel counts (odd ones included), image sizes, activations and biases; for FCNs a
random depth, widths, activation and biases; then random O and batch sizes.  The GPU result
must match the Jacobian-contraction oracle (float32 layer storage) to the parity bar, under
the default schedule and with X2 = X1, and then under one seeded choice of output / batch
variant, contraction order of the 3x3 convolutions and method.  The seeds are fixed, so every
run checks the same networks.
"""
import numpy as np
import pytest

import oracle
import workloads as wl
from tests.gpu_helpers import TOL, errors, gpu_ntk, report, scaled_errors, variant_of, variant_scale

pytestmark = pytest.mark.gpu
S = "fp32"
ACTS = ["relu", "erf", "none"]


def random_cnn(seed):
    rng = np.random.default_rng(seed)
    H, W = (int(rng.integers(1, 5)) * 2, int(rng.integers(1, 5)) * 2) if rng.random() < 0.8 else \
        (int(rng.integers(1, 8)), int(rng.integers(1, 8)))
    c_in = int(rng.choice([1, 2, 3, 4, 5, 8]))
    blocks, c, h, w, params = [], c_in, H, W, 0
    for _ in range(int(rng.integers(1, 6))):
        kinds = ["conv3x3", "conv1x1", "dwconv3x3", "scale"] + (["avgpool2"] if h % 2 == 0 and w % 2 == 0 else [])
        k = str(rng.choice(kinds))
        act, bias = str(rng.choice(ACTS)), bool(rng.random() < 0.5)
        if k in ("conv3x3", "conv1x1"):
            c = int(rng.choice([1, 3, 4, 7, 8, 16, 32]))
            blocks.append((k, c, act, bias))
            params += 1
        elif k in ("dwconv3x3", "scale"):
            blocks.append((k, act, bias))
            params += 1
        else:
            blocks.append((k,))
            h, w = h // 2, w // 2
    if params == 0:
        blocks.append(("conv3x3", 4, "relu", True))
    O = int(rng.integers(1, 13))
    spec = wl.cnn_layers_spec(f"rcnn{seed}", (H, W), c_in, blocks, O)
    return spec, int(rng.integers(1, 10)), int(rng.integers(1, 10))


def random_fcn(seed):
    rng = np.random.default_rng(seed)
    d_in = int(rng.integers(1, 70))
    widths = [int(rng.integers(1, 130)) for _ in range(int(rng.integers(0, 5)))]
    O = int(rng.integers(1, 13))
    spec = wl.fcn_spec(f"rfcn{seed}", d_in, widths, O, act=str(rng.choice(["relu", "erf"])),
                       bias=bool(rng.random() < 0.5))
    return spec, int(rng.integers(1, 40)), int(rng.integers(1, 40))


def _check(name, spec, n1, n2, seed):
    params = wl.make_params(spec, 5000 + seed, "2/fan_in", bias_var=0.1)
    X1 = wl.make_inputs(spec, n1, 6000 + seed)
    X2 = wl.make_inputs(spec, n2, 7000 + seed)
    layers = [L["kind"] + (f"{L['out']}" if "out" in L else "") for L in spec["layers"]]
    print(f"[random] {name}: input {tuple(spec['input_shape'])} layers {layers} n1={n1} n2={n2}", flush=True)
    got = gpu_ntk(spec, params, X1, X2)
    ref, d1, d2 = oracle.ntk_jc_with_norms(spec, params, X1, X2, layer_storage=S)
    cs, nw = errors(got, ref, d1, d2)
    report(name, cs, nw)
    assert got.shape == ref.shape and cs <= TOL and nw <= TOL
    got = gpu_ntk(spec, params, X1, X1)
    ref, d1, _ = oracle.ntk_jc_with_norms(spec, params, X1, X1, layer_storage=S)
    cs, nw = errors(got, ref, d1, d1)
    report(name + " aliased", cs, nw)
    assert cs <= TOL and nw <= TOL
    # one seeded choice of variant, conv order and method
    from paper_2206_08720_amd import _lib
    rng = np.random.default_rng(8000 + seed)
    output = str(rng.choice(["full", "trace", "logit"]))
    batch = str(rng.choice(["full", "diagonal"]))
    O = spec["layers"][-1]["out"]
    logit = int(rng.integers(0, O))
    opts = {_lib.NTK_OPT_CONV_ORDER: int(rng.choice([_lib.NTK_CONV_ORDER_AUTO, _lib.NTK_CONV_ORDER_OUTSIDE_IN,
                                                     _lib.NTK_CONV_ORDER_INSIDE_OUT])),
            _lib.NTK_OPT_METHOD: int(rng.choice([_lib.NTK_METHOD_STRUCTURED, _lib.NTK_METHOD_JACOBIAN]))}
    Xb = X2 if batch == "full" else wl.make_inputs(spec, n1, 9000 + seed)
    full, d1, d2 = oracle.ntk_jc_with_norms(spec, params, X1, Xb, layer_storage=S)
    print(f"[random] {name}: variant {output}/{batch} logit {logit} options {opts}", flush=True)
    got = gpu_ntk(spec, params, X1, Xb, options=opts, variant=(output, batch, logit))
    ref = variant_of(full, output, batch, logit)
    cs, nw = scaled_errors(got, ref, variant_scale(d1, d2, output, batch, logit))
    report(f"{name} {output}/{batch}", cs, nw)
    assert got.shape == ref.shape and cs <= TOL and nw <= TOL


@pytest.mark.parametrize("seed", range(64))
def test_random_cnn(seed):
    spec, n1, n2 = random_cnn(seed)
    _check(f"random cnn {seed}", spec, n1, n2, seed)


@pytest.mark.parametrize("seed", range(32))
def test_random_fcn(seed):
    spec, n1, n2 = random_fcn(100 + seed)
    _check(f"random fcn {seed}", spec, n1, n2, 100 + seed)
