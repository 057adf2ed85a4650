"""Seeded synthetic workloads: network specifications, parameters and inputs.

This module holds no NTK arithmetic.  It only describes networks as plain data
and draws their parameters and inputs from seeded numpy generators (PCG64), in
float32.  The same float32 buffers are handed to the fp64 CPU oracle (which
upcasts them exactly) and to the GPU library, so the two never need matching
random-number streams.

Network specification (a plain dict)::

    {"name": str,
     "input_shape": (d0,)  for a fully-connected net, or (H, W, C) NHWC for a CNN,
     "layers": [ {"kind": "dense",     "in": int, "out": int, "act": "relu"|"erf"|"none", "bias": bool},
                 {"kind": "conv3x3",   "in": int, "out": int, "act": ..., "bias": bool},
                 {"kind": "conv1x1",   "in": int, "out": int, "act": ..., "bias": bool},
                 {"kind": "dwconv3x3", "in": C,   "out": C,   "act": ..., "bias": bool},
                 {"kind": "scale",     "in": C,   "out": C,   "act": ..., "bias": bool},
                 {"kind": "avgpool2"},
                 {"kind": "gap"} ]}

Parameter order: layer by layer, the weight first and then the bias if the
layer has one.  Dense and pointwise (1x1 convolution) weights are [out, in] row-major;
3x3 convolution weights are [Cout, 3, 3, Cin] (OHWI); depthwise 3x3 weights are [3, 3, C] (one 3x3
filter per channel, channel fastest); scale weights are [C].  The forward map
is z = h W^T (+ b) for a dense layer and, at every pixel, for a pointwise layer, a SAME
(zero pad 1), stride-1 cross-correlation for a 3x3 conv layer (per channel for the depthwise one),
z = h * w (+ b) broadcast over the pixels for a scale layer, and
h_next = act(z).  "avgpool2" is the mean over non-overlapping 2x2 windows
(stride 2; H and W even) and "gap" the mean over all pixels; neither has
parameters or an activation.  The last layer is a dense layer with act
"none"; its output is f.

The five reference workloads follow the fully-connected and convolutional
networks of the paper's Section 4 ("Examples"): Section 4.1's FCN with L hidden
layers of width W, and Section 4.2's CNN (3x3 SAME unit-stride convolutions,
global average pooling before the readout).  Inputs are MNIST-, CIFAR-10-shaped
or generic random arrays; no dataset item is reproduced.
"""
from __future__ import annotations

import copy
import numpy as np

__all__ = [
    "WORKLOADS",
    "workload_names",
    "fcn_spec",
    "cnn_spec",
    "cnn_layers_spec",
    "PARAM_KINDS",
    "make_params",
    "make_inputs",
    "make_workload",
    "param_shapes",
    "output_dim",
]


def fcn_spec(name, d_in, widths, d_out, act="relu", bias=False):
    """Fully-connected net d_in -> widths[0] -> ... -> widths[-1] -> d_out."""
    dims = [d_in] + list(widths) + [d_out]
    layers = []
    for i in range(len(dims) - 1):
        last = i == len(dims) - 2
        layers.append({"kind": "dense", "in": dims[i], "out": dims[i + 1],
                       "act": "none" if last else act, "bias": bool(bias)})
    return {"name": name, "input_shape": (d_in,), "layers": layers}


def cnn_spec(name, hw, c_in, channels, d_out, act="relu", bias=False):
    """CNN: len(channels) x [conv3x3 SAME -> act], global average pool, dense readout."""
    H, W = hw
    layers = []
    cin = c_in
    for c in channels:
        layers.append({"kind": "conv3x3", "in": cin, "out": c, "act": act, "bias": bool(bias)})
        cin = c
    layers.append({"kind": "gap"})
    layers.append({"kind": "dense", "in": cin, "out": d_out, "act": "none", "bias": False})
    return {"name": name, "input_shape": (H, W, c_in), "layers": layers}


def cnn_layers_spec(name, hw, c_in, blocks, d_out):
    """CNN from a list of blocks, then global average pooling and a dense readout.

    Each block is one of ("conv3x3", c_out, act, bias), ("conv1x1", c_out, act, bias),
    ("dwconv3x3", act, bias), ("scale", act, bias) or ("avgpool2",).
    """
    H, W = hw
    layers = []
    c = c_in
    for b in blocks:
        kind = b[0]
        if kind in ("conv3x3", "conv1x1"):
            _, co, act, bias = b
            layers.append({"kind": kind, "in": c, "out": co, "act": act, "bias": bool(bias)})
            c = co
        elif kind in ("dwconv3x3", "scale"):
            _, act, bias = b
            layers.append({"kind": kind, "in": c, "out": c, "act": act, "bias": bool(bias)})
        elif kind == "avgpool2":
            layers.append({"kind": kind})
        else:
            raise ValueError(f"unknown block {kind!r}")
    layers.append({"kind": "gap"})
    layers.append({"kind": "dense", "in": c, "out": d_out, "act": "none", "bias": False})
    return {"name": name, "input_shape": (H, W, c_in), "layers": layers}


# layer kinds that carry parameters (a weight, then an optional bias) and an activation
PARAM_KINDS = ("dense", "conv3x3", "conv1x1", "dwconv3x3", "scale")


def param_shapes(spec):
    """Shapes of the parameter tensors in order (weight, then bias if present)."""
    shapes = []
    for L in spec["layers"]:
        if L["kind"] in ("dense", "conv1x1"):
            shapes.append((L["out"], L["in"]))
            if L["bias"]:
                shapes.append((L["out"],))
        elif L["kind"] == "conv3x3":
            shapes.append((L["out"], 3, 3, L["in"]))
            if L["bias"]:
                shapes.append((L["out"],))
        elif L["kind"] == "dwconv3x3":
            shapes.append((3, 3, L["out"]))
            if L["bias"]:
                shapes.append((L["out"],))
        elif L["kind"] == "scale":
            shapes.append((L["out"],))
            if L["bias"]:
                shapes.append((L["out"],))
    return shapes


def output_dim(spec):
    return spec["layers"][-1]["out"]


def make_params(spec, seed, weight_var="1/fan_in", bias_var=0.01):
    """Draw float32 parameters.  weight_var is "1/fan_in" or "2/fan_in" (a variance).

    fan_in is `in` for a dense or pointwise layer, 9*Cin for a 3x3 convolution and 9
    for a depthwise one.  Scale weights are drawn around 1, as N(1, 0.01), like the
    affine scale of a normalisation layer.  Biases are N(0, bias_var)
    (bias_var is a variance).
    """
    rng = np.random.default_rng(seed)
    scale = {"1/fan_in": 1.0, "2/fan_in": 2.0}[weight_var]
    params = []
    for L in spec["layers"]:
        if L["kind"] in ("dense", "conv1x1"):
            fan_in = L["in"]
            shape = (L["out"], L["in"])
        elif L["kind"] == "conv3x3":
            fan_in = 9 * L["in"]
            shape = (L["out"], 3, 3, L["in"])
        elif L["kind"] == "dwconv3x3":
            fan_in = 9
            shape = (3, 3, L["out"])
        elif L["kind"] == "scale":
            params.append((1.0 + 0.1 * rng.standard_normal((L["out"],))).astype(np.float32))
            if L["bias"]:
                params.append((rng.standard_normal((L["out"],)) * np.sqrt(bias_var)).astype(np.float32))
            continue
        else:
            continue
        std = np.sqrt(scale / fan_in)
        params.append((rng.standard_normal(shape) * std).astype(np.float32))
        if L["bias"]:
            params.append((rng.standard_normal((L["out"],)) * np.sqrt(bias_var)).astype(np.float32))
    return params


def make_inputs(spec, n, seed, dist="normal"):
    """Draw a float32 batch [n, *input_shape]: N(0,1) or uniform[0,1)."""
    rng = np.random.default_rng(seed)
    shape = (n,) + tuple(spec["input_shape"])
    if dist == "normal":
        x = rng.standard_normal(shape)
    elif dist == "uniform":
        x = rng.random(shape)
    else:
        raise ValueError(dist)
    return x.astype(np.float32)


# The reference workloads.  "depth D" = D hidden layers of width W plus a
# dense readout (D + 1 weight matrices), the paper's FCN of Section 4.1.
WORKLOADS = {
    "tiny_relu_mlp": dict(
        index=1, spec=fcn_spec("tiny_relu_mlp", 16, [32, 32], 4, act="relu", bias=True),
        n1=8, n2=8, weight_var="1/fan_in", bias_var=0.01, x_dist="normal", x2_is_x1=False),
    "relu_mlp_d4_w512": dict(
        index=2, spec=fcn_spec("relu_mlp_d4_w512", 784, [512] * 4, 10, act="relu"),
        n1=128, n2=128, weight_var="1/fan_in", x_dist="uniform", x2_is_x1=True),
    "relu_mlp_d8_w2048": dict(
        index=3, spec=fcn_spec("relu_mlp_d8_w2048", 3072, [2048] * 8, 10, act="relu"),
        n1=512, n2=512, weight_var="2/fan_in", x_dist="normal", x2_is_x1=False),
    "erf_mlp_d3_w4096": dict(
        index=4, spec=fcn_spec("erf_mlp_d3_w4096", 1024, [4096] * 3, 100, act="erf"),
        n1=128, n2=128, weight_var="1/fan_in", x_dist="normal", x2_is_x1=False),
    "cnn4_c64_32x32": dict(
        index=5, spec=cnn_spec("cnn4_c64_32x32", (32, 32), 3, [64] * 4, 10, act="relu"),
        n1=64, n2=64, weight_var="2/fan_in", x_dist="normal", x2_is_x1=False),
    # The further structure rules of the paper's appendix on structured derivatives, one
    # layer kind each: convolution biases (output block-tiled), a depthwise convolution
    # (block-diagonal) followed by a pointwise one (a depthwise-separable block), a
    # per-channel scale with bias (block-diagonal over channels and output block-tiled over
    # pixels), and a 2x2 average pool between convolutions.
    "cnn_struct_c64_32x32": dict(
        index=6, spec=cnn_layers_spec(
            "cnn_struct_c64_32x32", (32, 32), 3,
            [("conv3x3", 64, "relu", True), ("dwconv3x3", "relu", True), ("conv1x1", 64, "relu", True),
             ("avgpool2",), ("conv3x3", 64, "relu", True), ("scale", "relu", True),
             ("conv3x3", 64, "relu", True)],
            10),
        n1=64, n2=64, weight_var="2/fan_in", bias_var=0.01, x_dist="normal", x2_is_x1=False),
    # The 4-layer CNN on 4x4 images (D = 16): the cost model of the appendix "CNN NTK
    # Complexity" contracts the three 64->64 convolutions inside-out (about 9x cheaper than
    # outside-in there) and the 3-channel one outside-in.
    "cnn4_c64_4x4": dict(
        index=7, spec=cnn_spec("cnn4_c64_4x4", (4, 4), 3, [64] * 4, 10, act="relu"),
        n1=64, n2=64, weight_var="2/fan_in", x_dist="normal", x2_is_x1=False),
}


def workload_names():
    return list(WORKLOADS)


def make_workload(name, n1=None, n2=None):
    """Return (spec, params, X1, X2) for a named workload.

    Seeds: parameters 1000+i, X1 2000+i, X2 3000+i (i = the workload's index).
    n1/n2 may shrink the batches (the first rows of the full batches are kept,
    so a smaller call sees exactly a prefix of the full-size inputs).  When the
    workload has X2 = X1, the returned X2 is the same array object as X1.
    """
    w = WORKLOADS[name]
    spec = copy.deepcopy(w["spec"])
    i = w["index"]
    params = make_params(spec, 1000 + i, w["weight_var"], w.get("bias_var", 0.01))
    X1 = make_inputs(spec, w["n1"], 2000 + i, w["x_dist"])
    if w["x2_is_x1"]:
        X2 = X1
    else:
        X2 = make_inputs(spec, w["n2"], 3000 + i, w["x_dist"])
    if n1 is not None:
        X1 = X1[:n1]
        if w["x2_is_x1"]:
            X2 = X1
    if n2 is not None and not w["x2_is_x1"]:
        X2 = X2[:n2]
    return spec, params, X1, X2
