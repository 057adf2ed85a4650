"""Empirical NTK by explicit Jacobian contraction, in float64.  TEST INFRASTRUCTURE ONLY.

The network is described by the plain-data spec of the `workloads` module.
Every step follows the paper's definitions:

* Theta(x1, x2) = [df(x1)/dtheta] [df(x2)/dtheta]^T, an O x O block per input
  pair, which is a sum over the weight tensors theta^l of
  [df(x1)/dtheta^l] [df(x2)/dtheta^l]^T  (Section 3.1.1, Eq. "ntk_def_main").
* The Jacobian df/dtheta is the reverse-mode Jacobian: O vector-Jacobian
  products, one per row of the identity I_O (Section 3.1.3).  Each VJP pulls
  a one-hot output cotangent back through the layers; the cotangent of a
  weight tensor is then formed explicitly (Section 3.1.2, Eq. "jvp_vjp_main").
* The contraction of the two Jacobians is the "Jacobian contraction" baseline
  of Section 3.2: N1 N2 O^2 P multiply-adds.

Layer storage: with layer_storage="fp64" (default) every intermediate value is
float64, the plain definition.  With layer_storage="fp32" each layer's output
h_{l+1} = act(z_l) is rounded to float32 before it feeds the next layer, as in
a network evaluated in the paper's 32-bit precision (appendix "Experimental
Details"); pre-activations are still accumulated in float64.  ReLU is
discontinuous in its derivative, so whether act'(z) is 0 or 1 for a
pre-activation within rounding distance of 0 depends on the exact stored
inputs; this mode makes that decision a function of float32-stored layer
inputs, the values the GPU library decides on.

Conventions (the paper leaves them to the framework): ReLU'(0) = 0;
erf'(z) = 2/sqrt(pi) exp(-z^2); convolutions are SAME (zero pad 1), stride 1,
cross-correlation, NHWC activations, OHWI weights ([3, 3, C] for a depthwise
convolution, [Cout, Cin] for a pointwise 1x1 convolution); a scale layer multiplies channel c (or feature c) by w[c];
"avgpool2" is the mean over 2x2 windows with stride 2; "gap" is the mean over
the H*W pixels.  Inputs arrive as float32 and are upcast exactly to float64.

Layer kinds and the structure of their weight-space Jacobian dz/dtheta (the
paper's appendix on structured derivatives; the oracle forms each block
explicitly all the same):
* dense, conv3x3, conv1x1: constant-block-diagonal (a matrix product along one axis);
* dwconv3x3: block-diagonal over channels (channel c's filter only feeds
  output channel c);
* scale: block-diagonal over channels, and for images also output block-tiled
  (the same w[c] multiplies every pixel);
* biases of conv, depthwise and scale layers: output block-tiled (one value
  broadcast over the pixels).
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf as _erf

__all__ = ["forward", "jacobian", "ntk_jc", "ntk_jc_with_norms", "param_count",
           "jacobian_blocks"]


# ----------------------------------------------------------------------------- activations
def _phi(act, z):
    if act == "relu":
        return np.maximum(z, 0.0)
    if act == "erf":
        return _erf(z)
    if act == "none":
        return z
    raise ValueError(f"unknown activation {act!r}")


def _dphi(act, z):
    if act == "relu":
        return (z > 0.0).astype(np.float64)
    if act == "erf":
        return (2.0 / math.sqrt(math.pi)) * np.exp(-z * z)
    if act == "none":
        return np.ones_like(z)
    raise ValueError(f"unknown activation {act!r}")


# ----------------------------------------------------------------------------- 3x3 SAME patches
def _patches(h):
    """h [N, H, W, C] -> patches [N, H*W, 9*C], k = (kh, kw, ci); zero padding of 1.

    Output pixel (y, x) and tap (kh, kw) read input pixel (y + kh - 1, x + kw - 1).
    """
    N, H, W, C = h.shape
    hp = np.zeros((N, H + 2, W + 2, C))
    hp[:, 1:H + 1, 1:W + 1, :] = h
    taps = [hp[:, kh:kh + H, kw:kw + W, :] for kh in range(3) for kw in range(3)]
    return np.stack(taps, axis=3).reshape(N, H * W, 9 * C)


def _patches_transpose(dp, H, W, C):
    """Adjoint of `_patches` on a leading batch: dp [..., H*W, 9*C] -> [..., H, W, C]."""
    lead = dp.shape[:-2]
    dp = dp.reshape(lead + (H, W, 3, 3, C))
    out = np.zeros(lead + (H + 2, W + 2, C))
    for kh in range(3):
        for kw in range(3):
            out[..., kh:kh + H, kw:kw + W, :] += dp[..., kh, kw, :]
    return out[..., 1:H + 1, 1:W + 1, :]


# ----------------------------------------------------------------------------- parameters
# layer kinds with a weight (then an optional bias) and an activation
_PARAM_KINDS = ("dense", "conv3x3", "conv1x1", "dwconv3x3", "scale")


def _split_params(spec, params):
    """Pair each parametrised layer with its (weight, bias-or-None), as float64."""
    out = []
    i = 0
    for L in spec["layers"]:
        if L["kind"] in _PARAM_KINDS:
            w = np.asarray(params[i], dtype=np.float64)
            i += 1
            b = None
            if L["bias"]:
                b = np.asarray(params[i], dtype=np.float64)
                i += 1
            out.append((w, b))
        else:
            out.append(None)
    if i != len(params):
        raise ValueError("parameter list does not match the spec")
    return out


def param_count(spec):
    P = 0
    for L in spec["layers"]:
        if L["kind"] in ("dense", "conv1x1"):
            P += L["out"] * L["in"] + (L["out"] if L["bias"] else 0)
        elif L["kind"] == "conv3x3":
            P += L["out"] * 9 * L["in"] + (L["out"] if L["bias"] else 0)
        elif L["kind"] == "dwconv3x3":
            P += 9 * L["out"] + (L["out"] if L["bias"] else 0)
        elif L["kind"] == "scale":
            P += L["out"] + (L["out"] if L["bias"] else 0)
    return P


# ----------------------------------------------------------------------------- forward pass
def _store(h, layer_storage):
    if layer_storage == "fp64":
        return h
    if layer_storage == "fp32":
        return h.astype(np.float32).astype(np.float64)
    raise ValueError(f"unknown layer_storage {layer_storage!r}")


def _forward_record(spec, params, X, layer_storage="fp64"):
    """Run f on a batch, keeping each layer's input h and pre-activation z."""
    layers = spec["layers"]
    wb = _split_params(spec, params)
    h = np.asarray(X, dtype=np.float64)
    rec = []
    for L, p in zip(layers, wb):
        if L["kind"] == "dense":
            w, b = p
            z = h @ w.T
            if b is not None:
                z = z + b
            rec.append({"h": h, "z": z})
            h = _store(_phi(L["act"], z), layer_storage)
        elif L["kind"] == "conv3x3":
            w, b = p
            N, H, W, C = h.shape
            pt = _patches(h)
            z = pt @ w.reshape(w.shape[0], -1).T
            if b is not None:
                z = z + b
            z = z.reshape(N, H, W, w.shape[0])
            rec.append({"h": h, "z": z, "patches": pt})
            h = _store(_phi(L["act"], z), layer_storage)
        elif L["kind"] == "conv1x1":
            w, b = p                                          # [Cout, Cin], every pixel
            z = h @ w.T
            if b is not None:
                z = z + b
            rec.append({"h": h, "z": z})
            h = _store(_phi(L["act"], z), layer_storage)
        elif L["kind"] == "dwconv3x3":
            w, b = p                                          # [3, 3, C]
            N, H, W, C = h.shape
            pt = _patches(h).reshape(N, H * W, 9, C)          # tap t = (kh, kw), channel c
            z = np.einsum("nptc,tc->npc", pt, w.reshape(9, C))
            if b is not None:
                z = z + b
            z = z.reshape(N, H, W, C)
            rec.append({"h": h, "z": z, "patches": pt})
            h = _store(_phi(L["act"], z), layer_storage)
        elif L["kind"] == "scale":
            w, b = p                                          # [C], on the last axis
            z = h * w
            if b is not None:
                z = z + b
            rec.append({"h": h, "z": z})
            h = _store(_phi(L["act"], z), layer_storage)
        elif L["kind"] == "avgpool2":
            N, H, W, C = h.shape
            if H % 2 or W % 2:
                raise ValueError("avgpool2 needs an even image height and width")
            rec.append({"h": h})
            h = _store(h.reshape(N, H // 2, 2, W // 2, 2, C).mean(axis=(2, 4)), layer_storage)
        elif L["kind"] == "gap":
            rec.append({"h": h})
            h = _store(h.mean(axis=(1, 2)), layer_storage)
        else:
            raise ValueError(f"unknown layer kind {L['kind']!r}")
    return rec, h


def forward(spec, params, X, layer_storage="fp64"):
    """f(theta, X) in float64: [N, O]."""
    return _forward_record(spec, params, X, layer_storage)[1]


# ----------------------------------------------------------------------------- reverse-mode Jacobian
def _output_cotangents(spec, params, rec, outputs):
    """Pull the one-hot output cotangents (rows `outputs` of I_O) back through f.

    Returns, per layer, the cotangent of that layer's pre-activation z
    (df_o/dz, shape [N, Os, *z.shape[1:]]) for parametrised layers, None otherwise.
    """
    layers = spec["layers"]
    wb = _split_params(spec, params)
    O = layers[-1]["out"]
    N = rec[0]["h"].shape[0]
    seed = np.eye(O)[list(outputs)]                       # rows of I_O
    g = np.broadcast_to(seed, (N,) + seed.shape).copy()   # df/dz_last: [N, Os, O]
    G = [None] * len(layers)
    for li in range(len(layers) - 1, -1, -1):
        L = layers[li]
        if L["kind"] == "dense":
            G[li] = g
            w, _ = wb[li]
            g = g @ w                                     # df/dh_li: [N, Os, in]
        elif L["kind"] == "conv3x3":
            G[li] = g
            w, _ = wb[li]
            N_, H, W, Cout = rec[li]["z"].shape
            Cin = w.shape[3]
            dp = g.reshape(N, g.shape[1], H * W, Cout) @ w.reshape(Cout, -1)   # [N,Os,D,9Cin]
            g = _patches_transpose(dp, H, W, Cin)        # df/dh_li: [N, Os, H, W, Cin]
        elif L["kind"] == "conv1x1":
            G[li] = g
            w, _ = wb[li]
            g = g @ w                                     # df/dh_li: [N, Os, H, W, Cin]
        elif L["kind"] == "dwconv3x3":
            G[li] = g
            w, _ = wb[li]
            N_, H, W, C = rec[li]["z"].shape
            # patch entry (p, t, c) fed z[p, c] with weight w[t, c]
            dp = g.reshape(N, g.shape[1], H * W, 1, C) * w.reshape(9, C)      # [N,Os,D,9,C]
            g = _patches_transpose(dp.reshape(N, g.shape[1], H * W, 9 * C), H, W, C)
        elif L["kind"] == "scale":
            G[li] = g
            w, _ = wb[li]
            g = g * w
        elif L["kind"] == "avgpool2":
            # every input pixel of a 2x2 window feeds that window's mean with weight 1/4
            g = np.repeat(np.repeat(g, 2, axis=2), 2, axis=3) / 4.0
        elif L["kind"] == "gap":
            hin = rec[li]["h"]
            D = hin.shape[1] * hin.shape[2]
            g = np.broadcast_to(g[:, :, None, None, :] / D,
                                g.shape[:2] + hin.shape[1:]).copy()
        if li > 0 and layers[li - 1]["kind"] in _PARAM_KINDS:
            # through the activation of the previous layer: h_li = phi(z_{li-1})
            zprev = rec[li - 1]["z"]
            g = g * _dphi(layers[li - 1]["act"], zprev)[:, None]
    return G


def jacobian_blocks(spec, params, X, outputs=None, max_block_bytes=256 << 20, chunk_rows=None,
                    layer_storage="fp64"):
    """Yield the weight-space Jacobian, block by block: arrays [N*Os, p] (float64).

    Concatenating every yielded block along the last axis gives df/dtheta in the
    parameter order of the spec (row (n, o), column = flat parameter index).
    Large weight tensors are yielded in several column chunks (over the output
    unit c) so that no block exceeds `max_block_bytes` for `chunk_rows` rows
    (default: this call's own row count).  Two calls with the same `chunk_rows`
    yield blocks with identical column ranges.
    """
    layers = spec["layers"]
    O = layers[-1]["out"]
    outputs = list(range(O)) if outputs is None else list(outputs)
    rec, _ = _forward_record(spec, params, X, layer_storage)
    G = _output_cotangents(spec, params, rec, outputs)
    N = np.asarray(X).shape[0]
    R = N * len(outputs)
    Rc = R if chunk_rows is None else max(1, int(chunk_rows))
    for li, L in enumerate(layers):
        if L["kind"] == "dense":
            h = rec[li]["h"]                               # [N, in]
            g = G[li]                                      # [N, Os, out]
            cout, cin = L["out"], L["in"]
            step = max(1, int(max_block_bytes // (8 * Rc * cin)))
            for c0 in range(0, cout, step):
                c1 = min(cout, c0 + step)
                # d z[c] / d W[c, j] = h[j]  ->  J[n, o, c, j] = G[n, o, c] h[n, j]
                J = g[:, :, c0:c1, None] * h[:, None, None, :]
                yield J.reshape(R, (c1 - c0) * cin)
            if L["bias"]:
                yield g.reshape(R, cout)
        elif L["kind"] == "conv3x3":
            pt = rec[li]["patches"]                        # [N, D, 9Cin]
            g = G[li]                                      # [N, Os, H, W, Cout]
            cout, k9 = L["out"], 9 * L["in"]
            D = pt.shape[1]
            gf = g.reshape(N, len(outputs), D, cout)
            step = max(1, int(max_block_bytes // (8 * Rc * k9)))
            for c0 in range(0, cout, step):
                c1 = min(cout, c0 + step)
                # weight sharing over pixels: J[n,o,c,k] = sum_p G[n,o,p,c] patch[n,p,k]
                J = np.swapaxes(gf[:, :, :, c0:c1], 2, 3) @ pt[:, None]   # [N,Os,cc,9Cin]
                yield J.reshape(R, (c1 - c0) * k9)
            if L["bias"]:
                yield gf.sum(axis=2).reshape(R, cout)
        elif L["kind"] == "conv1x1":
            h = rec[li]["h"]                               # [N, H, W, Cin]
            cout, cin = L["out"], L["in"]
            hf = h.reshape(N, -1, cin)                     # [N, D, Cin]
            gf = G[li].reshape(N, len(outputs), -1, cout)  # [N, Os, D, Cout]
            step = max(1, int(max_block_bytes // (8 * Rc * cin)))
            for c0 in range(0, cout, step):
                c1 = min(cout, c0 + step)
                # weight sharing over pixels: J[n,o,c,j] = sum_p G[n,o,p,c] h[n,p,j]
                J = np.swapaxes(gf[:, :, :, c0:c1], 2, 3) @ hf[:, None]    # [N,Os,cc,Cin]
                yield J.reshape(R, (c1 - c0) * cin)
            if L["bias"]:
                yield gf.sum(axis=2).reshape(R, cout)
        elif L["kind"] == "dwconv3x3":
            pt = rec[li]["patches"]                        # [N, D, 9, C]
            C = L["out"]
            D = pt.shape[1]
            gf = G[li].reshape(N, len(outputs), D, C)
            # dz[p, c] / dw[t, c'] = delta_{c c'} patch[p, t, c], shared by every pixel p:
            # J[n, o, t, c] = sum_p G[n, o, p, c] patch[n, p, t, c]
            J = np.einsum("nopc,nptc->notc", gf, pt, optimize=True)
            yield J.reshape(R, 9 * C)
            if L["bias"]:
                yield gf.sum(axis=2).reshape(R, C)
        elif L["kind"] == "scale":
            h = rec[li]["h"]                               # [N, C] or [N, H, W, C]
            C = L["out"]
            g = G[li].reshape(N, len(outputs), -1, C)      # pixels (if any) on axis 2
            # dz[p, c] / dw[c'] = delta_{c c'} h[p, c], shared by every pixel p
            J = (g * h.reshape(N, 1, -1, C)).sum(axis=2)
            yield J.reshape(R, C)
            if L["bias"]:
                yield g.sum(axis=2).reshape(R, C)


def jacobian(spec, params, X, outputs=None, layer_storage="fp64"):
    """Full per-sample Jacobian df/dtheta: [N, Os, P] float64 (tiny nets only)."""
    N = np.asarray(X).shape[0]
    O = spec["layers"][-1]["out"]
    Os = O if outputs is None else len(list(outputs))
    blocks = list(jacobian_blocks(spec, params, X, outputs, max_block_bytes=1 << 62,
                                  layer_storage=layer_storage))
    return np.concatenate(blocks, axis=1).reshape(N, Os, -1)


def ntk_jc_with_norms(spec, params, X1, X2, outputs1=None, outputs2=None,
                      max_block_bytes=256 << 20, layer_storage="fp64"):
    """Theta [N1, N2, Os1, Os2] plus squared Jacobian row norms [N1, Os1], [N2, Os2].

    The row norms give Theta(x1, x1)[o, o] and Theta(x2, x2)[o, o], the natural
    error scale of each entry.  Rows of a sample subset are exact: the NTK of
    a sub-batch is the corresponding sub-block of the NTK of the batch, and the
    NTK of a subset of outputs is the corresponding sub-block too.
    """
    O = spec["layers"][-1]["out"]
    o1 = list(range(O)) if outputs1 is None else list(outputs1)
    o2 = list(range(O)) if outputs2 is None else list(outputs2)
    N1, N2 = np.asarray(X1).shape[0], np.asarray(X2).shape[0]
    theta = np.zeros((N1 * len(o1), N2 * len(o2)))
    sq1 = np.zeros(N1 * len(o1))
    sq2 = np.zeros(N2 * len(o2))
    rows = max(N1 * len(o1), N2 * len(o2))
    it1 = jacobian_blocks(spec, params, X1, o1, max_block_bytes, rows, layer_storage)
    it2 = jacobian_blocks(spec, params, X2, o2, max_block_bytes, rows, layer_storage)
    for J1, J2 in zip(it1, it2):
        theta += J1 @ J2.T
        sq1 += np.einsum("rp,rp->r", J1, J1)
        sq2 += np.einsum("rp,rp->r", J2, J2)
    theta = theta.reshape(N1, len(o1), N2, len(o2)).transpose(0, 2, 1, 3)
    return np.ascontiguousarray(theta), sq1.reshape(N1, len(o1)), sq2.reshape(N2, len(o2))


def ntk_jc(spec, params, X1, X2, outputs1=None, outputs2=None, max_block_bytes=256 << 20,
           layer_storage="fp64"):
    """Theta(X1, X2) as [N1, N2, Os1, Os2] float64 by Jacobian contraction."""
    return ntk_jc_with_norms(spec, params, X1, X2, outputs1, outputs2, max_block_bytes,
                             layer_storage)[0]
