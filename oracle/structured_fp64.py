"""Secondary fp64 reference for fully-connected nets.  TEST INFRASTRUCTURE ONLY.

Evaluates the per-layer formula of the paper's Section 4.1 (FCN, "structured
derivatives"): for a dense layer y = theta x, dy/dtheta = I (kron) x^T, so the
layer's NTK summand is the scalar x1.x2 times the product of the two output
cotangent matrices (Eq. "mixed_product_example" applied in Section 4.1).  With
a bias the scalar becomes x1.x2 + 1.  The readout layer's cotangent is I_O.

This is *not* the definition: it is pinned by tests to `ntk_jc` (the plain
Jacobian contraction) on every small workload and on sample subsets of the big
ones, and then serves as the full-size fp64 reference where the Jacobian
contraction would take hours on a CPU.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf as _erf

__all__ = ["ntk_structured_fp64", "ntk_structured_diag_fp64"]


def _phi(act, z):
    return {"relu": lambda: np.maximum(z, 0.0), "erf": lambda: _erf(z),
            "none": lambda: z}[act]()


def _dphi(act, z):
    return {"relu": lambda: (z > 0.0).astype(np.float64),
            "erf": lambda: (2.0 / math.sqrt(math.pi)) * np.exp(-z * z),
            "none": lambda: np.ones_like(z)}[act]()


def _layer_inputs_and_cotangents(spec, params, X, layer_storage="fp64"):
    layers = spec["layers"]
    if any(L["kind"] != "dense" for L in layers):
        raise ValueError("ntk_structured_fp64 handles fully-connected nets only")
    ws, bs = [], []
    i = 0
    for L in layers:
        ws.append(np.asarray(params[i], np.float64))
        i += 1
        if L["bias"]:
            bs.append(np.asarray(params[i], np.float64))
            i += 1
        else:
            bs.append(None)
    h = np.asarray(X, np.float64)
    hs, zs = [], []
    for L, w, b in zip(layers, ws, bs):
        hs.append(h)
        z = h @ w.T + (0.0 if b is None else b)
        zs.append(z)
        h = _phi(L["act"], z)
        if layer_storage == "fp32":          # layer outputs stored in float32
            h = h.astype(np.float32).astype(np.float64)
        elif layer_storage != "fp64":
            raise ValueError(layer_storage)
    nl = len(layers)
    # cotangent of z_l for every output o: G_l [N, O, out_l]; G_{last} = I_O
    N = hs[0].shape[0]
    O = layers[-1]["out"]
    Gs = [None] * nl
    g = np.broadcast_to(np.eye(O), (N, O, O))
    Gs[nl - 1] = g
    for l in range(nl - 1, 0, -1):
        g = (g @ ws[l]) * _dphi(layers[l - 1]["act"], zs[l - 1])[:, None, :]
        Gs[l - 1] = g
    return hs, Gs


def ntk_structured_fp64(spec, params, X1, X2, layer_storage="fp64"):
    """Theta [N1, N2, O, O] float64 for a fully-connected spec.

    layer_storage has the meaning of `ntk_jc`'s argument of that name.
    """
    layers = spec["layers"]
    h1, G1 = _layer_inputs_and_cotangents(spec, params, X1, layer_storage)
    if X2 is X1:
        h2, G2 = h1, G1
    else:
        h2, G2 = _layer_inputs_and_cotangents(spec, params, X2, layer_storage)
    N1, N2 = h1[0].shape[0], h2[0].shape[0]
    O = layers[-1]["out"]
    theta = np.zeros((N1, N2, O, O))
    for l, L in enumerate(layers):
        gram = h1[l] @ h2[l].T + (1.0 if L["bias"] else 0.0)          # [N1, N2]
        if l == len(layers) - 1:
            theta += gram[:, :, None, None] * np.eye(O)
        else:
            a = G1[l].reshape(N1 * O, -1)
            b = G2[l].reshape(N2 * O, -1)
            cot = (a @ b.T).reshape(N1, O, N2, O).transpose(0, 2, 1, 3)
            cot *= gram[:, :, None, None]
            theta += cot
    return theta


def ntk_structured_diag_fp64(spec, params, X, layer_storage="fp64"):
    """Theta(x, x)[o, o] for every sample and output: [N, O] float64 (fully-connected spec).

    The same per-layer formula restricted to n1 = n2, o1 = o2:
    sum over hidden layers of (|h_l|^2 [+1]) |G_l[n, o, :]|^2, plus |h_L|^2 [+1].
    """
    layers = spec["layers"]
    hs, Gs = _layer_inputs_and_cotangents(spec, params, X, layer_storage)
    N = hs[0].shape[0]
    O = layers[-1]["out"]
    d = np.zeros((N, O))
    for l, L in enumerate(layers):
        sq = np.einsum("nj,nj->n", hs[l], hs[l]) + (1.0 if L["bias"] else 0.0)
        if l == len(layers) - 1:
            d += sq[:, None]
        else:
            d += sq[:, None] * np.einsum("noc,noc->no", Gs[l], Gs[l])
    return d
