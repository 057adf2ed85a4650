"""NTK-vector products Theta(X1, X2) v, by explicit Jacobians in float64.
TEST INFRASTRUCTURE ONLY.

The map v in R^{N2 O} -> Theta v in R^{N1 O} (Section 3.3, Eq. "ntk_vp_main"; its use in
power iteration and conjugate gradients is discussed in the appendix on applications):  (Theta v)[n1, o1] = sum_{n2, o2} Theta[n1, n2, o1, o2] v[n2, o2]
= J(x1) (J(x2)^T v).  Here it is evaluated in that order from the explicit Jacobian blocks:
first the weight-space vector J(x2)^T v, then its product with J(x1).

Alongside it returns the error scale of every entry, ||J(x1)[n1, o1]|| ||J(x2)^T v||, which
bounds |(Theta v)[n1, o1]| (Cauchy-Schwarz).
"""
from __future__ import annotations

import numpy as np

from .ntk_jc import jacobian_blocks

__all__ = ["ntk_vp"]


def ntk_vp(spec, params, X1, X2, v, max_block_bytes=256 << 20, layer_storage="fp64"):
    """(Theta(X1, X2) v [N1, O], error scale [N1, O]) for v [N2, O], float64."""
    O = spec["layers"][-1]["out"]
    N1, N2 = np.asarray(X1).shape[0], np.asarray(X2).shape[0]
    v = np.asarray(v, dtype=np.float64).reshape(N2 * O)
    rows = max(N1, N2) * O
    it1 = jacobian_blocks(spec, params, X1, None, max_block_bytes, rows, layer_storage)
    it2 = jacobian_blocks(spec, params, X2, None, max_block_bytes, rows, layer_storage)
    out = np.zeros(N1 * O)
    sq1 = np.zeros(N1 * O)
    tc_sq = 0.0
    for J1, J2 in zip(it1, it2):
        tc = J2.T @ v                          # this block of the weight-space vector J2^T v
        out += J1 @ tc
        sq1 += np.einsum("rp,rp->r", J1, J1)
        tc_sq += float(tc @ tc)
    scale = np.sqrt(sq1 * tc_sq)
    return out.reshape(N1, O), scale.reshape(N1, O)
