"""Output- and batch-axis variants of the empirical NTK, by Jacobian contraction in float64.
TEST INFRASTRUCTURE ONLY.

The paper's applications often use a part of Theta (appendix "Pseudo-NTK"; the batch
diagonal Theta(x, x)); compute-wise these are the NTK with a single output.  Each variant is
computed here directly from the explicit per-sample Jacobian rows, contracting only what the
variant keeps (not by slicing the full Theta):

* output "trace":  sum_o J(x1)[o] . J(x2)[o]                        [N1, N2]
* output "logit":  J(x1)[o*] . J(x2)[o*] (the NTK of output o* alone)   [N1, N2]
* batch "diagonal": the pairs (x1_n, x2_n) only, N1 == N2              [N, ...]

Alongside Theta it returns the error scale of every entry, the product of the Jacobian
norms of the two sides (Cauchy-Schwarz): |Theta| never exceeds it.
"""
from __future__ import annotations

import numpy as np

from .ntk_jc import jacobian_blocks

__all__ = ["ntk_jc_variant"]


def ntk_jc_variant(spec, params, X1, X2, output="full", batch="full", logit=0,
                   max_block_bytes=256 << 20, layer_storage="fp64"):
    """Theta's variant and its per-entry error scale, both float64.

    Shapes: full/full [N1,N2,O,O]; trace or logit/full [N1,N2]; full/diagonal [N,O,O];
    trace or logit/diagonal [N].
    """
    if output not in ("full", "trace", "logit") or batch not in ("full", "diagonal"):
        raise ValueError("output is full|trace|logit, batch is full|diagonal")
    O = spec["layers"][-1]["out"]
    outs = [int(logit)] if output == "logit" else list(range(O))
    Os = len(outs)
    N1, N2 = np.asarray(X1).shape[0], np.asarray(X2).shape[0]
    if batch == "diagonal" and N1 != N2:
        raise ValueError("the batch diagonal needs N1 == N2")
    rows = max(N1, N2) * Os
    it1 = jacobian_blocks(spec, params, X1, outs, max_block_bytes, rows, layer_storage)
    it2 = jacobian_blocks(spec, params, X2, outs, max_block_bytes, rows, layer_storage)
    keep_o = output == "full"
    if batch == "full":
        theta = np.zeros((N1 * Os, N2 * Os) if keep_o else (N1, N2))
    else:
        theta = np.zeros((N1, Os, Os) if keep_o else (N1,))
    sq1 = np.zeros((N1, Os))
    sq2 = np.zeros((N2, Os))
    for J1, J2 in zip(it1, it2):
        A = J1.reshape(N1, Os, -1)
        B = J2.reshape(N2, Os, -1)
        sq1 += np.einsum("nop,nop->no", A, A)
        sq2 += np.einsum("nop,nop->no", B, B)
        if batch == "full" and keep_o:
            theta += J1 @ J2.T
        elif batch == "full":
            # rows (n) of all kept outputs' columns: sum_o J1[n1, o] . J2[n2, o]
            theta += A.reshape(N1, -1) @ B.reshape(N2, -1).T
        elif keep_o:
            theta += np.einsum("nop,nqp->noq", A, B)
        else:
            theta += np.einsum("nop,nop->n", A, B)
    if batch == "full" and keep_o:
        theta = theta.reshape(N1, Os, N2, Os).transpose(0, 2, 1, 3)
        scale = np.sqrt(sq1[:, None, :, None] * sq2[None, :, None, :])
    elif batch == "full":
        scale = np.sqrt(sq1.sum(1)[:, None] * sq2.sum(1)[None, :])
    elif keep_o:
        scale = np.sqrt(sq1[:, :, None] * sq2[:, None, :])
    else:
        scale = np.sqrt(sq1.sum(1) * sq2.sum(1))
    return np.ascontiguousarray(theta), scale
