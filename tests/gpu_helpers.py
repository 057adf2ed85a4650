"""Helpers shared by the GPU parity tests: run the HIP path, compare with the oracle.

Error measures (both must be <= the tolerance):
* Cauchy-Schwarz-normalised: max |Theta_gpu - Theta_ref| / sqrt(Theta(x1,x1)[o1,o1] Theta(x2,x2)[o2,o2]),
  i.e. the error of each entry relative to the norms of the two Jacobian rows it
  is the dot product of (|Theta[n1,n2,o1,o2]| <= that product).  An elementwise
  relative error is unusable: Theta has exact zeros and many near-zero
  off-diagonal (o1 != o2) entries whose fp32 rounding error is set by the row
  norms, not by the entry.
* normwise: max |Theta_gpu - Theta_ref| / max |Theta_ref|.
"""
import sys

import numpy as np

TOL = 1e-4   # maximum relative error allowed by the fp32-vs-fp64 parity bar


def to_dev(arrs):
    import torch
    return [torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda() for a in arrs]


def gpu_ntk(spec, params, X1, X2, symmetric=True, handle=None, max_n=None, options=None,
            profile=None, variant=None):
    """Theta from the HIP library.  options: {NTK_OPT_*: value}; profile: a dict that
    receives the per-kernel-class timing of this call; variant: (output, batch, logit) for
    NTK.set_variant."""
    import torch
    from paper_2206_08720_amd import _lib
    from paper_2206_08720_amd.ntk import NTK
    ps = to_dev(params)
    x1 = to_dev([X1])[0]
    x2 = x1 if X2 is X1 else to_dev([X2])[0]
    h = handle or NTK(spec, max_n or X1.shape[0], max_n or X2.shape[0])
    h.set_option(_lib.NTK_OPT_SYMMETRIC, 1 if symmetric else 0)
    for k, v in (options or {}).items():
        h.set_option(k, v)
    h.set_variant(*(variant or ("full", "full", 0)))
    if profile is not None:
        h.profile_read()
        h.profile_enable(True)
    out = h.compute(ps, x1, x2)
    torch.cuda.synchronize()
    if profile is not None:
        profile.update(h.profile_read())
        h.profile_enable(False)
    res = out.cpu().numpy()
    if handle is None:
        h.close()
    return res


def errors(got, ref, d1, d2):
    """(cs_err, normwise_err) of got vs ref; d1 [N1,O1], d2 [N2,O2] are Theta(x,x)[o,o]."""
    diff = np.abs(got.astype(np.float64) - ref)
    scale = np.sqrt(np.maximum(d1[:, None, :, None] * d2[None, :, None, :], 1e-300))
    cs = float(np.max(diff / scale)) if diff.size else 0.0
    nw = float(np.max(diff) / max(np.max(np.abs(ref)), 1e-300)) if diff.size else 0.0
    if diff.size and cs > TOL:
        loc = np.unravel_index(np.argmax(diff / scale), diff.shape)
        print(f"[parity] worst entry at (n1, n2, o1, o2) = {tuple(int(i) for i in loc)}: "
              f"got {got[loc]!r} ref {ref[loc]!r}", flush=True)
    return cs, nw


def scaled_errors(got, ref, scale):
    """(cs_err, normwise_err) of got vs ref for any shape, with the per-entry error scale."""
    diff = np.abs(got.astype(np.float64) - ref)
    if not diff.size:
        return 0.0, 0.0
    cs = float(np.max(diff / np.maximum(scale, 1e-300)))
    nw = float(np.max(diff) / max(np.max(np.abs(ref)), 1e-300))
    if cs > TOL:
        loc = np.unravel_index(np.argmax(diff / np.maximum(scale, 1e-300)), diff.shape)
        print(f"[parity] worst entry at {tuple(int(i) for i in loc)}: got {got[loc]!r} "
              f"ref {ref[loc]!r} scale {scale[loc]!r}", flush=True)
    return cs, nw


def variant_of(full, output, batch, logit=0):
    """The variant read off a full Theta [N1, N2, O, O] (or its error scale)."""
    if batch == "diagonal":
        n = np.arange(full.shape[0])
        full = full[n, n]
    if output == "trace":
        return np.trace(full, axis1=-2, axis2=-1)
    if output == "logit":
        return full[..., logit, logit]
    return full


def variant_scale(d1, d2, output, batch, logit=0):
    """Per-entry error scale of a variant from the Jacobian row norms d1 [N1,O], d2 [N2,O]."""
    if output == "trace":
        a, b = d1.sum(1), d2.sum(1)
    elif output == "logit":
        a, b = d1[:, logit], d2[:, logit]
    else:
        a, b = d1, d2
    if batch == "diagonal":
        return np.sqrt(a[:, :, None] * b[:, None, :]) if output == "full" else np.sqrt(a * b)
    if output == "full":
        return np.sqrt(a[:, None, :, None] * b[None, :, None, :])
    return np.sqrt(a[:, None] * b[None, :])


def diag_norms(theta_xx):
    """Theta(x, x)[o, o] from a full square [N, N, O, O] block."""
    return np.einsum("nnoo->no", theta_xx)


def report(name, cs, nw):
    print(f"[parity] {name}: cs_err={cs:.3e} normwise={nw:.3e}", flush=True)
    sys.stdout.flush()
