"""fp64 CPU oracle for the empirical finite-width NTK.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this package.  The GPU library never calls it, and it shares no code with the
GPU library (the only shared module is the seeded input generator `workloads`,
which holds no NTK arithmetic).

Contents
--------
* `ntk_jc` -- the plain definition: Theta = J(x1) J(x2)^T (the paper's Eq.
  "ntk_outer_product" / Eq. "ntk_def_main", Section 3.1.1), computed the
  baseline way of Section 3.2 ("Jacobian contraction"): explicit per-sample
  Jacobian blocks from the reverse-mode Jacobian (O vector-Jacobian products on
  rows of I_O, Section 3.1.3), contracted block by block in float64.
* `jacobian` -- the full per-sample Jacobian [N, O, P] for tiny nets.
* `forward` -- the network function f(theta, x) itself.
* `ntk_jc_variant` -- the output-trace, single-logit and batch-diagonal parts of
  Theta, contracted directly from the Jacobian rows they need (appendix
  "Pseudo-NTK").
* `ntk_vp` -- the NTK-vector product Theta(X1, X2) v = J(x1) (J(x2)^T v)
  (Section 3.3), from the explicit Jacobian blocks.
* `ntk_structured_fp64` -- a secondary fp64 reference for fully-connected nets
  that evaluates the per-layer formula of Section 4.1 (input Gram times
  cotangent Gram, summed over layers).  It is not the definition: the tests pin
  it to `ntk_jc` and it only serves full-size coverage where the Jacobian
  contraction is too expensive on a CPU.

Parity status: every function here is pinned by tests under `tests/` against
torch autograd Jacobians (an independent library), central finite
differences, closed forms, hand-worked examples (`tests/golden/`), symmetry,
positive semi-definiteness and homogeneity.
"""
from .ntk_jc import forward, jacobian, ntk_jc, ntk_jc_with_norms, param_count
from .structured_fp64 import ntk_structured_diag_fp64, ntk_structured_fp64
from .variants import ntk_jc_variant
from .vector_product import ntk_vp

__all__ = ["forward", "jacobian", "ntk_jc", "ntk_jc_with_norms", "param_count",
           "ntk_structured_fp64", "ntk_structured_diag_fp64", "ntk_jc_variant", "ntk_vp"]
