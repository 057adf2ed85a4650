"""Write the direct Jacobian-contraction reference blocks of the two large fully-connected
workloads, for the GPU parity tests (tests/test_gpu_fcn.py).

    python tests/golden/make_jc_blocks.py [relu_mlp_d8_w2048] [erf_mlp_d3_w4096]

Only the oracle (`oracle.ntk_jc_with_norms`, the plain definition Theta = J(x1) J(x2)^T of
Section 3.1.1, Eq. ntk_def_main, contracted block by block in fp64) and the seeded workload
generator are called.  A block Theta(X1[R1], X2[R2]) is exactly the block [R1, R2] of the full
Theta, so each file holds one block with every output:

* relu_mlp_d8_w2048: 64 + 64 samples, spread so that rows n = 0 and n = 511 are included and
  every 128-row tile of the contraction's rows (n, o) of each batch holds at least one of them
  (5120 rows per batch, 40 tiles);
* erf_mlp_d3_w4096: 16 + 16 samples, n = 0 and n = 127 included, all 100 outputs.

Stored with float32 values (rounding the fp64 results adds at most 6e-8 relative error, far
below the 1e-4 parity bar): theta [R1, R2, O, O], the squared Jacobian row norms sq1 [R1, O] and
sq2 [R2, O] (the Cauchy-Schwarz error scale), and the sample indices.  The fp32 layer-storage
reading is used, as by every GPU parity reference.
"""
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
import workloads as wl  # noqa: E402

BLOCKS = {"relu_mlp_d8_w2048": 64, "erf_mlp_d3_w4096": 16}


def sample_rows(n_total, k):
    """k sample indices from 0 to n_total - 1, evenly spread."""
    return sorted(set(int(round(i * (n_total - 1) / (k - 1))) for i in range(k)))


def path_of(name):
    return os.path.join(HERE, f"jc_block_{name}.npz")


def main(names):
    for name in names:
        k = BLOCKS[name]
        spec, params, X1, X2 = wl.make_workload(name)
        r1 = sample_rows(X1.shape[0], k)
        r2 = sample_rows(X2.shape[0], k)
        t0 = time.time()
        th, s1, s2 = oracle.ntk_jc_with_norms(spec, params, X1[r1], X2[r2], layer_storage="fp32")
        print(f"{name}: block {len(r1)} x {len(r2)} x {th.shape[2]} x {th.shape[3]} in "
              f"{time.time() - t0:.0f} s", flush=True)
        np.savez(path_of(name), rows1=np.array(r1, np.int32), rows2=np.array(r2, np.int32),
                 theta=th.astype(np.float32), sq1=s1.astype(np.float32), sq2=s2.astype(np.float32))


if __name__ == "__main__":
    main(sys.argv[1:] or list(BLOCKS))
