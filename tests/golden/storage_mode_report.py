"""How much the fp32 layer-storage reading moves the oracle, on the full large FCN workloads.

    python tests/golden/storage_mode_report.py [relu_mlp_d8_w2048] [erf_mlp_d3_w4096]

Every GPU parity reference stores each layer's output in fp32 and sums the pre-activations in
fp64 (the oracle's layer_storage="fp32"; the paper's experiments use 32-bit precision).  This
script evaluates the same fp64 per-layer formula (oracle.ntk_structured_fp64, itself pinned to the
Jacobian contraction) in both storage modes on the full batches and records, per workload:
  * the number of hidden pre-activations whose ReLU decision (z > 0) differs between the modes,
    for X1 and X2 (erf networks have no decisions);
  * the Cauchy-Schwarz-normalised difference max |Theta_fp32store - Theta_fp64| /
    sqrt(Theta_fp64(x1, x1)[o1, o1] Theta_fp64(x2, x2)[o2, o2]) and the normwise one
    max |diff| / max |Theta_fp64|.
Only the oracle and the seeded workload generator are called.  Output: storage_mode_report.json
beside this script.
"""
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
import workloads as wl  # noqa: E402
from oracle.structured_fp64 import _layer_inputs_and_cotangents  # noqa: E402


def relu_decisions(spec, params, X, mode):
    hs, _ = _layer_inputs_and_cotangents(spec, params, X, mode)
    acts = [L["act"] for L in spec["layers"][:-1]]
    return [hs[l + 1] > 0.0 for l, a in enumerate(acts) if a == "relu"]


def report(name):
    spec, params, X1, X2 = wl.make_workload(name)
    t0 = time.time()
    out = {"workload": name, "n1": int(X1.shape[0]), "n2": int(X2.shape[0])}
    flips = {}
    for tag, X in (("X1", X1), ("X2", X2)):
        m32 = relu_decisions(spec, params, X, "fp32")
        m64 = relu_decisions(spec, params, X, "fp64")
        flips[tag] = {"decisions": int(sum(m.size for m in m64)),
                      "differing": int(sum(int((a != b).sum()) for a, b in zip(m32, m64)))}
    out["relu_decisions"] = flips
    t32 = oracle.ntk_structured_fp64(spec, params, X1, X2, layer_storage="fp32")
    t64 = oracle.ntk_structured_fp64(spec, params, X1, X2, layer_storage="fp64")
    d1 = oracle.ntk_structured_diag_fp64(spec, params, X1, layer_storage="fp64")
    d2 = oracle.ntk_structured_diag_fp64(spec, params, X2, layer_storage="fp64")
    diff = np.abs(t32 - t64)
    scale = np.sqrt(d1[:, None, :, None] * d2[None, :, None, :])
    cs = diff / scale
    loc = np.unravel_index(int(np.argmax(cs)), cs.shape)
    out["cs_normalised_max"] = float(cs.max())
    out["cs_normalised_worst_entry"] = [int(i) for i in loc]
    out["normwise"] = float(diff.max() / np.abs(t64).max())
    out["entries_above_1e-4_cs"] = int((cs > 1e-4).sum())
    out["seconds"] = round(time.time() - t0, 1)
    print(json.dumps(out), flush=True)
    return out


if __name__ == "__main__":
    names = sys.argv[1:] or ["relu_mlp_d8_w2048", "erf_mlp_d3_w4096"]
    res = [report(n) for n in names]
    path = os.path.join(HERE, "storage_mode_report.json")
    old = json.load(open(path)) if os.path.exists(path) else []
    keep = [r for r in old if r["workload"] not in names]
    json.dump(keep + res, open(path, "w"), indent=1)
