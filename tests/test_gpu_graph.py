"""NTK_OPT_GRAPH: ntk_compute recorded into a HIP graph and replayed (needs an MI355X).

Every replay must give the eager result bit for bit, also with the program's own eager work
and synchronisations between replays, after the input buffers' contents change (same
pointers), and after a change of arguments (a new recording).
"""
import numpy as np
import pytest

import workloads as wl
from tests.gpu_helpers import to_dev

pytestmark = pytest.mark.gpu

CASES = [
    ("tiny relu mlp with biases", wl.fcn_spec("g1", 16, [32, 32], 4, bias=True), 8, 8, {}),
    ("relu mlp, symmetric", wl.fcn_spec("g2", 64, [96, 96], 10), 40, None, {}),
    ("cnn, both orders", wl.cnn_spec("g3", (4, 4), 3, [16, 16], 6), 6, 5, {}),
    ("trace over outputs", wl.fcn_spec("g4", 24, [40, 40], 5), 9, 7, {"output": "trace"}),
    ("batch diagonal", wl.fcn_spec("g5", 24, [40, 40], 5), 9, 9, {"batch": "diagonal"}),
    ("Jacobian contraction", wl.fcn_spec("g6", 12, [20], 3, bias=True), 5, 4, {"method": "jacobian"}),
    # the full depth-8 width-2048 shape: second stream (transposes, Grams, half of the
    # backward's rows), stream-K contraction, direct-to-LDS loops
    ("depth 8, width 2048, 512 + 512 samples", wl.fcn_spec("g7", 3072, [2048] * 8, 10), 512, 512, {}),
    ("4 conv layers of 64 channels, 64 + 64 images", wl.cnn_spec("g8", (32, 32), 3, [64] * 4, 10), 64, 64, {}),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_graph_replays_match_eager(case):
    import torch
    from paper_2206_08720_amd import _lib
    from paper_2206_08720_amd.ntk import NTK
    label, spec, n1, n2, opts = case
    params = to_dev(wl.make_params(spec, 3100 + n1, "2/fan_in", bias_var=0.1))
    X1 = to_dev([wl.make_inputs(spec, n1, 3200 + n1)])[0]
    X2 = X1 if n2 is None else to_dev([wl.make_inputs(spec, n2, 3300 + n2)])[0]
    h = NTK(spec, n1, X2.shape[0])
    try:
        h.set_variant(opts.get("output", "full"), opts.get("batch", "full"))
        h.set_method(opts.get("method", "structured"))
        eager = h.compute(params, X1, X2).clone()
        torch.cuda.synchronize()
        h.set_option(_lib.NTK_OPT_GRAPH, 1)
        out = torch.empty_like(eager)
        for rep in range(4):
            out.fill_(float("nan"))                        # eager work between replays
            h.compute(params, X1, X2, out=out)
            torch.cuda.synchronize()
            assert torch.equal(out, eager), f"{label}: replay {rep} differs from the eager result"
        # same pointers, new contents: the replay reads the current values
        X1.mul_(0.5)
        h.set_option(_lib.NTK_OPT_GRAPH, 0)
        eager2 = h.compute(params, X1, X2).clone()
        h.set_option(_lib.NTK_OPT_GRAPH, 1)
        h.compute(params, X1, X2, out=out)                 # records again (option was reset)
        h.compute(params, X1, X2, out=out)                 # replay
        torch.cuda.synchronize()
        assert torch.equal(out, eager2)
        # a different output buffer: a new recording
        out2 = torch.empty_like(eager)
        h.compute(params, X1, X2, out=out2)
        torch.cuda.synchronize()
        assert torch.equal(out2, eager2)
    finally:
        h.close()
