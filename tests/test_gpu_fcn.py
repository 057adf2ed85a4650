"""GPU parity of the fully-connected path against the fp64 oracle (needs an MI355X).

Every case calls the HIP library through its C ABI (via the thin binding) and
compares element by element with the Jacobian-contraction oracle on the same
seeded float32 inputs, to the 1e-4 relative bar (see tests/gpu_helpers.py for
the two error measures).  At the full sizes of the two large workloads the
whole output is compared with the fp64 structured reference (itself pinned to
the oracle), and sampled rows/outputs with the oracle directly.

The references store layer outputs in float32 (layer_storage="fp32"), the
precision the GPU stores them in, so that ReLU decisions on pre-activations
within rounding distance of zero are taken on the same values on both sides
(the GPU accumulates pre-activations in fp64 for that decision).
"""
import json
import os

import numpy as np
import pytest

import oracle
import workloads as wl
from tests.gpu_helpers import TOL, diag_norms, errors, gpu_ntk, report

pytestmark = pytest.mark.gpu
S = "fp32"   # layer storage of the references


def _vs_jc(name, spec, params, X1, X2, symmetric=True):
    got = gpu_ntk(spec, params, X1, X2, symmetric=symmetric)
    ref, d1, d2 = oracle.ntk_jc_with_norms(spec, params, X1, X2, layer_storage=S)
    cs, nw = errors(got, ref, d1, d2)
    report(name, cs, nw)
    assert got.shape == ref.shape
    assert cs <= TOL and nw <= TOL
    return got


@pytest.mark.parametrize("fname", ["fcn_hand_relu.json", "fcn_hand_relu_bias.json"])
def test_hand_worked_golden_on_gpu(golden_dir, fname):
    d = json.load(open(os.path.join(golden_dir, fname)))
    params = [np.array(p, dtype=np.float32) for p in d["params"]]
    X = np.array(d["X"], dtype=np.float32)
    for sym in (True, False):
        got = gpu_ntk(d["spec"], params, X, X, symmetric=sym)
        np.testing.assert_allclose(got, np.array(d["theta"]), rtol=1e-6, atol=1e-6)


def test_tiny_relu_mlp_full():
    spec, params, X1, X2 = wl.make_workload("tiny_relu_mlp")
    _vs_jc("tiny_relu_mlp", spec, params, X1, X2)


@pytest.mark.parametrize("symmetric", [True, False])
def test_relu_mlp_d4_w512_full(symmetric):
    spec, params, X1, X2 = wl.make_workload("relu_mlp_d4_w512")
    assert X2 is X1
    got = gpu_ntk(spec, params, X1, X2, symmetric=symmetric)
    ref = oracle.ntk_structured_fp64(spec, params, X1, X2, layer_storage=S)
    d = oracle.ntk_structured_diag_fp64(spec, params, X1, layer_storage=S)
    cs, nw = errors(got, ref, d, d)
    report(f"relu_mlp_d4_w512 sym={symmetric} vs structured fp64", cs, nw)
    assert cs <= TOL and nw <= TOL
    # sampled rows against the definition itself
    rows = [0, 1, 63, 64, 127]
    sub, s1, s2 = oracle.ntk_jc_with_norms(spec, params, X1[rows], X1[rows], layer_storage=S)
    cs, nw = errors(got[np.ix_(rows, rows)], sub, s1, s2)
    report(f"relu_mlp_d4_w512 sym={symmetric} rows vs JC", cs, nw)
    assert cs <= TOL and nw <= TOL


@pytest.mark.parametrize("name,rows1,rows2,outs", [
    ("relu_mlp_d8_w2048", [0, 300, 511], [0, 127, 511], [0, 4, 9]),
    ("erf_mlp_d3_w4096", [0, 77, 127], [1, 64, 127], [0, 57, 99]),
])
def test_large_fcn_full_size(name, rows1, rows2, outs):
    spec, params, X1, X2 = wl.make_workload(name)
    got = gpu_ntk(spec, params, X1, X2)
    print(f"[parity] {name}: GPU done, computing fp64 references", flush=True)
    ref = oracle.ntk_structured_fp64(spec, params, X1, X2, layer_storage=S)
    d1 = oracle.ntk_structured_diag_fp64(spec, params, X1, layer_storage=S)
    d2 = oracle.ntk_structured_diag_fp64(spec, params, X2, layer_storage=S)
    cs, nw = errors(got, ref, d1, d2)
    report(f"{name} full vs structured fp64", cs, nw)
    assert cs <= TOL and nw <= TOL
    del ref
    sub, s1, s2 = oracle.ntk_jc_with_norms(spec, params, X1[rows1], X2[rows2], outs, outs,
                                           layer_storage=S)
    cs, nw = errors(got[np.ix_(rows1, rows2, outs, outs)], sub, s1, s2)
    report(f"{name} sampled entries vs JC", cs, nw)
    assert cs <= TOL and nw <= TOL
    # the stored block of the Jacobian contraction itself (tests/golden/make_jc_blocks.py): every
    # output, samples spread over the batches (for the depth-8 network one in every 128-row
    # tile of the contraction's rows (n, o))
    blk = np.load(os.path.join(os.path.dirname(__file__), "golden", f"jc_block_{name}.npz"))
    r1, r2 = blk["rows1"], blk["rows2"]
    cs, nw = errors(got[np.ix_(r1, r2)], blk["theta"].astype(np.float64), blk["sq1"].astype(np.float64),
                    blk["sq2"].astype(np.float64))
    report(f"{name} {len(r1)} x {len(r2)} samples, all outputs, vs stored JC block", cs, nw)
    assert cs <= TOL and nw <= TOL


EDGE = [
    # (label, spec, n1, n2, weight_var)
    ("n1=n2=1", wl.fcn_spec("e1", 16, [32, 32], 4, bias=True), 1, 1),
    ("ragged 3x70 O=7", wl.fcn_spec("e2", 20, [48, 24], 7, act="erf"), 3, 70),
    ("O=1", wl.fcn_spec("e3", 10, [33, 65], 1), 17, 9),
    ("widths not multiple of 4, bias", wl.fcn_spec("e4", 13, [37, 19, 41], 7, bias=True), 29, 41),
    ("single readout layer, bias", wl.fcn_spec("e5", 9, [], 3, bias=True), 5, 6),
    ("two linear layers", wl.fcn_spec("e6", 6, [11], 5, act="none"), 7, 4),
    ("input size 3 (paper's FCN inputs), deep", wl.fcn_spec("e7", 3, [64] * 9, 10), 12, 12),
    ("tile-spanning R=N*O, erf", wl.fcn_spec("e8", 64, [96, 96], 10, act="erf"), 29, 41),
    ("64 hidden layers (the maximum)", wl.fcn_spec("e9", 8, [16] * 64, 3, bias=True), 6, 5),
    ("one hidden layer of width 8192", wl.fcn_spec("e10", 16, [8192], 10), 8, 7),
    ("O=128 outputs", wl.fcn_spec("e11", 12, [40], 128, act="erf"), 6, 4),
    # more 64 x 64 Gram tiles than CUs: the first backward layer and the Grams in two launches
    ("Grams past the 16x16-block form, 700 x 700", wl.fcn_spec("e12", 24, [64, 64], 2, bias=True), 700, 700),
]


@pytest.mark.parametrize("case", EDGE, ids=[c[0] for c in EDGE])
def test_edge_shapes(case):
    label, spec, n1, n2 = case
    params = wl.make_params(spec, 500 + n1, bias_var=0.2)
    X1 = wl.make_inputs(spec, n1, 600 + n1)
    X2 = wl.make_inputs(spec, n2, 700 + n2)
    _vs_jc(label, spec, params, X1, X2)


def test_unaligned_parameters_and_inputs():
    """Weights, biases and inputs at 4-byte (not 16-byte) aligned addresses: the backward then
    reads per-call transposed weights instead of W itself, and the forward and the Grams take
    their scalar-load forms; Theta still matches the Jacobian contraction."""
    import torch
    from paper_2206_08720_amd.ntk import NTK
    spec = wl.fcn_spec("unal", 32, [64, 64, 64], 5, act="relu", bias=True)
    params = wl.make_params(spec, 41, bias_var=0.2)
    X1 = wl.make_inputs(spec, 40, 42)
    X2 = wl.make_inputs(spec, 33, 43)

    def shifted(a):   # a contiguous view one float past a 256-byte aligned allocation
        buf = torch.empty(a.size + 1, dtype=torch.float32, device="cuda")
        v = buf[1:].view(a.shape)
        v.copy_(torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)))
        assert v.data_ptr() % 16 == 4
        return v

    h = NTK(spec, 40, 40)
    try:
        out = h.compute([shifted(p) for p in params], shifted(X1), shifted(X2))
        torch.cuda.synchronize()
        got = out.cpu().numpy()
    finally:
        h.close()
    ref, d1, d2 = oracle.ntk_jc_with_norms(spec, params, X1, X2, layer_storage=S)
    cs, nw = errors(got, ref, d1, d2)
    report("unaligned parameters and inputs", cs, nw)
    assert cs <= TOL and nw <= TOL


@pytest.mark.parametrize("symmetric", [True, False])
def test_aliased_inputs(symmetric):
    spec = wl.fcn_spec("alias", 30, [70, 50], 6, act="relu", bias=True)
    params = wl.make_params(spec, 801, bias_var=0.2)
    X = wl.make_inputs(spec, 45, 802)
    got = _vs_jc(f"aliased sym={symmetric}", spec, params, X, X, symmetric=symmetric)
    # Theta(X, X) is symmetric as an NO x NO matrix
    N, O = got.shape[0], got.shape[2]
    M = got.transpose(0, 2, 1, 3).reshape(N * O, N * O)
    np.testing.assert_allclose(M, M.T, rtol=0, atol=1e-5 * np.abs(M).max())


def test_handle_reuse_with_smaller_batches_and_determinism():
    from paper_2206_08720_amd.ntk import NTK
    spec = wl.fcn_spec("reuse", 24, [40, 40], 5, act="erf", bias=True)
    params = wl.make_params(spec, 901, bias_var=0.2)
    X1 = wl.make_inputs(spec, 33, 902)
    X2 = wl.make_inputs(spec, 21, 903)
    h = NTK(spec, 40, 40)
    try:
        a = gpu_ntk(spec, params, X1, X2, handle=h)
        b = gpu_ntk(spec, params, X1, X2, handle=h)
        assert np.array_equal(a, b), "two calls must be bit-identical"
        c = gpu_ntk(spec, params, X1[:5], X2[:7], handle=h)
        ref, d1, d2 = oracle.ntk_jc_with_norms(spec, params, X1[:5], X2[:7], layer_storage=S)
        cs, nw = errors(c, ref, d1, d2)
        assert cs <= TOL and nw <= TOL
    finally:
        h.close()


def test_argument_errors_leave_output_untouched():
    import torch
    from paper_2206_08720_amd import _lib
    from paper_2206_08720_amd.ntk import NTK
    from tests.gpu_helpers import to_dev
    spec = wl.fcn_spec("err", 8, [16], 3)
    params = to_dev(wl.make_params(spec, 1))
    X = to_dev([wl.make_inputs(spec, 6, 2)])[0]
    h = NTK(spec, 4, 4)
    try:
        out = torch.full((6, 6, 3, 3), 7.0, device="cuda")
        with pytest.raises(_lib.NTKError) as ei:
            h.compute(params, X, X, out=out)          # n = 6 > max 4
        assert ei.value.code == _lib.NTK_E_ARG
        torch.cuda.synchronize()
        assert bool((out == 7.0).all())
    finally:
        h.close()


# ---- stream-K schedule of the contraction (used once the output has at least as many 128 x 128
# tiles as persistent workgroups: two per compute unit, 512 on the 256 CUs of an MI355X) ----
SK_CASES = [
    # label, spec, n1, n2, X2 is X1
    # symmetric: 23 x 23 tiles -> 276 triangle tiles x 8 layers over 512 ranges, so a tile
    # spans about 2 ranges
    ("tiles over 2-3 ranges, 8 hidden layers, symmetric", wl.fcn_spec("sk1", 24, [64] * 8, 10), 290, 290, True),
    ("split tiles, 2 hidden layers, symmetric", wl.fcn_spec("sk1b", 24, [64, 64], 10), 300, 300, True),
    # one hidden layer: a unit is a whole tile (no splits); 276 units over 512 ranges leaves
    # empty ranges
    ("one hidden layer, symmetric, empty ranges", wl.fcn_spec("sk2", 16, [24], 10, bias=True),
     290, 290, True),
    ("ragged R1 != R2, 3 layers", wl.fcn_spec("sk3", 20, [48, 40], 8, act="erf", bias=True), 420, 310, False),
    ("8 hidden layers, R1 != R2", wl.fcn_spec("sk4", 12, [32] * 8, 9), 330, 301, False),
]


@pytest.mark.parametrize("case", SK_CASES, ids=[c[0] for c in SK_CASES])
def test_stream_k_contraction(case):
    label, spec, n1, n2, alias = case
    params = wl.make_params(spec, 900 + n1, bias_var=0.2)
    X1 = wl.make_inputs(spec, n1, 910 + n1)
    X2 = X1 if alias else wl.make_inputs(spec, n2, 920 + n2)
    O = spec["layers"][-1]["out"]
    assert -(-n1 * O // 128) * -(-n2 * O // 128) >= 512, "case must take the stream-K path"
    got = _vs_jc(f"stream-K {label}", spec, params, X1, X2)
    if alias:
        N = got.shape[0]
        M = got.transpose(0, 2, 1, 3).reshape(N * O, N * O)
        np.testing.assert_allclose(M, M.T, rtol=0, atol=1e-5 * np.abs(M).max())


def test_width_2048_with_a_partial_last_round_of_backward_tiles():
    # 480 stacked samples x O = 10 -> 38 x 16 = 608 backward tiles of 128 x 128, a partial
    # second round over the 512 slots of two workgroups per CU
    spec = wl.fcn_spec("bwsk", 64, [2048, 2048], 10)
    params = wl.make_params(spec, 61, "2/fan_in")
    X1 = wl.make_inputs(spec, 250, 62)
    X2 = wl.make_inputs(spec, 230, 63)
    got = gpu_ntk(spec, params, X1, X2)
    ref = oracle.ntk_structured_fp64(spec, params, X1, X2, layer_storage=S)
    d1 = oracle.ntk_structured_diag_fp64(spec, params, X1, layer_storage=S)
    d2 = oracle.ntk_structured_diag_fp64(spec, params, X2, layer_storage=S)
    cs, nw = errors(got, ref, d1, d2)
    report("width 2048, partial last backward round, vs structured fp64", cs, nw)
    assert cs <= TOL and nw <= TOL
    # the structured reference itself against the Jacobian contraction on a few rows
    sub = [0, 117, 249]
    jc, e1, e2 = oracle.ntk_jc_with_norms(spec, params, X1[sub], X2[[0, 229]], layer_storage=S)
    cs, nw = errors(got[np.ix_(sub, [0, 229])], jc, e1, e2)
    assert cs <= TOL and nw <= TOL


def test_backward_split_over_two_streams_with_an_odd_batch():
    # 411 + 412 stacked samples: each half (411 and 412 samples x O = 10 rows) still has
    # 33 x 16 = 528 >= 2 x 256 backward tiles, so the two halves of the backward run on the
    # two streams; the odd total puts the boundary inside no sample
    spec = wl.fcn_spec("bwsplit", 64, [2048, 2048, 2048], 10)
    params = wl.make_params(spec, 71, "2/fan_in")
    X1 = wl.make_inputs(spec, 411, 72)
    X2 = wl.make_inputs(spec, 412, 73)
    got = gpu_ntk(spec, params, X1, X2)
    print("[parity] split backward: GPU done, computing fp64 references", flush=True)
    ref = oracle.ntk_structured_fp64(spec, params, X1, X2, layer_storage=S)
    d1 = oracle.ntk_structured_diag_fp64(spec, params, X1, layer_storage=S)
    d2 = oracle.ntk_structured_diag_fp64(spec, params, X2, layer_storage=S)
    cs, nw = errors(got, ref, d1, d2)
    report("backward split over two streams, vs structured fp64", cs, nw)
    assert cs <= TOL and nw <= TOL
    # rows on both sides of the split (stacked sample 411 = X2[0]) against the definition
    jc, e1, e2 = oracle.ntk_jc_with_norms(spec, params, X1[[0, 410]], X2[[0, 1, 411]], layer_storage=S)
    cs, nw = errors(got[np.ix_([0, 410], [0, 1, 411])], jc, e1, e2)
    assert cs <= TOL and nw <= TOL


def test_sample_halves_schedule_matches_one_stream_bit_for_bit():
    # 512 + 512 samples of a width-2048 FCN: the forward, seed and backward run as two sample
    # halves on the two streams (each half still makes 8 x 32 forward tiles, no split-K, and
    # 40 x 16 backward tiles); with per-kernel profiling on, the forward runs on one stream.  Every
    # row's sums keep their order either way, so the two Theta are equal bit for bit.
    spec = wl.fcn_spec("halves", 64, [2048, 2048], 10)
    params = wl.make_params(spec, 81, "2/fan_in")
    X1 = wl.make_inputs(spec, 512, 82)
    X2 = wl.make_inputs(spec, 512, 83)
    got = gpu_ntk(spec, params, X1, X2)
    prof = {}
    one_stream = gpu_ntk(spec, params, X1, X2, profile=prof)
    assert "dense_fwd" in prof
    assert np.array_equal(got, one_stream)
    sub1, sub2 = [0, 255, 511], [0, 256, 511]
    jc, e1, e2 = oracle.ntk_jc_with_norms(spec, params, X1[sub1], X2[sub2], layer_storage=S)
    cs, nw = errors(got[np.ix_(sub1, sub2)], jc, e1, e2)
    report("sample-halves schedule, sampled rows vs JC", cs, nw)
    assert cs <= TOL and nw <= TOL
