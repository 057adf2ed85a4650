"""CPU-side checks of the C ABI (no GPU): the library loads, exports every symbol
include/ntk.h declares, and rejects bad descriptors/arguments before touching the GPU."""
import ctypes
import os
import re

import pytest

import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    from paper_2206_08720_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2206_08720_amd.build import build
        build()
    return _lib.load()


def _declared_symbols():
    txt = open(os.path.join(ROOT, "include", "ntk.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(ntk_[a-z_]+)\s*\(", txt)))


def test_header_declares_the_expected_entry_points():
    from paper_2206_08720_amd import _lib
    assert set(_declared_symbols()) == set(_lib.EXPORTED_SYMBOLS)


def test_library_exports_every_declared_symbol(lib):
    for name in _declared_symbols():
        assert hasattr(lib, name), name


def _init(lib, spec, n1=4, n2=4):
    from paper_2206_08720_amd import _lib
    desc, keep = _lib.model_desc(spec)
    h = ctypes.c_void_p()
    rc = lib.ntk_init(ctypes.byref(desc), n1, n2, None, ctypes.byref(h))
    return rc, h


def test_init_rejects_bad_models_before_any_device_call(lib):
    from paper_2206_08720_amd import _lib
    bad_chain = wl.fcn_spec("b", 8, [16], 3)
    bad_chain["layers"][1]["in"] = 15
    rc, h = _init(lib, bad_chain)
    assert rc == _lib.NTK_E_SHAPE and not h.value
    assert "in" in _lib.last_error()

    act_readout = wl.fcn_spec("b", 8, [16], 3)
    act_readout["layers"][-1]["act"] = "relu"
    assert _init(lib, act_readout)[0] == _lib.NTK_E_UNSUPPORTED

    # a CNN readout takes no bias
    readout_bias = wl.cnn_spec("b", (4, 4), 3, [8], 2)
    readout_bias["layers"][-1]["bias"] = True
    assert _init(lib, readout_bias)[0] == _lib.NTK_E_UNSUPPORTED

    no_gap = wl.cnn_spec("b", (4, 4), 3, [8], 2)
    del no_gap["layers"][1]
    assert _init(lib, no_gap)[0] == _lib.NTK_E_UNSUPPORTED

    assert _init(lib, wl.fcn_spec("b", 8, [16], 3), 0, 4)[0] == _lib.NTK_E_ARG

    # 64 hidden layers is the limit; 65 are refused before any device call
    assert _init(lib, wl.fcn_spec("b", 8, [4] * 65, 3))[0] == _lib.NTK_E_UNSUPPORTED
    assert "hidden layers" in _lib.last_error()

    desc = _lib.ntk_model_desc(0, None, 1, 1, 8, 3)
    h = ctypes.c_void_p()
    assert lib.ntk_init(ctypes.byref(desc), 4, 4, None, ctypes.byref(h)) == _lib.NTK_E_ARG


def test_null_handle_calls(lib):
    from paper_2206_08720_amd import _lib
    assert lib.ntk_free(None) == _lib.NTK_OK
    assert lib.ntk_compute(None, None, None, 1, None, 1, None) == _lib.NTK_E_ARG
    assert lib.ntk_set_option(None, 1, 1) == _lib.NTK_E_ARG
    assert lib.ntk_vector_product(None, None, None, 1, None, 1, None, None) == _lib.NTK_E_ARG
    assert lib.ntk_workspace_bytes(None) == 0
    assert isinstance(lib.ntk_last_error(None), bytes)


def test_diagnostics_reject_bad_arguments_before_any_device_call(lib):
    from paper_2206_08720_amd import _lib
    out = ctypes.c_double(0.0)
    assert lib.ntk_mfma_peak(2, ctypes.byref(out)) == _lib.NTK_E_ARG
    assert lib.ntk_mfma_peak(0, None) == _lib.NTK_E_ARG
    cu = ctypes.c_int(0)
    assert lib.ntk_device_info(ctypes.byref(cu), None) == _lib.NTK_E_ARG


def _struct(blocks, hw=(4, 6), c=4):
    return wl.cnn_layers_spec("s", hw, c, blocks, 3)


def test_init_validates_the_structured_layer_kinds(lib):
    from paper_2206_08720_amd import _lib
    # an average pool needs an even image, and takes no activation
    assert _init(lib, _struct([("conv3x3", 4, "relu", True), ("avgpool2",)], hw=(5, 6)))[0] == _lib.NTK_E_SHAPE
    assert "even" in _lib.last_error()
    s = _struct([("conv3x3", 4, "relu", True), ("avgpool2",)])
    s["layers"][1]["act"] = "relu"
    assert _init(lib, s)[0] == _lib.NTK_E_UNSUPPORTED
    # a second pool of a 2 x 2 image leaves 1 x 1; a third would need an even 1 x 1 image
    assert _init(lib, _struct([("scale", "none", False)] + [("avgpool2",)] * 3, hw=(4, 4)))[0] == \
        _lib.NTK_E_SHAPE
    # depthwise and scale layers keep the channel count
    s = _struct([("dwconv3x3", "relu", True)])
    s["layers"][0]["out"] = 8
    assert _init(lib, s)[0] == _lib.NTK_E_SHAPE
    s = _struct([("scale", "relu", True)])
    s["layers"][0]["in"] = 3
    assert _init(lib, s)[0] == _lib.NTK_E_SHAPE
    # at least one layer with parameters before the global pool
    assert _init(lib, _struct([("avgpool2",)]))[0] == _lib.NTK_E_UNSUPPORTED
    # spatial kinds are not accepted between dense layers
    fcn = wl.fcn_spec("f", 8, [8], 3)
    fcn["layers"].insert(1, {"kind": "scale", "in": 8, "out": 8, "act": "none", "bias": False})
    assert _init(lib, fcn)[0] == _lib.NTK_E_UNSUPPORTED


def test_init_accepts_the_structured_layer_kinds(lib):
    from paper_2206_08720_amd import _lib
    spec = _struct([("conv3x3", 4, "relu", True), ("dwconv3x3", "erf", True), ("avgpool2",),
                    ("scale", "none", True), ("conv3x3", 6, "relu", False)])
    rc, h = _init(lib, spec)
    try:
        # validation passes; without a GPU the first device call then fails
        assert rc in (_lib.NTK_OK, _lib.NTK_E_HIP), _lib.last_error()
    finally:
        if h.value:
            lib.ntk_free(h)


def test_init_refuses_sizes_past_the_32_bit_index_range(lib):
    """Every array the kernels index must hold fewer than 2^31 elements; a plan that breaks this
    is refused with NTK_E_UNSUPPORTED before any HIP call (so here, without a GPU, the code is
    not NTK_E_HIP), and the message names the array."""
    from paper_2206_08720_amd import _lib
    # theta [n1, n2, O, O] alone: 2^16 x 2^16 samples x 10 x 10 outputs
    assert _init(lib, wl.fcn_spec("f", 8, [16], 10), 1 << 16, 1 << 16)[0] == _lib.NTK_E_UNSUPPORTED
    assert "theta" in _lib.last_error() and "2^31" in _lib.last_error()
    # a small theta (256 x 256 x 100 x 100), but the cotangents of a wide layer:
    # (n1 + n2) * O * width = 512 * 100 * 65536
    rc, _ = _init(lib, wl.fcn_spec("f", 64, [65536], 100), 256, 256)
    assert rc == _lib.NTK_E_UNSUPPORTED and "cotangents" in _lib.last_error()
    # 8192 images, O = 100, 64 x 64 pixels, 8 channels: 3.4e9 cotangent rows, 2.7e10 cotangent
    # elements (and a theta of 1.7e11 elements)
    rc, _ = _init(lib, wl.cnn_spec("c", (64, 64), 3, [8], 100), 4096, 4096)
    assert rc == _lib.NTK_E_UNSUPPORTED and "would hold" in _lib.last_error()
    # a small theta, but the conv cotangents [(n1 + n2) O, 256, 256, 64] = 2.1e10 elements
    rc, _ = _init(lib, wl.cnn_spec("c", (256, 256), 3, [64], 10), 256, 256)
    assert rc == _lib.NTK_E_UNSUPPORTED and "cotangents" in _lib.last_error()
    # the outside-in weight-space columns J [(n1 + n2) O, 9 Cin Cout]: 512-channel layers
    rc, _ = _init(lib, wl.cnn_spec("c", (4, 4), 3, [512, 512], 10), 512, 512)
    assert rc == _lib.NTK_E_UNSUPPORTED and "J" in _lib.last_error()
    # saturating arithmetic: dimensions near 2^31 each do not wrap into a small product
    huge = wl.cnn_spec("c", (1 << 15, 1 << 15), 1 << 15, [1 << 15], 1 << 15)
    assert _init(lib, huge, 1 << 30, 1 << 30)[0] == _lib.NTK_E_UNSUPPORTED
    # n1 + n2 itself past 2^31
    assert _init(lib, wl.fcn_spec("f", 1, [1], 1), (1 << 31) - 1, (1 << 31) - 1)[0] == \
        _lib.NTK_E_UNSUPPORTED


def test_init_accepts_the_largest_workloads(lib):
    """The benchmarked shapes stay inside the range: validation passes, and without a GPU the
    first device call then fails with NTK_E_HIP (or succeeds on a GPU host)."""
    from paper_2206_08720_amd import _lib
    for name in ("relu_mlp_d8_w2048", "erf_mlp_d3_w4096", "cnn4_c64_32x32", "cnn_struct_c64_32x32"):
        w = wl.WORKLOADS[name]
        rc, h = _init(lib, w["spec"], w["n1"], w["n2"])
        try:
            assert rc in (_lib.NTK_OK, _lib.NTK_E_HIP), (name, _lib.last_error())
        finally:
            if h.value:
                lib.ntk_free(h)


def _static(lib, spec, n1, n2):
    """ntk_compute_static with dummy non-null device pointers: every check it makes before the
    first HIP call runs, and nothing is dereferenced on the host.  Only for calls that fail
    before any kernel launch, or on hosts without a GPU: on a GPU the dummy addresses would be
    read by the kernels."""
    from paper_2206_08720_amd import _lib
    desc, keep = _lib.model_desc(spec)
    nparams = len(wl.param_shapes(spec))
    ptrs = (ctypes.c_void_p * nparams)(*([256] * nparams))
    dummy = ctypes.c_void_p(256)
    return lib.ntk_compute_static(ctypes.byref(desc), ptrs, dummy, n1, dummy, n2, dummy, None)


def test_static_entry_checks_before_any_device_call(lib):
    """The entry point that allocates nothing refuses, before any HIP call, null pointers,
    malformed models and workspaces beyond its fixed scratch (naming the bytes needed); shapes
    that fit get as far as the first device call (NTK_E_HIP without a GPU)."""
    from paper_2206_08720_amd import _lib
    desc, keep = _lib.model_desc(wl.fcn_spec("f", 8, [16], 3))
    assert lib.ntk_compute_static(ctypes.byref(desc), None, None, 1, None, 1, None, None) == _lib.NTK_E_ARG
    bad = wl.fcn_spec("b", 8, [16], 3)
    bad["layers"][1]["in"] = 15
    assert _static(lib, bad, 4, 4) == _lib.NTK_E_SHAPE
    # the depth-8 width-2048 FCN at 512 + 512 samples needs ~0.9 GB: refused, with the size
    big = wl.WORKLOADS["relu_mlp_d8_w2048"]["spec"]
    assert _static(lib, big, 512, 512) == _lib.NTK_E_UNSUPPORTED
    msg = _lib.last_error()
    assert "static scratch" in msg and str(_lib.STATIC_SCRATCH_BYTES) in msg
    # Shapes that fit pass every check and reach the first device call, which fails without a
    # GPU.  Where a GPU is visible the dummy addresses would reach the kernels, so this part runs
    # only on hosts without one (counting devices does not initialise the runtime).
    import torch
    if torch.cuda.device_count() > 0:
        return
    for name in ("tiny_relu_mlp", "relu_mlp_d4_w512"):
        w = wl.WORKLOADS[name]
        assert _static(lib, w["spec"], w["n1"], w["n2"]) == _lib.NTK_E_HIP, _lib.last_error()
