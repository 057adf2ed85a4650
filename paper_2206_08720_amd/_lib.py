"""ctypes binding of the C ABI in include/ntk.h (argument marshalling only).

Every computation runs in the HIP kernels of libntk.so; this module only
converts Python values to the C structs and pointers the library takes.  It
raises if the library has not been built: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libntk.so")

NTK_OK = 0
NTK_E_ARG = -1
NTK_E_SHAPE = -2
NTK_E_UNSUPPORTED = -3
NTK_E_OOM = -4
NTK_E_HIP = -5
ERROR_NAMES = {NTK_E_ARG: "NTK_E_ARG", NTK_E_SHAPE: "NTK_E_SHAPE",
               NTK_E_UNSUPPORTED: "NTK_E_UNSUPPORTED", NTK_E_OOM: "NTK_E_OOM",
               NTK_E_HIP: "NTK_E_HIP"}

NTK_DENSE, NTK_CONV3X3_SAME, NTK_GAP = 0, 1, 2
NTK_DWCONV3X3_SAME, NTK_SCALE, NTK_AVGPOOL2, NTK_CONV1X1 = 3, 4, 5, 6
NTK_ACT_NONE, NTK_ACT_RELU, NTK_ACT_ERF = 0, 1, 2
NTK_OPT_SYMMETRIC, NTK_OPT_CONV_ORDER = 1, 2
NTK_CONV_ORDER_AUTO, NTK_CONV_ORDER_OUTSIDE_IN, NTK_CONV_ORDER_INSIDE_OUT = 0, 1, 2
NTK_OPT_OUTPUT, NTK_OPT_LOGIT, NTK_OPT_BATCH = 3, 4, 5
NTK_OUTPUT_FULL, NTK_OUTPUT_TRACE, NTK_OUTPUT_LOGIT = 0, 1, 2
NTK_BATCH_FULL, NTK_BATCH_DIAGONAL = 0, 1
NTK_OPT_METHOD, NTK_METHOD_STRUCTURED, NTK_METHOD_JACOBIAN = 6, 0, 1
NTK_OPT_GRAPH = 7

EXPORTED_SYMBOLS = ("ntk_init", "ntk_compute", "ntk_free", "ntk_last_error", "ntk_set_option",
                    "ntk_set_stream", "ntk_workspace_bytes", "ntk_profile_enable",
                    "ntk_profile_read", "ntk_device_info", "ntk_mfma_peak",
                    "ntk_vector_product", "ntk_compute_static")
STATIC_SCRATCH_BYTES = 64 * 1024 * 1024   # NTK_STATIC_SCRATCH_BYTES


class ntk_layer_desc(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int), ("in_", ctypes.c_int), ("out", ctypes.c_int),
                ("act", ctypes.c_int), ("has_bias", ctypes.c_int)]


class ntk_model_desc(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int), ("layers", ctypes.POINTER(ntk_layer_desc)),
                ("in_h", ctypes.c_int), ("in_w", ctypes.c_int), ("in_c", ctypes.c_int),
                ("out_dim", ctypes.c_int)]


class NTKError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{ERROR_NAMES.get(code, code)}: {msg}")
        self.code = code


_lib = None


def load():
    """Load libntk.so (built in-tree by paper_2206_08720_amd.build); raise if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2206_08720_amd.build` (no CPU fallback exists)")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    lib.ntk_init.argtypes = [ctypes.POINTER(ntk_model_desc), ctypes.c_int, ctypes.c_int, P,
                             ctypes.POINTER(P)]
    lib.ntk_init.restype = ctypes.c_int
    lib.ntk_compute.argtypes = [P, ctypes.POINTER(P), P, ctypes.c_int, P, ctypes.c_int, P]
    lib.ntk_compute.restype = ctypes.c_int
    lib.ntk_free.argtypes = [P]
    lib.ntk_free.restype = ctypes.c_int
    lib.ntk_last_error.argtypes = [P]
    lib.ntk_last_error.restype = ctypes.c_char_p
    lib.ntk_set_option.argtypes = [P, ctypes.c_int, ctypes.c_int]
    lib.ntk_set_option.restype = ctypes.c_int
    lib.ntk_set_stream.argtypes = [P, P]
    lib.ntk_set_stream.restype = ctypes.c_int
    lib.ntk_workspace_bytes.argtypes = [P]
    lib.ntk_workspace_bytes.restype = ctypes.c_longlong
    lib.ntk_profile_enable.argtypes = [P, ctypes.c_int]
    lib.ntk_profile_enable.restype = ctypes.c_int
    lib.ntk_profile_read.argtypes = [P, ctypes.POINTER(ctypes.c_char_p),
                                     ctypes.POINTER(ctypes.c_double),
                                     ctypes.POINTER(ctypes.c_longlong), ctypes.c_int]
    lib.ntk_profile_read.restype = ctypes.c_int
    lib.ntk_vector_product.argtypes = [P, ctypes.POINTER(P), P, ctypes.c_int, P, ctypes.c_int, P, P]
    lib.ntk_vector_product.restype = ctypes.c_int
    lib.ntk_compute_static.argtypes = [ctypes.POINTER(ntk_model_desc), ctypes.POINTER(P), P, ctypes.c_int, P,
                                       ctypes.c_int, P, P]
    lib.ntk_compute_static.restype = ctypes.c_int
    lib.ntk_device_info.argtypes = [ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_int)]
    lib.ntk_device_info.restype = ctypes.c_int
    lib.ntk_mfma_peak.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
    lib.ntk_mfma_peak.restype = ctypes.c_int
    _lib = lib
    return lib


def device_info():
    """(compute units, peak engine clock in kHz) of the current HIP device."""
    cu, clk = ctypes.c_int(0), ctypes.c_int(0)
    check(load().ntk_device_info(ctypes.byref(cu), ctypes.byref(clk)))
    return cu.value, clk.value


def mfma_peak(which="fp32"):
    """Measured matrix-core ceiling (TFLOP/s) of the current device: "fp32" or "fp64"."""
    out = ctypes.c_double(0.0)
    check(load().ntk_mfma_peak({"fp32": 0, "fp64": 1}[which], ctypes.byref(out)))
    return out.value


def last_error(handle=None):
    return load().ntk_last_error(handle).decode()


def check(rc, handle=None):
    if rc != NTK_OK:
        raise NTKError(rc, last_error(handle))
    return rc


_KIND = {"dense": NTK_DENSE, "conv3x3": NTK_CONV3X3_SAME, "gap": NTK_GAP,
         "dwconv3x3": NTK_DWCONV3X3_SAME, "scale": NTK_SCALE, "avgpool2": NTK_AVGPOOL2,
         "conv1x1": NTK_CONV1X1}
_ACT = {"none": NTK_ACT_NONE, "relu": NTK_ACT_RELU, "erf": NTK_ACT_ERF}


def model_desc(spec):
    """Build (ntk_model_desc, keep-alive array) from a workloads-style spec dict."""
    layers = spec["layers"]
    arr = (ntk_layer_desc * len(layers))()
    for i, L in enumerate(layers):
        arr[i].kind = _KIND[L["kind"]]
        arr[i].in_ = int(L.get("in", 0))
        arr[i].out = int(L.get("out", 0))
        arr[i].act = _ACT[L.get("act", "none")]
        arr[i].has_bias = 1 if L.get("bias", False) else 0
    shp = tuple(spec["input_shape"])
    if len(shp) == 1:
        h, w, c = 1, 1, shp[0]
    else:
        h, w, c = shp
    out_dim = layers[-1]["out"]
    d = ntk_model_desc(len(layers), ctypes.cast(arr, ctypes.POINTER(ntk_layer_desc)), h, w, c,
                       out_dim)
    return d, arr
