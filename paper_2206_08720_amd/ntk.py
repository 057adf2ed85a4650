"""Python front end of the MI355X structured-derivatives NTK library.

    theta = compute(spec, params, X1, X2)      # torch tensor [N1, N2, O, O] on the GPU

`spec` is a network description in the `workloads` format; `params` and the
inputs are float32 torch tensors on the current GPU.  PyTorch supplies device
memory and the current HIP stream only: every step runs in libntk.so.
"""
from __future__ import annotations

import ctypes

import torch

from . import _lib


class NTK:
    """A handle bound to one network, maximum batch sizes, device and stream."""

    def __init__(self, spec, max_n1, max_n2, stream=None, device=None):
        self._lib = _lib.load()
        if not torch.cuda.is_available():
            raise RuntimeError("no GPU visible: the NTK library runs on an MI355X only")
        self.spec = spec
        self.out_dim = spec["layers"][-1]["out"]
        self.max_n1, self.max_n2 = int(max_n1), int(max_n2)
        self.device = torch.device("cuda", torch.cuda.current_device() if device is None
                                   else torch.device(device).index or 0)
        desc, self._keep = _lib.model_desc(spec)
        h = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            s = torch.cuda.current_stream() if stream is None else stream
            self._stream = s
            _lib.check(self._lib.ntk_init(ctypes.byref(desc), self.max_n1, self.max_n2,
                                          ctypes.c_void_p(s.cuda_stream), ctypes.byref(h)))
        self._h = h
        self._output = _lib.NTK_OUTPUT_FULL
        self._batch = _lib.NTK_BATCH_FULL

    # -- options -----------------------------------------------------------------------
    def set_option(self, option, value):
        _lib.check(self._lib.ntk_set_option(self._h, option, value), self._h)
        if option == _lib.NTK_OPT_OUTPUT:
            self._output = value
        elif option == _lib.NTK_OPT_BATCH:
            self._batch = value

    def set_variant(self, output="full", batch="full", logit=0):
        """output: "full" | "trace" | "logit" (with `logit` = o*); batch: "full" | "diagonal"."""
        self.set_option(_lib.NTK_OPT_OUTPUT, {"full": _lib.NTK_OUTPUT_FULL, "trace": _lib.NTK_OUTPUT_TRACE,
                                              "logit": _lib.NTK_OUTPUT_LOGIT}[output])
        self.set_option(_lib.NTK_OPT_LOGIT, int(logit))
        self.set_option(_lib.NTK_OPT_BATCH, {"full": _lib.NTK_BATCH_FULL,
                                             "diagonal": _lib.NTK_BATCH_DIAGONAL}[batch])

    def set_method(self, method="structured"):
        """"structured" (Section 3.4, the default) or "jacobian" (the Jacobian-contraction
        baseline of Section 3.2, explicit Jacobians contracted on the GPU)."""
        self.set_option(_lib.NTK_OPT_METHOD, {"structured": _lib.NTK_METHOD_STRUCTURED,
                                              "jacobian": _lib.NTK_METHOD_JACOBIAN}[method])

    def out_shape(self, n1, n2):
        """Shape of theta for batches of n1 and n2 under the current variant options."""
        O = self.out_dim
        inner = (O, O) if self._output == _lib.NTK_OUTPUT_FULL else ()
        outer = (n1,) if self._batch == _lib.NTK_BATCH_DIAGONAL else (n1, n2)
        return outer + inner

    def set_stream(self, stream):
        self._stream = stream
        _lib.check(self._lib.ntk_set_stream(self._h, ctypes.c_void_p(stream.cuda_stream)), self._h)

    def workspace_bytes(self):
        return int(self._lib.ntk_workspace_bytes(self._h))

    # -- compute -----------------------------------------------------------------------
    def _check_tensor(self, t, name):
        if not isinstance(t, torch.Tensor) or t.device != self.device or t.dtype != torch.float32:
            raise TypeError(f"{name} must be a float32 tensor on {self.device}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")

    def compute(self, params, X1, X2=None, out=None):
        """Enqueue Theta(X1, X2) on the handle's stream; returns the [N1,N2,O,O] tensor (or the
        variant's shape, `out_shape`)."""
        if X2 is None:
            X2 = X1
        for i, p in enumerate(params):
            self._check_tensor(p, f"params[{i}]")
        self._check_tensor(X1, "X1")
        self._check_tensor(X2, "X2")
        n1, n2 = X1.shape[0], X2.shape[0]
        shape = self.out_shape(n1, n2)
        if out is None:
            out = torch.empty(shape, dtype=torch.float32, device=self.device)
        else:
            self._check_tensor(out, "out")
            if tuple(out.shape) != shape:
                raise ValueError(f"out has shape {tuple(out.shape)}, expected {shape}")
        ptrs = (ctypes.c_void_p * len(params))(*[p.data_ptr() for p in params])
        _lib.check(self._lib.ntk_compute(self._h, ptrs, ctypes.c_void_p(X1.data_ptr()), n1,
                                         ctypes.c_void_p(X2.data_ptr()), n2,
                                         ctypes.c_void_p(out.data_ptr())), self._h)
        return out

    def vector_product(self, params, X1, X2, v, out=None):
        """Enqueue Theta(X1, X2) v for v [n2, O] without forming Theta; returns [n1, O]."""
        for i, p in enumerate(params):
            self._check_tensor(p, f"params[{i}]")
        self._check_tensor(X1, "X1")
        self._check_tensor(X2, "X2")
        self._check_tensor(v, "v")
        n1, n2, O = X1.shape[0], X2.shape[0], self.out_dim
        if tuple(v.shape) != (n2, O):
            raise ValueError(f"v has shape {tuple(v.shape)}, expected {(n2, O)}")
        if out is None:
            out = torch.empty((n1, O), dtype=torch.float32, device=self.device)
        else:
            self._check_tensor(out, "out")
            if tuple(out.shape) != (n1, O):
                raise ValueError(f"out has shape {tuple(out.shape)}, expected {(n1, O)}")
        ptrs = (ctypes.c_void_p * len(params))(*[p.data_ptr() for p in params])
        _lib.check(self._lib.ntk_vector_product(
            self._h, ptrs, ctypes.c_void_p(X1.data_ptr()), n1, ctypes.c_void_p(X2.data_ptr()), n2,
            ctypes.c_void_p(v.data_ptr()), ctypes.c_void_p(out.data_ptr())), self._h)
        return out

    # -- per-kernel timing -------------------------------------------------------------
    def profile_enable(self, on=True):
        _lib.check(self._lib.ntk_profile_enable(self._h, 1 if on else 0), self._h)

    def profile_read(self):
        """{kernel class: (total ms, launches)} since the last read (synchronises)."""
        n = 32
        names = (ctypes.c_char_p * n)()
        ms = (ctypes.c_double * n)()
        cnt = (ctypes.c_longlong * n)()
        k = self._lib.ntk_profile_read(self._h, names, ms, cnt, n)
        if k < 0:
            _lib.check(k, self._h)
        return {names[i].decode(): (ms[i], cnt[i]) for i in range(k)}

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            self._lib.ntk_free(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def compute(spec, params, X1, X2=None, output="full", batch="full", logit=0, method="structured"):
    """One-shot Theta(X1, X2) (allocates a handle sized for these batches)."""
    X2 = X1 if X2 is None else X2
    h = NTK(spec, X1.shape[0], X2.shape[0])
    try:
        h.set_variant(output, batch, logit)
        h.set_method(method)
        out = h.compute(params, X1, X2)
        torch.cuda.current_stream().synchronize()
        return out
    finally:
        h.close()


def compute_static(spec, params, X1, X2=None, out=None, stream=None):
    """Enqueue the full Theta(X1, X2) through ntk_compute_static: no handle, and no device
    memory allocated by the library (its workspace is the library's fixed per-GPU scratch
    array of _lib.STATIC_SCRATCH_BYTES).  `out` [n1, n2, O, O] may be given so that nothing at
    all is allocated; otherwise it is allocated here, by torch.  Asynchronous on `stream`
    (default: the current stream)."""
    lib = _lib.load()
    X2 = X1 if X2 is None else X2
    O = spec["layers"][-1]["out"]
    n1, n2 = X1.shape[0], X2.shape[0]
    for i, t in enumerate(list(params) + [X1, X2]):
        if not isinstance(t, torch.Tensor) or not t.is_cuda or t.dtype != torch.float32 \
                or not t.is_contiguous():
            raise TypeError(f"argument {i} must be a contiguous float32 tensor on the GPU")
    if out is None:
        out = torch.empty((n1, n2, O, O), dtype=torch.float32, device=X1.device)
    elif tuple(out.shape) != (n1, n2, O, O) or out.dtype != torch.float32 or not out.is_contiguous():
        raise ValueError(f"out must be a contiguous float32 tensor of shape {(n1, n2, O, O)}")
    desc, keep = _lib.model_desc(spec)
    ptrs = (ctypes.c_void_p * len(params))(*[p.data_ptr() for p in params])
    s = torch.cuda.current_stream() if stream is None else stream
    _lib.check(lib.ntk_compute_static(ctypes.byref(desc), ptrs, ctypes.c_void_p(X1.data_ptr()), n1,
                                      ctypes.c_void_p(X2.data_ptr()), n2, ctypes.c_void_p(out.data_ptr()),
                                      ctypes.c_void_p(s.cuda_stream)))
    return out
