"""Python binding of the SLORR C ABI: argument marshalling only.

Every step of the regularizer runs in the HIP kernels of libslorr.so; this
module turns torch tensors into device pointers and the current torch stream
into a hipStream_t. PyTorch supplies device memory (weights, gradients,
values and the plan workspace) and streams.
"""
from __future__ import annotations

import ctypes
from typing import Optional, Sequence, Tuple

import numpy as np

from . import _lib
from ._lib import ACCUMULATE, AUX, DEFER_GRAD, NO_GRAPH, VALUES_ONLY, SlorrError, check, lib

__all__ = ["Plan", "pe_coefficients", "SlorrError", "HOYER", "NUCLEAR"]

HOYER, NUCLEAR = "hoyer", "nuclear"
_KIND = {HOYER: _lib.HOYER, NUCLEAR: _lib.NUCLEAR}
_DTYPE = {"f32": _lib.F32, "bf16": _lib.BF16}


def pe_coefficients(iters: int = 6, ell: float = 1e-3, degree: int = 5) -> np.ndarray:
    """The library's greedy Polar Express schedule, rows (a_t, b_t, c_t)."""
    out = (ctypes.c_double * (3 * iters))()
    check(lib().slorr_pe_coefficients(float(ell), int(degree), int(iters), out), "slorr_pe_coefficients")
    return np.ctypeslib.as_array(out).reshape(iters, 3).copy()


def _shapes_array(shapes: Sequence[Tuple[int, int]]):
    arr = (_lib.Shape * max(1, len(shapes)))()
    for i, (r, c) in enumerate(shapes):
        arr[i].rows, arr[i].cols = int(r), int(c)
    return arr


class Plan:
    """A plan for a fixed weight set: shapes, dtype, regularizer and options.

    plan(weights, grads) runs the forward + backward of the whole set on the
    current torch stream and returns the device tensor of values
    [L_0 .. L_{n-1}, sum] (plus n_hat and ||W||_F with aux=True).
    With defer_grad=True the call writes no gradient; plan.grad(weights,
    grads, scales) writes it afterwards from the state the call left.
    grad_dtype is the element type of the gradient buffers ("f32" / "bf16").
    """

    def __init__(self, shapes: Sequence[Tuple[int, int]], dtype: str = "bf16", kind: str = HOYER,
                 iters: int = 6, degree: int = 5, ell: float = 1e-3, coeffs=None, eps: float = 0.0,
                 safety: float = 0.01,
                 accumulate: bool = False, values_only: bool = False, graph: bool = True,
                 aux: bool = False, defer_grad: bool = False, grad_dtype: str = "f32",
                 device=None, create_workspace: bool = True):
        self.shapes = [(int(r), int(c)) for r, c in shapes]
        self.n = len(self.shapes)
        self.dtype, self.kind, self.iters = dtype, kind, int(iters)
        self.grad_dtype = grad_dtype
        self.flags = ((ACCUMULATE if accumulate else 0) | (VALUES_ONLY if values_only else 0)
                      | (0 if graph else NO_GRAPH) | (AUX if aux else 0)
                      | (DEFER_GRAD if defer_grad else 0))
        self.generation = 0          # forward calls enqueued so far
        self._c_shapes = _shapes_array(self.shapes)
        if grad_dtype not in _DTYPE:
            raise ValueError(f"grad_dtype must be one of {list(_DTYPE)}")
        opts = _lib.Options()
        lib().slorr_default_options(ctypes.byref(opts))
        opts.iters, opts.degree, opts.ell, opts.eps, opts.flags = int(iters), int(degree), float(ell), float(eps), self.flags
        opts.grad_dtype = _DTYPE[grad_dtype]
        opts.safety = float(safety) if safety > 0 else -1.0     # 0: no stabilisation
        self._coeffs = None
        if coeffs is not None:
            c = np.ascontiguousarray(np.asarray(coeffs, dtype=np.float64).reshape(-1))
            if c.size != 3 * int(iters):
                raise ValueError("coeffs must have iters x 3 entries")
            self._coeffs = (ctypes.c_double * c.size)(*c.tolist())
            opts.coeffs = ctypes.cast(self._coeffs, ctypes.POINTER(ctypes.c_double))
        self._handle = ctypes.c_void_p()
        ws = ctypes.c_size_t()
        if dtype not in _DTYPE or kind not in _KIND:
            raise ValueError(f"dtype must be one of {list(_DTYPE)}, kind one of {list(_KIND)}")
        check(lib().slorr_plan(ctypes.byref(self._handle), self.n, self._c_shapes, _DTYPE[dtype],
                               _KIND[kind], ctypes.byref(opts), ctypes.byref(ws)), "slorr_plan")
        self.workspace_bytes = int(ws.value)
        self.workspace = None
        self.device = None
        if create_workspace:
            self.attach_workspace(device)

    # ------------------------------------------------------------ workspace
    def attach_workspace(self, device=None):
        import torch
        dev = torch.device(device if device is not None else "cuda", )
        if dev.index is None:
            dev = torch.device("cuda", torch.cuda.current_device())
        with torch.cuda.device(dev):
            ws = torch.empty(self.workspace_bytes + 256, dtype=torch.uint8, device=dev)
            off = (-ws.data_ptr()) % 256
            view = ws[off:off + self.workspace_bytes]
            check(lib().slorr_plan_set_workspace(self._handle, ctypes.c_void_p(view.data_ptr()),
                                                 self.workspace_bytes), "slorr_plan_set_workspace")
        self.workspace, self.device = ws, dev

    # ------------------------------------------------------------- the call
    def values_size(self) -> int:
        return (3 * self.n + 1) if (self.flags & AUX) else (self.n + 1)

    def _check_weights(self, weights):
        import torch
        if self.workspace is None:
            raise RuntimeError("plan has no workspace")
        if len(weights) != self.n:
            raise ValueError(f"expected {self.n} weights, got {len(weights)}")
        want_dtype = torch.bfloat16 if self.dtype == "bf16" else torch.float32
        for i, (w, s) in enumerate(zip(weights, self.shapes)):
            if tuple(w.shape) != s or w.dtype != want_dtype or not w.is_contiguous() or w.device != self.device:
                raise ValueError(f"weights[{i}] must be a contiguous {want_dtype} {s} tensor on {self.device}")
        return (ctypes.c_void_p * max(1, self.n))(*[w.data_ptr() for w in weights])

    def _grad_ptrs(self, grads):
        import torch
        want = torch.bfloat16 if self.grad_dtype == "bf16" else torch.float32
        if grads is None or len(grads) != self.n:
            raise ValueError(f"grads: one {want} tensor per weight is required")
        for i, (g, s) in enumerate(zip(grads, self.shapes)):
            if tuple(g.shape) != s or g.dtype != want or not g.is_contiguous() or g.device != self.device:
                raise ValueError(f"grads[{i}] must be a contiguous {want} {s} tensor on {self.device}")
        return (ctypes.c_void_p * max(1, self.n))(*[g.data_ptr() for g in grads])

    def _marshal(self, weights, grads, out_vals, stream):
        import torch
        wp = self._check_weights(weights)
        want_grad = not (self.flags & (VALUES_ONLY | DEFER_GRAD))
        gp = self._grad_ptrs(grads) if want_grad else None
        if out_vals is None:
            out_vals = torch.empty(self.values_size(), dtype=torch.float32, device=self.device)
        elif out_vals.numel() < self.values_size() or out_vals.dtype != torch.float32:
            raise ValueError("out_vals too small or not float32")
        if stream is None:
            stream = torch.cuda.current_stream(self.device)
        return wp, gp, out_vals, stream

    def __call__(self, weights, grads=None, grad_scale: float = 1.0, out_vals=None, stream=None):
        """Enqueue the forward + backward on `stream` (default: current torch stream)."""
        import torch
        wp, gp, out_vals, stream = self._marshal(weights, grads, out_vals, stream)
        with torch.cuda.device(self.device):
            check(lib().slorr_reg_fwd_bwd(self._handle, self.n, wp, self._c_shapes, _KIND[self.kind], self.iters,
                                          ctypes.c_void_p(out_vals.data_ptr()), gp, float(grad_scale),
                                          ctypes.c_void_p(stream.cuda_stream)), "slorr_reg_fwd_bwd")
        self.generation += 1
        return out_vals

    def grad(self, weights, grads, scales=None, grad_scale: float = 1.0, stream=None):
        """Enqueue the gradient of the last forward call: grads[i] = g_i dL_i/dW_i
        (added with accumulate=True), g_i = grad_scale * scales[i] with scales a
        device float32 tensor of n entries (or grad_scale alone)."""
        import torch
        wp = self._check_weights(weights)
        gp = self._grad_ptrs(grads)
        sp = None
        if scales is not None:
            if scales.dtype != torch.float32 or scales.numel() != self.n or not scales.is_contiguous() \
                    or scales.device != self.device:
                raise ValueError(f"scales must be a contiguous float32 tensor of {self.n} entries on {self.device}")
            sp = ctypes.c_void_p(scales.data_ptr())
        if stream is None:
            stream = torch.cuda.current_stream(self.device)
        with torch.cuda.device(self.device):
            check(lib().slorr_reg_grad(self._handle, self.n, wp, self._c_shapes, _KIND[self.kind], self.iters,
                                       gp, sp, float(grad_scale), ctypes.c_void_p(stream.cuda_stream)),
                  "slorr_reg_grad")
        return grads

    def apply_update(self, weights, grads, step: float, steps=None, stream=None):
        """Enqueue W_i <- W_i - s_i grads[i] in place, s_i = step * steps[i]
        (steps: device float32 tensor of n entries) or step (App. E.2, Alg. 1)."""
        import torch
        wp = self._check_weights(weights)
        gp = self._grad_ptrs(grads)
        sp = None
        if steps is not None:
            if steps.dtype != torch.float32 or steps.numel() != self.n or not steps.is_contiguous() \
                    or steps.device != self.device:
                raise ValueError(f"steps must be a contiguous float32 tensor of {self.n} entries on {self.device}")
            sp = ctypes.c_void_p(steps.data_ptr())
        if stream is None:
            stream = torch.cuda.current_stream(self.device)
        with torch.cuda.device(self.device):
            check(lib().slorr_decoupled_apply(self._handle, self.n, wp, self._c_shapes, gp, sp, float(step),
                                              ctypes.c_void_p(stream.cuda_stream)), "slorr_decoupled_apply")
        return weights

    def profiled(self, weights, grads=None, grad_scale: float = 1.0, out_vals=None, stream=None):
        """One call enqueued launch by launch on `stream`, each launch timed
        by HIP events that take the kernel's own start and end; blocks. Returns (out_vals, [(op name, ms), ...])."""
        import torch
        wp, gp, out_vals, stream = self._marshal(weights, grads, out_vals, stream)
        nl = self.info()["launches"]
        ms = (ctypes.c_float * nl)()
        ops = (ctypes.c_int32 * nl)()
        with torch.cuda.device(self.device):
            check(lib().slorr_reg_fwd_bwd_profiled(self._handle, self.n, wp, self._c_shapes, _KIND[self.kind],
                                                   self.iters, ctypes.c_void_p(out_vals.data_ptr()), gp,
                                                   float(grad_scale), ctypes.c_void_p(stream.cuda_stream),
                                                   ms, ops), "slorr_reg_fwd_bwd_profiled")
        self.generation += 1
        return out_vals, [(_lib.OPS[ops[i]], float(ms[i])) for i in range(nl)]

    # ------------------------------------------------------------------ info
    def launches(self) -> list:
        """The schedule in launch order: [(op name, algorithmic flops, tile
        edge), ...] (the products each launch performs, counted in full on the
        unpadded shapes, 0 for the memory-bound kernels; the block tile edge of
        a product launch, 0 for the others)."""
        nl = self.info()["launches"]
        ops = (ctypes.c_int32 * max(1, nl))()
        fl = (ctypes.c_double * max(1, nl))()
        te = (ctypes.c_int32 * max(1, nl))()
        check(lib().slorr_plan_get_launches(self._handle, ops, fl, te), "slorr_plan_get_launches")
        return [(_lib.OPS[ops[i]], float(fl[i]), int(te[i])) for i in range(nl)]

    def info(self) -> dict:
        inf = _lib.PlanInfo()
        check(lib().slorr_plan_get_info(self._handle, ctypes.byref(inf)), "slorr_plan_get_info")
        return {k: getattr(inf, k) for k, _ in _lib.PlanInfo._fields_}

    def close(self):
        if getattr(self, "_handle", None) and self._handle.value:
            lib().slorr_plan_destroy(self._handle)
            self._handle = ctypes.c_void_p()
        self.workspace = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
