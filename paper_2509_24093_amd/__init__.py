"""MI355X (gfx950) global Clebsch-Gordan convolution (arXiv 2509.24093, §4.1).

Thin ctypes binding of ``libcgconv.so`` (built in-tree by ``build.py``).
Every step of the computation runs in the library's HIP kernels; this module
only marshals arguments.  PyTorch supplies device memory and the stream.
There is no CPU fallback: if the library is missing, every entry point
raises.

The module-level functions carry the C ABI's names and arguments
(``include/cgconv.h``); :class:`Plan` wraps them for torch tensors.
"""

from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcgconv.so")

CGCONV_OK = 0
CGCONV_ERR_INVALID_ARG = -1
CGCONV_ERR_UNSUPPORTED = -2
CGCONV_ERR_ALIGNMENT = -3
CGCONV_ERR_OUT_OF_MEMORY = -4
CGCONV_ERR_HIP = -5
CGCONV_LMAX = 8
CGCONV_NMAX = 65536
CGCONV_BOUNDARY_CYCLIC = 0
CGCONV_BOUNDARY_LINEAR = 1
CGCONV_GRAPH_NMAX = 16384

_lib = None


class CgconvError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"cgconv error {status}: {message}")
        self.status = status


def library() -> ctypes.CDLL:
    """Load ``libcgconv.so`` (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2509_24093_amd.build` "
                           "(or __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    lib.cgconv_plan_create.argtypes = [i64, i64, i32, i64]
    lib.cgconv_plan_create.restype = vp
    lib.cgconv_plan_create_boundary.argtypes = [i64, i64, i32, i64, i32]
    lib.cgconv_plan_create_boundary.restype = vp
    lib.cgconv_plan_create_graph.argtypes = [i64, i64, i32, i64]
    lib.cgconv_plan_create_graph.restype = vp
    lib.cgconv_forward_graph.argtypes = [vp, vp, vp, vp, vp, vp]
    lib.cgconv_forward_graph.restype = ctypes.c_int
    lib.cgconv_backward_graph.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp]
    lib.cgconv_backward_graph.restype = ctypes.c_int
    lib.cgconv_forward.argtypes = [vp, vp, vp, vp, vp]
    lib.cgconv_forward.restype = ctypes.c_int
    lib.cgconv_forward_bf16.argtypes = [vp, vp, vp, vp, vp]
    lib.cgconv_forward_bf16.restype = ctypes.c_int
    lib.cgconv_forward_mixed.argtypes = [vp, vp, vp, vp, vp, vp]
    lib.cgconv_forward_mixed.restype = ctypes.c_int
    lib.cgconv_forward_interchannel.argtypes = [vp, i32, i32, vp, vp, vp, vp, vp]
    lib.cgconv_forward_interchannel.restype = ctypes.c_int
    lib.cgconv_backward.argtypes = [vp, vp, vp, vp, vp, vp, vp]
    lib.cgconv_backward.restype = ctypes.c_int
    lib.cgconv_gate_value.argtypes = [vp, vp, vp, vp, vp]
    lib.cgconv_gate_value.restype = ctypes.c_int
    lib.cgconv_gate_value_noalloc.argtypes = [i64, i64, i32, i64, vp, vp, vp, vp]
    lib.cgconv_gate_value_noalloc.restype = ctypes.c_int
    lib.cgconv_gate_value_backward.argtypes = [vp, vp, vp, vp, vp, vp, vp]
    lib.cgconv_gate_value_backward.restype = ctypes.c_int
    lib.cgconv_paths.argtypes = [i32, ctypes.POINTER(i32), i64]
    lib.cgconv_paths.restype = i64
    lib.cgconv_plan_destroy.argtypes = [vp]
    lib.cgconv_plan_destroy.restype = None
    lib.cgconv_plan_info.argtypes = [vp, ctypes.POINTER(i64), ctypes.POINTER(i64), ctypes.POINTER(sz)]
    lib.cgconv_plan_info.restype = ctypes.c_int
    lib.cgconv_plan_contraction_info.argtypes = [vp, ctypes.POINTER(i64), ctypes.POINTER(i64)]
    lib.cgconv_plan_contraction_info.restype = ctypes.c_int
    lib.cgconv_plan_export_table.argtypes = [vp, ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_double), i64]
    lib.cgconv_plan_export_table.restype = i64
    lib.cgconv_cg_table.argtypes = [i32, ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_double), i64]
    lib.cgconv_cg_table.restype = i64
    lib.cgconv_contract_host.argtypes = [i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                         ctypes.POINTER(ctypes.c_double)]
    lib.cgconv_contract_host.restype = ctypes.c_int
    lib.cgconv_plan_enable_timing.argtypes = [vp, i32]
    lib.cgconv_plan_enable_timing.restype = ctypes.c_int
    lib.cgconv_plan_stage_times.argtypes = [vp, ctypes.POINTER(ctypes.c_double), i32, ctypes.POINTER(i32),
                                            ctypes.POINTER(i32)]
    lib.cgconv_plan_stage_times.restype = ctypes.c_int
    lib.cgconv_plan_stage_name.argtypes = [vp, i32]
    lib.cgconv_plan_stage_name.restype = ctypes.c_char_p
    lib.cgconv_last_error.argtypes = []
    lib.cgconv_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


# ---- C ABI, same names -------------------------------------------------------

def cgconv_last_error() -> str:
    return library().cgconv_last_error().decode()


def _check(status: int) -> int:
    if status < 0:
        raise CgconvError(status, cgconv_last_error())
    return status


def cgconv_plan_create(batch: int, N: int, L_max: int, C: int) -> int:
    h = library().cgconv_plan_create(batch, N, L_max, C)
    if not h:
        raise CgconvError(CGCONV_ERR_INVALID_ARG, cgconv_last_error())
    return h


def cgconv_plan_create_boundary(batch: int, N: int, L_max: int, C: int, boundary: int) -> int:
    h = library().cgconv_plan_create_boundary(batch, N, L_max, C, boundary)
    if not h:
        raise CgconvError(CGCONV_ERR_INVALID_ARG, cgconv_last_error())
    return h


def cgconv_plan_create_graph(batch: int, N: int, L_max: int, C: int) -> int:
    h = library().cgconv_plan_create_graph(batch, N, L_max, C)
    if not h:
        raise CgconvError(CGCONV_ERR_INVALID_ARG, cgconv_last_error())
    return h


def cgconv_forward_graph(plan: int, U: int, q: int, k: int, out: int, stream: int) -> int:
    """CG convolution in the graph Fourier basis U (device [B][N][N] fp32)."""
    return _check(library().cgconv_forward_graph(plan, U, q, k, out, stream))


def cgconv_backward_graph(plan: int, U: int, q: int, k: int, grad_out: int, grad_q, grad_k, stream: int) -> int:
    """Gradients of the graph Fourier convolution (grad_q or grad_k may be None)."""
    return _check(library().cgconv_backward_graph(plan, U, q, k, grad_out, grad_q, grad_k, stream))


def cgconv_forward(plan: int, q: int, k: int, out: int, stream: int) -> int:
    """Device pointers as integers; returns the status (raises on error)."""
    return _check(library().cgconv_forward(plan, q, k, out, stream))


def cgconv_forward_bf16(plan: int, q: int, k: int, out: int, stream: int) -> int:
    return _check(library().cgconv_forward_bf16(plan, q, k, out, stream))


def cgconv_forward_mixed(plan: int, q: int, k: int, weights: int, out: int, stream: int) -> int:
    """Per-path channel mixing; weights: device fp32 [n_paths][C][C]."""
    return _check(library().cgconv_forward_mixed(plan, q, k, weights, out, stream))


def cgconv_forward_interchannel(plan: int, heads: int, m_out: int, q: int, k: int, weights: int, out: int,
                                stream: int) -> int:
    """Inter-channel product reduced per degree; weights: device fp32
    [heads][L_max+1][m_out][m*m], out: [batch, N, K, heads*m_out]."""
    return _check(library().cgconv_forward_interchannel(plan, heads, m_out, q, k, weights, out, stream))


def cgconv_backward(plan: int, q: int, k: int, grad_out: int, grad_q, grad_k, stream: int) -> int:
    """Gradients of a scalar loss with respect to q and k given grad_out
    (device pointers; grad_q or grad_k may be None to skip it)."""
    return _check(library().cgconv_backward(plan, q, k, grad_out, grad_q, grad_k, stream))


def cgconv_gate_value(plan: int, u: int, v: int, f: int, stream: int) -> int:
    """Invariant softmax gating of u and its token-wise CG product with v."""
    return _check(library().cgconv_gate_value(plan, u, v, f, stream))


def cgconv_gate_value_noalloc(batch: int, N: int, L_max: int, C: int, u: int, v: int, f: int, stream: int) -> int:
    """cgconv_gate_value without a plan and without allocation (the library's
    static device scratch array holds the softmax statistics)."""
    return _check(library().cgconv_gate_value_noalloc(batch, N, L_max, C, u, v, f, stream))


def cgconv_gate_value_backward(plan: int, u: int, v: int, grad_f: int, grad_u, grad_v, stream: int) -> int:
    """Gradients of a scalar loss through cgconv_gate_value with respect to u
    and v given grad_f (device pointers; grad_u or grad_v may be None)."""
    return _check(library().cgconv_gate_value_backward(plan, u, v, grad_f, grad_u, grad_v, stream))


def cgconv_paths(L_max: int):
    """The CG paths (l1, l2, J) in the order of the mixing weights (host only);
    returns an int32 (n_paths, 3) array."""
    import numpy as np
    lib = library()
    n = _check(lib.cgconv_paths(L_max, None, 0))
    out = np.zeros((n, 3), dtype=np.int32)
    got = _check(lib.cgconv_paths(L_max, out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), n))
    assert got == n
    return out


def cgconv_plan_destroy(plan: int) -> None:
    library().cgconv_plan_destroy(plan)


def cgconv_plan_info(plan: int):
    """Returns (n_paths, nnz, workspace_bytes); nnz counts the real-basis
    entries of the tensor the plan evaluates."""
    a, b, d = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_size_t()
    _check(library().cgconv_plan_info(plan, ctypes.byref(a), ctypes.byref(b), ctypes.byref(d)))
    return a.value, b.value, d.value


def cgconv_plan_contraction_info(plan: int):
    """Returns (complex-basis terms, distinct complex products) of the plan's
    contraction."""
    a, b = ctypes.c_int64(), ctypes.c_int64()
    _check(library().cgconv_plan_contraction_info(plan, ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


def cgconv_plan_export_table(plan: int):
    """The real-basis tensor the plan evaluates (host copy).
    Returns (idx int32 (n, 6) = l1, m1, l2, m2, J, M; coef float64 (n,))."""
    import numpy as np
    lib = library()
    n = _check(lib.cgconv_plan_export_table(plan, None, None, 0))
    idx = np.zeros((n, 6), dtype=np.int32)
    coef = np.zeros(n, dtype=np.float64)
    got = _check(lib.cgconv_plan_export_table(plan, idx.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                              coef.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), n))
    assert got == n
    return idx, coef


def cgconv_plan_enable_timing(plan: int, max_calls: int) -> None:
    _check(library().cgconv_plan_enable_timing(plan, max_calls))


def cgconv_plan_stage_times(plan: int):
    """Returns ({stage name: summed ms}, number of timed calls)."""
    lib = library()
    ms = (ctypes.c_double * 8)()
    ns, nc = ctypes.c_int32(), ctypes.c_int32()
    _check(lib.cgconv_plan_stage_times(plan, ms, 8, ctypes.byref(ns), ctypes.byref(nc)))
    return {lib.cgconv_plan_stage_name(plan, i).decode(): ms[i] for i in range(ns.value)}, nc.value


def cgconv_cg_table(L_max: int):
    """Real-basis CG non-zeros as built by the library (host only).
    Returns (idx int32 (n, 6) = l1, m1, l2, m2, J, M; coef float64 (n,))."""
    import numpy as np
    lib = library()
    n = _check(lib.cgconv_cg_table(L_max, None, None, 0))
    idx = np.zeros((n, 6), dtype=np.int32)
    coef = np.zeros(n, dtype=np.float64)
    got = _check(lib.cgconv_cg_table(L_max, idx.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                     coef.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), n))
    assert got == n
    return idx, coef


def cgconv_contract_host(L_max: int, qhat, khat):
    """Host self-check of the frequency-domain contraction: qhat, khat complex
    (K,) arrays; returns the complex (K,) output."""
    import numpy as np
    K = (L_max + 1) ** 2
    q = np.ascontiguousarray(qhat, dtype=np.complex128)
    k = np.ascontiguousarray(khat, dtype=np.complex128)
    if q.shape != (K,) or k.shape != (K,):
        raise ValueError(f"expected ({K},) complex arrays")
    u = np.zeros(K, dtype=np.complex128)
    P = ctypes.POINTER(ctypes.c_double)
    _check(library().cgconv_contract_host(L_max, q.ctypes.data_as(P), k.ctypes.data_as(P), u.ctypes.data_as(P)))
    return u


# ---- torch convenience -------------------------------------------------------

class Plan:
    """A plan for q, k, out of shape [batch, N, (L_max+1)^2, C] on the current
    GPU.  ``plan(q, k)`` returns out; fp32 or bfloat16 tensors.  ``boundary``
    is "cyclic" (default) or "linear" (zero padding, causal sum)."""

    def __init__(self, batch: int, N: int, L_max: int, C: int, boundary: str = "cyclic"):
        if boundary not in ("cyclic", "linear"):
            raise ValueError("boundary must be 'cyclic' or 'linear'")
        self.shape = (int(batch), int(N), (int(L_max) + 1) ** 2, int(C))
        self.L_max = int(L_max)
        self.boundary = boundary
        code = CGCONV_BOUNDARY_LINEAR if boundary == "linear" else CGCONV_BOUNDARY_CYCLIC
        self._h = cgconv_plan_create_boundary(int(batch), int(N), int(L_max), int(C), code)

    def info(self):
        """(n_paths, nnz real-basis, workspace_bytes)."""
        return cgconv_plan_info(self._h)

    def contraction_info(self):
        """(complex-basis terms, distinct complex products)."""
        return cgconv_plan_contraction_info(self._h)

    def export_table(self):
        return cgconv_plan_export_table(self._h)

    def enable_timing(self, max_calls: int):
        cgconv_plan_enable_timing(self._h, max_calls)

    def stage_times(self):
        return cgconv_plan_stage_times(self._h)

    def _args(self, q, k, out, dtype):
        import torch
        for name, t in (("q", q), ("k", k), ("out", out)):
            if not isinstance(t, torch.Tensor) or not t.is_cuda:
                raise ValueError(f"{name} must be a GPU tensor")
            if tuple(t.shape) != self.shape or t.dtype != dtype or not t.is_contiguous():
                raise ValueError(f"{name} must be a contiguous {dtype} tensor of shape {self.shape}")
        return torch.cuda.current_stream().cuda_stream

    def forward(self, q, k, out=None):
        import torch
        if out is None:
            out = torch.empty(self.shape, dtype=q.dtype, device=q.device)
        if q.dtype == torch.float32:
            s = self._args(q, k, out, torch.float32)
            cgconv_forward(self._h, q.data_ptr(), k.data_ptr(), out.data_ptr(), s)
        elif q.dtype == torch.bfloat16:
            s = self._args(q, k, out, torch.bfloat16)
            cgconv_forward_bf16(self._h, q.data_ptr(), k.data_ptr(), out.data_ptr(), s)
        else:
            raise ValueError("q, k must be float32 or bfloat16")
        return out

    def forward_mixed(self, q, k, weights, out=None):
        """Per-path channel mixing (fp32): weights [n_paths, C, C], paths in
        the order of :func:`cgconv_paths`."""
        import torch
        if out is None:
            out = torch.empty(self.shape, dtype=torch.float32, device=q.device)
        s = self._args(q, k, out, torch.float32)
        P = self.info()[0]
        C = self.shape[3]
        if (not isinstance(weights, torch.Tensor) or not weights.is_cuda or weights.dtype != torch.float32
                or tuple(weights.shape) != (P, C, C) or not weights.is_contiguous()):
            raise ValueError(f"weights must be a contiguous float32 GPU tensor of shape {(P, C, C)}")
        cgconv_forward_mixed(self._h, q.data_ptr(), k.data_ptr(), weights.data_ptr(), out.data_ptr(), s)
        return out

    def forward_interchannel(self, q, k, weights, heads: int, out=None):
        """Inter-channel product of every channel pair of each head, reduced
        per output degree (fp32): weights [heads, L_max+1, m_out, m*m] with
        m = C // heads; returns [batch, N, K, heads*m_out]."""
        import torch
        B, N, K, C = self.shape
        if not isinstance(weights, torch.Tensor) or weights.ndim != 4 or not weights.is_cuda:
            raise ValueError("weights must be a GPU tensor of shape [heads, L_max+1, m_out, m*m]")
        m_out = int(weights.shape[2])
        m = C // int(heads) if heads else 0
        if (weights.dtype != torch.float32 or not weights.is_contiguous()
                or tuple(weights.shape) != (int(heads), self.L_max + 1, m_out, m * m)):
            raise ValueError(f"weights must be a contiguous float32 tensor of shape "
                             f"{(int(heads), self.L_max + 1, m_out, m * m)}")
        if out is None:
            out = torch.empty((B, N, K, int(heads) * m_out), dtype=torch.float32, device=q.device)
        for name, t in (("q", q), ("k", k)):
            if not isinstance(t, torch.Tensor) or not t.is_cuda or tuple(t.shape) != self.shape \
                    or t.dtype != torch.float32 or not t.is_contiguous():
                raise ValueError(f"{name} must be a contiguous float32 GPU tensor of shape {self.shape}")
        if (not out.is_cuda or tuple(out.shape) != (B, N, K, int(heads) * m_out) or out.dtype != torch.float32
                or not out.is_contiguous()):
            raise ValueError(f"out must be a contiguous float32 GPU tensor of shape {(B, N, K, int(heads) * m_out)}")
        s = torch.cuda.current_stream().cuda_stream
        cgconv_forward_interchannel(self._h, int(heads), m_out, q.data_ptr(), k.data_ptr(), weights.data_ptr(),
                                    out.data_ptr(), s)
        return out

    def gate_value(self, u, v, out=None):
        """Invariant softmax gating of u and the token-wise CG product with
        v (fp32 tensors of the plan's shape)."""
        import torch
        if out is None:
            out = torch.empty(self.shape, dtype=torch.float32, device=u.device)
        s = self._args(u, v, out, torch.float32)
        cgconv_gate_value(self._h, u.data_ptr(), v.data_ptr(), out.data_ptr(), s)
        return out

    def gate_value_backward(self, u, v, grad_f, need_u: bool = True, need_v: bool = True):
        """(grad_u, grad_v) of a scalar loss through gate_value given grad_f
        (fp32); a gradient that is not needed is returned as None."""
        import torch
        if not (need_u or need_v):
            return None, None
        gu = torch.empty(self.shape, dtype=torch.float32, device=u.device) if need_u else None
        gv = torch.empty(self.shape, dtype=torch.float32, device=u.device) if need_v else None
        s = self._args(u, v, grad_f, torch.float32)
        for t in (gu, gv):
            if t is not None:
                self._args(t, t, t, torch.float32)
        cgconv_gate_value_backward(self._h, u.data_ptr(), v.data_ptr(), grad_f.data_ptr(),
                                   gu.data_ptr() if gu is not None else None,
                                   gv.data_ptr() if gv is not None else None, s)
        return gu, gv

    def backward(self, q, k, grad_out, need_q: bool = True, need_k: bool = True):
        """(grad_q, grad_k) of a scalar loss given grad_out = dL/dout (fp32);
        a gradient that is not needed is returned as None."""
        import torch
        if not (need_q or need_k):
            return None, None
        gq = torch.empty(self.shape, dtype=torch.float32, device=q.device) if need_q else None
        gk = torch.empty(self.shape, dtype=torch.float32, device=q.device) if need_k else None
        s = self._args(q, k, grad_out, torch.float32)
        for name, t in (("grad_q", gq), ("grad_k", gk)):
            if t is not None:
                self._args(t, t, t, torch.float32)
        cgconv_backward(self._h, q.data_ptr(), k.data_ptr(), grad_out.data_ptr(),
                        gq.data_ptr() if gq is not None else None, gk.data_ptr() if gk is not None else None, s)
        return gq, gk

    __call__ = forward

    def close(self):
        if getattr(self, "_h", None):
            cgconv_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


_autograd_fn = None


def cgconv(q, k, plan: Plan):
    """Differentiable CG convolution of fp32 tensors: the forward and the
    backward are the plan's cgconv_forward and cgconv_backward."""
    global _autograd_fn
    if _autograd_fn is None:
        import torch

        class _CgconvFn(torch.autograd.Function):
            @staticmethod
            def forward(ctx, q, k, plan):
                ctx.save_for_backward(q, k)
                ctx.plan = plan
                return plan.forward(q, k)

            @staticmethod
            def backward(ctx, grad_out):
                q, k = ctx.saved_tensors
                gq, gk = ctx.plan.backward(q, k, grad_out.contiguous(), need_q=ctx.needs_input_grad[0],
                                           need_k=ctx.needs_input_grad[1])
                return gq, gk, None

        _autograd_fn = _CgconvFn
    return _autograd_fn.apply(q, k, plan)


class GraphPlan(Plan):
    """A graph Fourier plan: ``plan(U, q, k)`` with U [batch, N, N] (columns
    = graph frequencies) and q, k fp32 [batch, N, (L_max+1)^2, C];
    ``gate_value`` works as on a token plan."""

    def __init__(self, batch: int, N: int, L_max: int, C: int):
        self.shape = (int(batch), int(N), (int(L_max) + 1) ** 2, int(C))
        self.L_max = int(L_max)
        self.boundary = "graph"
        self._h = cgconv_plan_create_graph(int(batch), int(N), int(L_max), int(C))

    def forward(self, U, q, k, out=None):
        import torch
        if out is None:
            out = torch.empty(self.shape, dtype=torch.float32, device=q.device)
        s = self._args(q, k, out, torch.float32)
        B, N = self.shape[0], self.shape[1]
        if (not isinstance(U, torch.Tensor) or not U.is_cuda or U.dtype != torch.float32
                or tuple(U.shape) != (B, N, N) or not U.is_contiguous()):
            raise ValueError(f"U must be a contiguous float32 GPU tensor of shape {(B, N, N)}")
        cgconv_forward_graph(self._h, U.data_ptr(), q.data_ptr(), k.data_ptr(), out.data_ptr(), s)
        return out

    def backward(self, U, q, k, grad_out, need_q: bool = True, need_k: bool = True):
        """(grad_q, grad_k) given grad_out (fp32); an unneeded one is None."""
        import torch
        if not (need_q or need_k):
            return None, None
        s = self._args(q, k, grad_out, torch.float32)
        B, N = self.shape[0], self.shape[1]
        if (not isinstance(U, torch.Tensor) or not U.is_cuda or U.dtype != torch.float32
                or tuple(U.shape) != (B, N, N) or not U.is_contiguous()):
            raise ValueError(f"U must be a contiguous float32 GPU tensor of shape {(B, N, N)}")
        gq = torch.empty(self.shape, dtype=torch.float32, device=q.device) if need_q else None
        gk = torch.empty(self.shape, dtype=torch.float32, device=q.device) if need_k else None
        cgconv_backward_graph(self._h, U.data_ptr(), q.data_ptr(), k.data_ptr(), grad_out.data_ptr(),
                              gq.data_ptr() if gq is not None else None, gk.data_ptr() if gk is not None else None, s)
        return gq, gk

    __call__ = forward


_gate_fn = None


def cgconv_gate(u, v, plan: Plan):
    """Differentiable gating + value tensor product of fp32 tensors in u and
    v: the forward and the backward are the plan's cgconv_gate_value and
    cgconv_gate_value_backward."""
    global _gate_fn
    if _gate_fn is None:
        import torch

        class _GateFn(torch.autograd.Function):
            @staticmethod
            def forward(ctx, u, v, plan):
                ctx.save_for_backward(u, v)
                ctx.plan = plan
                return plan.gate_value(u, v)

            @staticmethod
            def backward(ctx, grad_f):
                u, v = ctx.saved_tensors
                gu, gv = ctx.plan.gate_value_backward(u, v, grad_f.contiguous(), need_u=ctx.needs_input_grad[0],
                                                      need_v=ctx.needs_input_grad[1])
                return gu, gv, None

        _gate_fn = _GateFn
    return _gate_fn.apply(u, v, plan)


_graph_fn = None


def cgconv_graph(U, q, k, plan: GraphPlan):
    """Differentiable graph CG convolution of fp32 tensors in q and k: the
    forward and the backward are the plan's cgconv_forward_graph and
    cgconv_backward_graph.  U is a constant here (no gradient flows to it)."""
    global _graph_fn
    if getattr(U, "requires_grad", False):
        raise ValueError("cgconv_graph gives no gradient with respect to U; pass U.detach()")
    if _graph_fn is None:
        import torch

        class _GraphFn(torch.autograd.Function):
            @staticmethod
            def forward(ctx, U, q, k, plan):
                ctx.save_for_backward(U, q, k)
                ctx.plan = plan
                return plan.forward(U, q, k)

            @staticmethod
            def backward(ctx, grad_out):
                U, q, k = ctx.saved_tensors
                gq, gk = ctx.plan.backward(U, q, k, grad_out.contiguous(), need_q=ctx.needs_input_grad[1],
                                           need_k=ctx.needs_input_grad[2])
                return None, gq, gk, None

        _graph_fn = _GraphFn
    return _graph_fn.apply(U, q, k, plan)
