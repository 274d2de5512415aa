"""MI355X (gfx950) Sliding Window Recurrence: thin Python binding of ``libswr.so``.

The functions below mirror the C ABI in ``include/swr.h`` (same names, same
arguments) and only marshal torch tensors into pointers, strides and the
current HIP stream; every step of the computation runs in the library's HIP
kernels.  There is no CPU fallback: without the built library, or without a
GPU, the calls raise.

Layouts: ``x, b, c, y, dy, dx, db, dc`` are ``[B, T, H, D]`` (channels
contiguous, all with the same strides); ``a`` is ``[B, T, H]`` in the same
dtype; ``da`` is float32 with ``a``'s shape.  Supported dtypes: float32 and
bfloat16.
"""
import ctypes
import os

from . import build as _build

__all__ = ["SwrError", "swr_forward", "swr_backward", "swr_error_string", "swr_abi_version",
           "swr_launch_info", "SWRFunction", "library_path", "load"]

SWR_ABI_VERSION = 1
SWR_DTYPE_F32 = 0
SWR_DTYPE_BF16 = 1
SWR_FLAG_RESIDUAL = 1


class SwrProblem(ctypes.Structure):
    _fields_ = [
        ("abi_version", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("B", ctypes.c_int64), ("T", ctypes.c_int64), ("H", ctypes.c_int64), ("D", ctypes.c_int64),
        ("block", ctypes.c_int64),
        ("flags", ctypes.c_uint32),
        ("reserved", ctypes.c_int32),
        ("sx_b", ctypes.c_int64), ("sx_t", ctypes.c_int64), ("sx_h", ctypes.c_int64),
        ("sa_b", ctypes.c_int64), ("sa_t", ctypes.c_int64), ("sa_h", ctypes.c_int64),
        ("run_len", ctypes.c_int64),
    ]


class SwrError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {swr_error_string(code)} (status {code})")
        self.code = code


_lib = None


def library_path() -> str:
    return _build.LIB


def load():
    """Load ``libswr.so`` (building it first if it has never been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        lib = ctypes.CDLL(_build.LIB)
        P = ctypes.POINTER(SwrProblem)
        vp = ctypes.c_void_p
        lib.swr_forward.argtypes = [P, vp, vp, vp, vp, vp, vp]
        lib.swr_forward.restype = ctypes.c_int
        lib.swr_backward.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        lib.swr_backward.restype = ctypes.c_int
        lib.swr_error_string.argtypes = [ctypes.c_int]
        lib.swr_error_string.restype = ctypes.c_char_p
        lib.swr_abi_version.restype = ctypes.c_int
        i64p = ctypes.POINTER(ctypes.c_int64)
        lib.swr_launch_info.argtypes = [P, i64p, i64p, i64p]
        lib.swr_launch_info.restype = ctypes.c_int
        if lib.swr_abi_version() != SWR_ABI_VERSION:
            raise RuntimeError("libswr.so ABI version does not match the binding")
        _lib = lib
    return _lib


def swr_error_string(code: int) -> str:
    return load().swr_error_string(int(code)).decode()


def swr_abi_version() -> int:
    return int(load().swr_abi_version())


def make_problem(B, T, H, D, block, dtype_code, x_strides, a_strides, residual=False, run_len=0):
    """A ``swr_problem_t`` from plain integers (strides in elements, [B, T, H] order)."""
    p = SwrProblem()
    p.abi_version = SWR_ABI_VERSION
    p.dtype = dtype_code
    p.B, p.T, p.H, p.D = int(B), int(T), int(H), int(D)
    p.block = int(block)
    p.flags = SWR_FLAG_RESIDUAL if residual else 0
    p.reserved = 0
    p.sx_b, p.sx_t, p.sx_h = (int(s) for s in x_strides)
    p.sa_b, p.sa_t, p.sa_h = (int(s) for s in a_strides)
    p.run_len = int(run_len)
    return p


def swr_launch_info(problem: SwrProblem):
    """(run_len, forward workgroups, backward workgroups) the library picks."""
    r, f, b = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    rc = load().swr_launch_info(ctypes.byref(problem), ctypes.byref(r), ctypes.byref(f),
                                ctypes.byref(b))
    if rc != 0:
        raise SwrError(rc, "swr_launch_info")
    return r.value, f.value, b.value


# ----------------------------------------------------------------------------- torch marshalling


def _torch():
    import torch
    return torch


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return SWR_DTYPE_BF16
    if t.dtype == torch.float32:
        return SWR_DTYPE_F32
    raise TypeError(f"unsupported dtype {t.dtype} (float32 or bfloat16)")


def _problem_from(x, a, block, residual, run_len):
    if x.dim() != 4 or a.dim() != 3 or tuple(a.shape) != tuple(x.shape[:3]):
        raise ValueError("x must be [B, T, H, D] and a must be [B, T, H]")
    if x.stride(3) != 1 and x.shape[3] > 1:
        raise ValueError("the channel dimension of x must be contiguous")
    if a.dtype != x.dtype:
        raise TypeError("a must have the dtype of x")
    B, T, H, D = x.shape
    return make_problem(B, T, H, D, block, _dtype_code(x), x.stride()[:3], a.stride(),
                        residual, run_len)


def _same_layout(ref, *others):
    for t in others:
        if t.shape != ref.shape or t.dtype != ref.dtype or t.stride() != ref.stride():
            raise ValueError("all [B, T, H, D] tensors must share shape, dtype and strides")
        if t.device != ref.device:
            raise ValueError("all tensors must be on the same device")


def _stream(stream, device):
    torch = _torch()
    s = torch.cuda.current_stream(device) if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


def swr_forward(x, a, b, c, block, residual=False, y=None, run_len=0, stream=None):
    """y = SWR(x, a, b, c) on the GPU (see ``include/swr.h``).  Returns y."""
    torch = _torch()
    problem = _problem_from(x, a, block, residual, run_len)
    _same_layout(x, b, c)
    if y is None:
        y = torch.empty_strided(x.shape, x.stride(), dtype=x.dtype, device=x.device)
    else:
        _same_layout(x, y)
    rc = load().swr_forward(ctypes.byref(problem), _ptr(x), _ptr(a), _ptr(b), _ptr(c), _ptr(y),
                            _stream(stream, x.device))
    if rc != 0:
        raise SwrError(rc, "swr_forward")
    return y


def swr_backward(x, a, b, c, dy, block, residual=False, outputs=None, run_len=0, stream=None):
    """(dx, da, db, dc) of the SWR forward given dy (see ``include/swr.h``)."""
    torch = _torch()
    problem = _problem_from(x, a, block, residual, run_len)
    _same_layout(x, b, c, dy)
    if outputs is None:
        dx, db, dc = (torch.empty_strided(x.shape, x.stride(), dtype=x.dtype, device=x.device)
                      for _ in range(3))
        da = torch.empty_strided(a.shape, a.stride(), dtype=torch.float32, device=a.device)
    else:
        dx, da, db, dc = outputs
        _same_layout(x, dx, db, dc)
        if da.dtype != torch.float32 or da.shape != a.shape or da.stride() != a.stride():
            raise ValueError("da must be float32 with the shape and strides of a")
    rc = load().swr_backward(ctypes.byref(problem), _ptr(x), _ptr(a), _ptr(b), _ptr(c), _ptr(dy),
                             _ptr(dx), _ptr(da), _ptr(db), _ptr(dc), _stream(stream, x.device))
    if rc != 0:
        raise SwrError(rc, "swr_backward")
    return dx, da, db, dc


def _autograd_function():
    torch = _torch()

    class _SWRFunction(torch.autograd.Function):
        """Autograd wrapper: forward and backward both run the HIP kernels;
        the backward recomputes what it needs from the saved inputs."""

        @staticmethod
        def forward(ctx, x, a, b, c, block, residual=False):
            ctx.block, ctx.residual = block, residual
            ctx.save_for_backward(x, a, b, c)
            return swr_forward(x, a, b, c, block, residual)

        @staticmethod
        def backward(ctx, dy):
            x, a, b, c = ctx.saved_tensors
            dy = dy if dy.stride() == x.stride() else torch.empty_strided(
                x.shape, x.stride(), dtype=x.dtype, device=x.device).copy_(dy)
            dx, da, db, dc = swr_backward(x, a, b, c, dy, ctx.block, ctx.residual)
            return dx, da.to(a.dtype), db, dc, None, None

    return _SWRFunction


class _Lazy:
    _fn = None

    def __get__(self, obj, owner):
        if _Lazy._fn is None:
            _Lazy._fn = _autograd_function()
        return _Lazy._fn


class _Namespace:
    SWRFunction = _Lazy()


def __getattr__(name):
    if name == "SWRFunction":
        return _Namespace.SWRFunction
    raise AttributeError(name)
