"""MI355X (gfx950) Sliding Window Recurrence: thin Python binding of ``libswr.so``.

The functions below mirror the C ABI in ``include/swr.h`` (same names, same
arguments) and only marshal torch tensors into pointers, strides and the
current HIP stream; every step of the computation runs in the library's HIP
kernels.  There is no CPU fallback: without the built library, or without a
GPU, the calls raise.

Layouts: ``x, b, c, y, dy, dx, db, dc`` are ``[B, T, H, D]`` (channels
contiguous, all with the same strides); ``a`` is ``[B, T, H]`` in the same
dtype (one decay per head), or ``[B, T, H, D]`` with x's strides (one decay
per channel, ``SWR_FLAG_PER_CHANNEL_DECAY``); ``da`` is float32 with ``a``'s
shape.  ``sigmoid_decay`` / ``sigmoid_pregate`` make ``a`` / ``b`` logits whose
sigmoids the kernels use (the Phalanx featurisation); the backward then
returns gradients with respect to those logits.  Supported dtypes: float32 and
bfloat16.  The block carriers that the forward saves for the backward are a
float32 ``[B, H, ceil(T / block), D]`` tensor (``carrier_shape``).
"""
import ctypes
import os

from . import build as _build

__all__ = ["SwrError", "swr_forward", "swr_backward", "swr_carriers", "swr_error_string",
           "swr_abi_version", "swr_launch_info", "swr_carrier_elems", "carrier_shape",
           "swr_exact_forward", "swr_exact_forward_noalloc", "swr_exact_backward", "swr_exact_workspace_bytes",
           "swr_step", "swr_exact_step", "swr_decode_state",
           "swr_uniform_forward", "swr_uniform_backward", "swr_uniform_launch_info",
           "swr_forward_shared_gates", "swr_backward_shared_gates", "swr_shared_gates_workspace_bytes",
           "SWRFunction", "SWRUniformFunction", "SWRSharedGatesFunction", "library_path", "load"]

SWR_ABI_VERSION = 1
SWR_DTYPE_F32 = 0
SWR_DTYPE_BF16 = 1
SWR_FLAG_RESIDUAL = 1
SWR_FLAG_PER_CHANNEL_DECAY = 2
SWR_FLAG_SIGMOID_DECAY = 4
SWR_FLAG_SIGMOID_PREGATE = 8
SWR_ERR_SCRATCH = -10
SWR_NOALLOC_SCRATCH_BYTES = 32 << 20


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
        lib.swr_forward.argtypes = [P, vp, vp, vp, vp, vp, vp, vp]
        lib.swr_forward.restype = ctypes.c_int
        lib.swr_carriers.argtypes = [P, vp, vp, vp, vp, vp]
        lib.swr_carriers.restype = ctypes.c_int
        lib.swr_backward.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        lib.swr_backward.restype = ctypes.c_int
        lib.swr_carrier_elems.argtypes = [P]
        lib.swr_carrier_elems.restype = ctypes.c_int64
        lib.swr_error_string.argtypes = [ctypes.c_int]
        lib.swr_error_string.restype = ctypes.c_char_p
        lib.swr_abi_version.restype = ctypes.c_int
        i64p = ctypes.POINTER(ctypes.c_int64)
        lib.swr_launch_info.argtypes = [P, i64p, i64p, i64p, i64p]
        lib.swr_launch_info.restype = ctypes.c_int
        lib.swr_exact_workspace_bytes.argtypes = [P]
        lib.swr_exact_workspace_bytes.restype = ctypes.c_int64
        lib.swr_exact_forward.argtypes = [P] + [vp] * 10
        lib.swr_exact_forward.restype = ctypes.c_int
        lib.swr_exact_forward_noalloc.argtypes = [P] + [vp] * 9
        lib.swr_exact_forward_noalloc.restype = ctypes.c_int
        lib.swr_exact_backward.argtypes = [P] + [vp] * 15
        lib.swr_exact_backward.restype = ctypes.c_int
        lib.swr_step.argtypes = [P, ctypes.c_int64] + [vp] * 7
        lib.swr_step.restype = ctypes.c_int
        lib.swr_exact_step.argtypes = [P] + [vp] * 7
        lib.swr_exact_step.restype = ctypes.c_int
        lib.swr_decode_state.argtypes = [P] + [vp] * 4
        lib.swr_decode_state.restype = ctypes.c_int
        lib.swr_uniform_forward.argtypes = [P] + [vp] * 6
        lib.swr_uniform_forward.restype = ctypes.c_int
        lib.swr_uniform_backward.argtypes = [P] + [vp] * 10
        lib.swr_uniform_backward.restype = ctypes.c_int
        lib.swr_uniform_launch_info.argtypes = [P, i64p, i64p, i64p, i64p]
        lib.swr_uniform_launch_info.restype = ctypes.c_int
        i64 = ctypes.c_int64
        lib.swr_shared_gates_workspace_bytes.argtypes = [P, i64]
        lib.swr_shared_gates_workspace_bytes.restype = i64
        lib.swr_forward_shared_gates.argtypes = [P, i64, vp] + [vp] * 7
        lib.swr_forward_shared_gates.restype = ctypes.c_int
        lib.swr_backward_shared_gates.argtypes = [P, i64, vp] + [vp] * 12
        lib.swr_backward_shared_gates.restype = ctypes.c_int
        if lib.swr_abi_version() != SWR_ABI_VERSION:
            raise RuntimeError("libswr.so ABI version does not match the binding")
        _lib = lib
    return _lib


def swr_error_string(code: int) -> str:
    return load().swr_error_string(int(code)).decode()


def swr_abi_version() -> int:
    return int(load().swr_abi_version())


def make_problem(B, T, H, D, block, dtype_code, x_strides, a_strides, residual=False, run_len=0,
                 per_channel=False, sigmoid_decay=False, sigmoid_pregate=False):
    """A ``swr_problem_t`` from plain integers (strides in elements, [B, T, H] order)."""
    p = SwrProblem()
    p.abi_version = SWR_ABI_VERSION
    p.dtype = dtype_code
    p.B, p.T, p.H, p.D = int(B), int(T), int(H), int(D)
    p.block = int(block)
    p.flags = ((SWR_FLAG_RESIDUAL if residual else 0) | (SWR_FLAG_PER_CHANNEL_DECAY if per_channel else 0)
               | (SWR_FLAG_SIGMOID_DECAY if sigmoid_decay else 0)
               | (SWR_FLAG_SIGMOID_PREGATE if sigmoid_pregate else 0))
    p.reserved = 0
    p.sx_b, p.sx_t, p.sx_h = (int(s) for s in x_strides)
    p.sa_b, p.sa_t, p.sa_h = (int(s) for s in a_strides)
    p.run_len = int(run_len)
    return p


def swr_launch_info(problem: SwrProblem):
    """{'fwd_run_len', 'fwd_workgroups', 'bwd_run_len', 'bwd_workgroups'} the library picks."""
    v = [ctypes.c_int64() for _ in range(4)]
    rc = load().swr_launch_info(ctypes.byref(problem), *(ctypes.byref(t) for t in v))
    if rc != 0:
        raise SwrError(rc, "swr_launch_info")
    return dict(zip(("fwd_run_len", "fwd_workgroups", "bwd_run_len", "bwd_workgroups"),
                    (t.value for t in v)))


def swr_carrier_elems(problem: SwrProblem) -> int:
    """Number of float32 block carriers of a problem."""
    n = int(load().swr_carrier_elems(ctypes.byref(problem)))
    if n < 0:
        raise SwrError(n, "swr_carrier_elems")
    return n


def carrier_shape(x, block):
    """Shape [B, H, ceil(T / block), D] of the block-carrier tensor for x."""
    B, T, H, D = x.shape
    return (B, H, -(-T // block), D)


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


def _problem_from(x, a, block, residual, run_len, sigmoid_decay=False, sigmoid_pregate=False):
    if x.dim() != 4:
        raise ValueError("x must be [B, T, H, D]")
    # The kernels dereference every pointer on the GPU: a host tensor would be
    # a memory fault, not an error, so it is refused here.
    if not x.is_cuda:
        raise ValueError("x must be a GPU tensor")
    if a.device != x.device:
        raise ValueError("a must be on x's device")
    per_channel = a.dim() == 4
    if per_channel:
        if a.shape != x.shape or a.stride() != x.stride():
            raise ValueError("a per-channel decay must have the shape and strides of x")
    elif a.dim() != 3 or tuple(a.shape) != tuple(x.shape[:3]):
        raise ValueError("a must be [B, T, H] (one decay per head) or [B, T, H, D] (per channel)")
    if x.stride(3) != 1 and x.shape[3] > 1:
        raise ValueError("the channel dimension of x must be contiguous")
    if a.dtype != x.dtype:
        raise TypeError("a must have the dtype of x")
    B, T, H, D = x.shape
    return make_problem(B, T, H, D, block, _dtype_code(x), x.stride()[:3],
                        x.stride()[:3] if per_channel else a.stride(), residual, run_len,
                        per_channel, sigmoid_decay, sigmoid_pregate)


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


def _da_check(da, a):
    torch = _torch()
    if (da.dtype != torch.float32 or da.shape != a.shape or da.stride() != a.stride()
            or da.device != a.device):
        raise ValueError("da must be float32 with the shape, strides and device of a")


def _carrier_tensor(x, block, carriers):
    torch = _torch()
    shape = carrier_shape(x, block)
    if carriers is None:
        return torch.empty(shape, dtype=torch.float32, device=x.device)
    if (tuple(carriers.shape) != shape or carriers.dtype != torch.float32
            or not carriers.is_contiguous() or carriers.device != x.device):
        raise ValueError(f"carriers must be a contiguous float32 tensor of shape {shape}")
    return carriers


def swr_forward(x, a, b, c, block, residual=False, y=None, carriers=None, save_carriers=False,
                run_len=0, stream=None, sigmoid_decay=False, sigmoid_pregate=False):
    """y = SWR(x, a, b, c) on the GPU (see ``include/swr.h``).

    Returns y, or (y, carriers) when ``save_carriers`` is true or a carrier
    tensor is passed in (it is filled)."""
    torch = _torch()
    problem = _problem_from(x, a, block, residual, run_len, sigmoid_decay, sigmoid_pregate)
    _same_layout(x, b, c)
    if y is None:
        y = torch.empty_strided(x.shape, x.stride(), dtype=x.dtype, device=x.device)
    else:
        _same_layout(x, y)
    want_v = save_carriers or carriers is not None
    v = _carrier_tensor(x, block, carriers) if want_v else None
    rc = load().swr_forward(ctypes.byref(problem), _ptr(x), _ptr(a), _ptr(b), _ptr(c), _ptr(y),
                            _ptr(v) if want_v else None, _stream(stream, x.device))
    if rc != 0:
        raise SwrError(rc, "swr_forward")
    return (y, v) if want_v else y


def swr_carriers(x, a, b, block, carriers=None, run_len=0, stream=None, sigmoid_decay=False,
                 sigmoid_pregate=False):
    """The block carriers swr_forward would save, computed from x, a, b alone."""
    problem = _problem_from(x, a, block, False, run_len, sigmoid_decay, sigmoid_pregate)
    _same_layout(x, b)
    v = _carrier_tensor(x, block, carriers)
    rc = load().swr_carriers(ctypes.byref(problem), _ptr(x), _ptr(a), _ptr(b), _ptr(v),
                             _stream(stream, x.device))
    if rc != 0:
        raise SwrError(rc, "swr_carriers")
    return v


def swr_backward(x, a, b, c, dy, carriers, block, residual=False, outputs=None, run_len=0,
                 stream=None, sigmoid_decay=False, sigmoid_pregate=False):
    """(dx, da, db, dc) of the SWR forward given dy and the forward's block
    carriers (see ``include/swr.h``), or carriers=None: the kernel then
    recomputes each carrier from the previous block's x, b, a."""
    torch = _torch()
    problem = _problem_from(x, a, block, residual, run_len, sigmoid_decay, sigmoid_pregate)
    _same_layout(x, b, c, dy)
    if carriers is not None:
        carriers = _carrier_tensor(x, block, carriers)
    if outputs is None:
        dx, db, dc = (torch.empty_strided(x.shape, x.stride(), dtype=x.dtype, device=x.device)
                      for _ in range(3))
        da = torch.empty_strided(a.shape, a.stride(), dtype=torch.float32, device=a.device)
    else:
        dx, da, db, dc = outputs
        _same_layout(x, dx, db, dc)
        _da_check(da, a)
    rc = load().swr_backward(ctypes.byref(problem), _ptr(x), _ptr(a), _ptr(b), _ptr(c), _ptr(dy),
                             _opt(carriers), _ptr(dx), _ptr(da), _ptr(db), _ptr(dc),
                             _stream(stream, x.device))
    if rc != 0:
        raise SwrError(rc, "swr_backward")
    return dx, da, db, dc


# ----------------------------------------------------------------------------- exact recurrence


def swr_exact_workspace_bytes(problem: SwrProblem) -> int:
    """Bytes of workspace the exact-recurrence calls need for a problem."""
    n = int(load().swr_exact_workspace_bytes(ctypes.byref(problem)))
    if n < 0:
        raise SwrError(n, "swr_exact_workspace_bytes")
    return n


def _workspace(problem, device, workspace):
    torch = _torch()
    nbytes = swr_exact_workspace_bytes(problem)
    if workspace is None:
        return torch.empty(max(nbytes // 4, 1), dtype=torch.float32, device=device)
    if (workspace.numel() * workspace.element_size() < nbytes or not workspace.is_contiguous()
            or workspace.device != device):
        raise ValueError(f"workspace must be a contiguous tensor of at least {nbytes} bytes on x's device")
    return workspace


def _state(t, x, what):
    """A [B, H, D] float32 state tensor (or None)."""
    torch = _torch()
    if t is None:
        return None
    B, T, H, D = x.shape
    if (tuple(t.shape) != (B, H, D) or t.dtype != torch.float32 or not t.is_contiguous()
            or t.device != x.device):
        raise ValueError(f"{what} must be a contiguous float32 tensor of shape {(B, H, D)}")
    return t


def _opt(t):
    return None if t is None else _ptr(t)


def _exact_forward(noalloc, x, a, b, c, block, h0, residual, y, carriers, save_carriers, h_last,
                   want_h_last, workspace, run_len, stream, sigmoid_decay, sigmoid_pregate):
    torch = _torch()
    problem = _problem_from(x, a, block, residual, run_len, sigmoid_decay, sigmoid_pregate)
    _same_layout(x, b, c)
    h0 = _state(h0, x, "h0")
    if y is None:
        y = torch.empty_strided(x.shape, x.stride(), dtype=x.dtype, device=x.device)
    else:
        _same_layout(x, y)
    want_v = save_carriers or carriers is not None
    v = _carrier_tensor(x, block, carriers) if want_v else None
    B, T, H, D = x.shape
    want_h_last = want_h_last or h_last is not None
    if h_last is None:
        hl = torch.empty((B, H, D), dtype=torch.float32, device=x.device) if want_h_last else None
    else:
        hl = _state(h_last, x, "h_last")
    if noalloc:
        rc = load().swr_exact_forward_noalloc(ctypes.byref(problem), _ptr(x), _ptr(a), _ptr(b), _ptr(c),
                                              _opt(h0), _ptr(y), _opt(v), _opt(hl), _stream(stream, x.device))
    else:
        ws = _workspace(problem, x.device, workspace)
        rc = load().swr_exact_forward(ctypes.byref(problem), _ptr(x), _ptr(a), _ptr(b), _ptr(c), _opt(h0),
                                      _ptr(y), _opt(v), _opt(hl), _ptr(ws), _stream(stream, x.device))
    if rc != 0:
        raise SwrError(rc, "swr_exact_forward_noalloc" if noalloc else "swr_exact_forward")
    out = (y,) + ((v,) if want_v else ()) + ((hl,) if want_h_last else ())
    return out[0] if len(out) == 1 else out


def swr_exact_forward(x, a, b, c, block, h0=None, residual=False, y=None, carriers=None,
                      save_carriers=False, want_h_last=False, workspace=None, run_len=0, stream=None,
                      sigmoid_decay=False, sigmoid_pregate=False, h_last=None):
    """The exact (untruncated) recurrence on the GPU (see ``include/swr.h``):
    returns y, plus the exact block carriers (``save_carriers`` or a
    ``carriers`` tensor) and the final state h_last ([B, H, D] float32,
    ``want_h_last`` or an ``h_last`` tensor), in that order.  ``h0`` is the
    initial state or None."""
    return _exact_forward(False, x, a, b, c, block, h0, residual, y, carriers, save_carriers, h_last,
                          want_h_last, workspace, run_len, stream, sigmoid_decay, sigmoid_pregate)


def swr_exact_forward_noalloc(x, a, b, c, block, h0=None, residual=False, y=None, carriers=None,
                              save_carriers=False, want_h_last=False, run_len=0, stream=None,
                              sigmoid_decay=False, sigmoid_pregate=False, h_last=None):
    """swr_exact_forward with its workspace in the library's static device
    array (``SWR_NOALLOC_SCRATCH_BYTES`` per GPU): the C call allocates no
    device memory.  Pass ``y`` (and ``carriers`` / ``h_last``) to make the
    whole call allocation-free; calls that overlap in time on one GPU race on
    the shared array."""
    return _exact_forward(True, x, a, b, c, block, h0, residual, y, carriers, save_carriers, h_last,
                          want_h_last, None, run_len, stream, sigmoid_decay, sigmoid_pregate)


def swr_exact_backward(x, a, b, c, dy, carriers, block, h0=None, dh_last=None, residual=False,
                       outputs=None, want_dh0=False, workspace=None, run_len=0, stream=None,
                       sigmoid_decay=False, sigmoid_pregate=False):
    """(dx, da, db, dc) of the exact recurrence, plus dh0 when ``want_dh0``;
    ``carriers`` are the exact forward's block carriers, ``dh_last`` the
    gradient flowing into its final state (or None)."""
    torch = _torch()
    problem = _problem_from(x, a, block, residual, run_len, sigmoid_decay, sigmoid_pregate)
    _same_layout(x, b, c, dy)
    if carriers is None:
        raise ValueError("swr_exact_backward needs the exact forward's block carriers")
    carriers = _carrier_tensor(x, block, carriers)
    h0, dh_last = _state(h0, x, "h0"), _state(dh_last, x, "dh_last")
    if outputs is None:
        dx, db, dc = (torch.empty_strided(x.shape, x.stride(), dtype=x.dtype, device=x.device)
                      for _ in range(3))
        da = torch.empty_strided(a.shape, a.stride(), dtype=torch.float32, device=a.device)
    else:
        dx, da, db, dc = outputs
        _same_layout(x, dx, db, dc)
        _da_check(da, a)
    B, T, H, D = x.shape
    dh0 = torch.empty((B, H, D), dtype=torch.float32, device=x.device) if want_dh0 else None
    ws = _workspace(problem, x.device, workspace)
    rc = load().swr_exact_backward(ctypes.byref(problem), _ptr(x), _ptr(a), _ptr(b), _ptr(c), _ptr(dy),
                                   _opt(h0), _ptr(carriers), _opt(dh_last), _ptr(dx), _ptr(da), _ptr(db),
                                   _ptr(dc), _opt(dh0), _ptr(ws), _stream(stream, x.device))
    if rc != 0:
        raise SwrError(rc, "swr_exact_backward")
    return (dx, da, db, dc, dh0) if want_dh0 else (dx, da, db, dc)


# ----------------------------------------------------------------------------- recurrent decoding


def _step_state(state, x, exact):
    torch = _torch()
    B, K, H, D = x.shape
    shape = (B, H, D) if exact else (B, H, 2, D)
    if state is None:
        return torch.zeros(shape, dtype=torch.float32, device=x.device)
    if (tuple(state.shape) != shape or state.dtype != torch.float32 or not state.is_contiguous()
            or state.device != x.device):
        raise ValueError(f"state must be a contiguous float32 tensor of shape {shape}")
    return state


def swr_step(x, a, b, c, block, t0, state=None, residual=False, y=None, stream=None,
             sigmoid_decay=False, sigmoid_pregate=False):
    """K = x.shape[1] tokens at sequence positions t0 .. t0+K-1 in recurrent
    form (see ``include/swr.h``).  ``state`` ([B, H, 2, D] float32; None =
    zeros, i.e. t0 = 0) is updated in place.  Returns (y, state)."""
    torch = _torch()
    problem = _problem_from(x, a, block, residual, 0, sigmoid_decay, sigmoid_pregate)
    _same_layout(x, b, c)
    state = _step_state(state, x, False)
    if y is None:
        y = torch.empty_strided(x.shape, x.stride(), dtype=x.dtype, device=x.device)
    else:
        _same_layout(x, y)
    rc = load().swr_step(ctypes.byref(problem), int(t0), _ptr(x), _ptr(a), _ptr(b), _ptr(c), _ptr(y),
                         _ptr(state), _stream(stream, x.device))
    if rc != 0:
        raise SwrError(rc, "swr_step")
    return y, state


def swr_exact_step(x, a, b, c, state=None, residual=False, y=None, stream=None,
                   sigmoid_decay=False, sigmoid_pregate=False):
    """K tokens of the exact recurrence from the state h ([B, H, D] float32,
    updated in place; None = zeros).  Returns (y, state)."""
    torch = _torch()
    problem = _problem_from(x, a, 16, residual, 0, sigmoid_decay, sigmoid_pregate)
    _same_layout(x, b, c)
    state = _step_state(state, x, True)
    if y is None:
        y = torch.empty_strided(x.shape, x.stride(), dtype=x.dtype, device=x.device)
    else:
        _same_layout(x, y)
    rc = load().swr_exact_step(ctypes.byref(problem), _ptr(x), _ptr(a), _ptr(b), _ptr(c), _ptr(y),
                               _ptr(state), _stream(stream, x.device))
    if rc != 0:
        raise SwrError(rc, "swr_exact_step")
    return y, state


def swr_decode_state(x, a, carriers, block, state=None, stream=None, sigmoid_decay=False):
    """swr_step's state after a jagged-window forward over all of x's tokens,
    from that forward's block carriers (x gives the shape and strides only)."""
    torch = _torch()
    problem = _problem_from(x, a, block, False, 0, sigmoid_decay, False)
    carriers = _carrier_tensor(x, block, carriers)
    B, T, H, D = x.shape
    if state is None:
        state = torch.empty((B, H, 2, D), dtype=torch.float32, device=x.device)
    else:
        state = _step_state(state, x, False)
    rc = load().swr_decode_state(ctypes.byref(problem), _ptr(a), _ptr(carriers), _ptr(state),
                                 _stream(stream, x.device))
    if rc != 0:
        raise SwrError(rc, "swr_decode_state")
    return state


# ----------------------------------------------------------------------------- shared gates


def _gates_check(x, b, group):
    B, T, H, D = x.shape
    if group < 1 or H % group != 0:
        raise ValueError("group must divide the number of heads")
    if tuple(b.shape) != (B, T, H // group, D):
        raise ValueError(f"shared gates must be [B, T, H / group, D] = {(B, T, H // group, D)}")
    if b.dtype != x.dtype or b.device != x.device or (b.stride(3) != 1 and D > 1):
        raise ValueError("shared gates need x's dtype and device and contiguous channels")


def _i64x3(strides):
    return (ctypes.c_int64 * 3)(*(int(s) for s in strides[:3]))


def swr_shared_gates_workspace_bytes(problem: SwrProblem, group: int) -> int:
    """Bytes of workspace swr_backward_shared_gates needs."""
    n = int(load().swr_shared_gates_workspace_bytes(ctypes.byref(problem), int(group)))
    if n < 0:
        raise SwrError(n, "swr_shared_gates_workspace_bytes")
    return n


def swr_forward_shared_gates(x, a, b, c, block, group, residual=False, y=None, carriers=None,
                             save_carriers=False, run_len=0, stream=None, sigmoid_decay=False,
                             sigmoid_pregate=False):
    """Jagged-window forward where heads g*group .. g*group+group-1 share the
    gates b[:, :, g] and c[:, :, g] (b, c: [B, T, H / group, D]).  Returns y,
    or (y, carriers) as swr_forward."""
    torch = _torch()
    problem = _problem_from(x, a, block, residual, run_len, sigmoid_decay, sigmoid_pregate)
    _gates_check(x, b, group)
    _same_layout(b, c)
    if y is None:
        y = torch.empty_strided(x.shape, x.stride(), dtype=x.dtype, device=x.device)
    else:
        _same_layout(x, y)
    want_v = save_carriers or carriers is not None
    v = _carrier_tensor(x, block, carriers) if want_v else None
    rc = load().swr_forward_shared_gates(ctypes.byref(problem), int(group), _i64x3(b.stride()), _ptr(x),
                                         _ptr(a), _ptr(b), _ptr(c), _ptr(y), _ptr(v) if want_v else None,
                                         _stream(stream, x.device))
    if rc != 0:
        raise SwrError(rc, "swr_forward_shared_gates")
    return (y, v) if want_v else y


def swr_backward_shared_gates(x, a, b, c, dy, carriers, block, group, residual=False, outputs=None,
                              workspace=None, run_len=0, stream=None, sigmoid_decay=False,
                              sigmoid_pregate=False):
    """(dx, da, db, dc) of swr_forward_shared_gates; db and dc have b's layout."""
    torch = _torch()
    problem = _problem_from(x, a, block, residual, run_len, sigmoid_decay, sigmoid_pregate)
    _gates_check(x, b, group)
    _same_layout(b, c)
    _same_layout(x, dy)
    carriers = _carrier_tensor(x, block, carriers)
    if outputs is None:
        dx = torch.empty_strided(x.shape, x.stride(), dtype=x.dtype, device=x.device)
        db, dc = (torch.empty_strided(b.shape, b.stride(), dtype=b.dtype, device=b.device) for _ in range(2))
        da = torch.empty_strided(a.shape, a.stride(), dtype=torch.float32, device=a.device)
    else:
        dx, da, db, dc = outputs
        _same_layout(x, dx)
        _same_layout(b, db, dc)
        _da_check(da, a)
    nbytes = swr_shared_gates_workspace_bytes(problem, group)
    if workspace is None:
        workspace = torch.empty(nbytes // 4, dtype=torch.float32, device=x.device) if nbytes else None
    elif (workspace.numel() * workspace.element_size() < nbytes or not workspace.is_contiguous()
          or workspace.device != x.device):
        raise ValueError(f"workspace must be a contiguous tensor of at least {nbytes} bytes on x's device")
    rc = load().swr_backward_shared_gates(ctypes.byref(problem), int(group), _i64x3(b.stride()), _ptr(x),
                                          _ptr(a), _ptr(b), _ptr(c), _ptr(dy), _ptr(carriers), _ptr(dx),
                                          _ptr(da), _ptr(db), _ptr(dc), _opt(workspace),
                                          _stream(stream, x.device))
    if rc != 0:
        raise SwrError(rc, "swr_backward_shared_gates")
    return dx, da, db, dc


# ----------------------------------------------------------------------------- uniform window


def swr_uniform_launch_info(problem: SwrProblem):
    """Launch shape of the uniform-window calls, as ``swr_launch_info``."""
    v = [ctypes.c_int64() for _ in range(4)]
    rc = load().swr_uniform_launch_info(ctypes.byref(problem), *(ctypes.byref(t) for t in v))
    if rc != 0:
        raise SwrError(rc, "swr_uniform_launch_info")
    return dict(zip(("fwd_run_len", "fwd_workgroups", "bwd_run_len", "bwd_workgroups"),
                    (t.value for t in v)))


def swr_uniform_forward(x, a, b, c, window, residual=False, y=None, run_len=0, stream=None,
                        sigmoid_decay=False, sigmoid_pregate=False):
    """y of the uniform-window recurrence (every token sees its ``window``
    most recent tokens; see ``include/swr.h``)."""
    torch = _torch()
    problem = _problem_from(x, a, window, residual, run_len, sigmoid_decay, sigmoid_pregate)
    _same_layout(x, b, c)
    if y is None:
        y = torch.empty_strided(x.shape, x.stride(), dtype=x.dtype, device=x.device)
    else:
        _same_layout(x, y)
    rc = load().swr_uniform_forward(ctypes.byref(problem), _ptr(x), _ptr(a), _ptr(b), _ptr(c), _ptr(y),
                                    _stream(stream, x.device))
    if rc != 0:
        raise SwrError(rc, "swr_uniform_forward")
    return y


def swr_uniform_backward(x, a, b, c, dy, window, residual=False, outputs=None, run_len=0, stream=None,
                         sigmoid_decay=False, sigmoid_pregate=False):
    """(dx, da, db, dc) of the uniform-window forward given dy."""
    torch = _torch()
    problem = _problem_from(x, a, window, residual, run_len, sigmoid_decay, sigmoid_pregate)
    _same_layout(x, b, c, dy)
    if outputs is None:
        dx, db, dc = (torch.empty_strided(x.shape, x.stride(), dtype=x.dtype, device=x.device)
                      for _ in range(3))
        da = torch.empty_strided(a.shape, a.stride(), dtype=torch.float32, device=a.device)
    else:
        dx, da, db, dc = outputs
        _same_layout(x, dx, db, dc)
        _da_check(da, a)
    rc = load().swr_uniform_backward(ctypes.byref(problem), _ptr(x), _ptr(a), _ptr(b), _ptr(c), _ptr(dy),
                                     _ptr(dx), _ptr(da), _ptr(db), _ptr(dc), _stream(stream, x.device))
    if rc != 0:
        raise SwrError(rc, "swr_uniform_backward")
    return dx, da, db, dc


def _autograd_function():
    torch = _torch()

    class _SWRFunction(torch.autograd.Function):
        """Autograd wrapper: forward and backward both run the HIP kernels;
        the backward recomputes what it needs from the saved inputs (and the
        block carriers, unless save_carriers is False: then it recomputes
        those too, and nothing but the inputs is kept)."""

        @staticmethod
        def forward(ctx, x, a, b, c, block, residual=False, sigmoid_decay=False, sigmoid_pregate=False,
                    save_carriers=True):
            ctx.block, ctx.residual = block, residual
            ctx.feat = dict(sigmoid_decay=sigmoid_decay, sigmoid_pregate=sigmoid_pregate)
            if save_carriers:
                y, v = swr_forward(x, a, b, c, block, residual, save_carriers=True, **ctx.feat)
            else:
                y, v = swr_forward(x, a, b, c, block, residual, **ctx.feat), None
            ctx.has_v = v is not None
            # the carriers are the only extra state
            ctx.save_for_backward(x, a, b, c, *((v,) if ctx.has_v else ()))
            return y

        @staticmethod
        def backward(ctx, dy):
            x, a, b, c, *rest = ctx.saved_tensors
            v = rest[0] if ctx.has_v else None
            dy = dy if dy.stride() == x.stride() else torch.empty_strided(
                x.shape, x.stride(), dtype=x.dtype, device=x.device).copy_(dy)
            dx, da, db, dc = swr_backward(x, a, b, c, dy, v, ctx.block, ctx.residual, **ctx.feat)
            return dx, da.to(a.dtype), db, dc, None, None, None, None, None

    class _SWRUniformFunction(torch.autograd.Function):
        """Autograd wrapper of the uniform window (nothing saved but the inputs)."""

        @staticmethod
        def forward(ctx, x, a, b, c, window, residual=False, sigmoid_decay=False, sigmoid_pregate=False):
            ctx.window, ctx.residual = window, residual
            ctx.feat = dict(sigmoid_decay=sigmoid_decay, sigmoid_pregate=sigmoid_pregate)
            ctx.save_for_backward(x, a, b, c)
            return swr_uniform_forward(x, a, b, c, window, residual, **ctx.feat)

        @staticmethod
        def backward(ctx, dy):
            x, a, b, c = ctx.saved_tensors
            dy = dy if dy.stride() == x.stride() else torch.empty_strided(
                x.shape, x.stride(), dtype=x.dtype, device=x.device).copy_(dy)
            dx, da, db, dc = swr_uniform_backward(x, a, b, c, dy, ctx.window, ctx.residual, **ctx.feat)
            return dx, da.to(a.dtype), db, dc, None, None, None, None

    class _SWRSharedGatesFunction(torch.autograd.Function):
        """Autograd wrapper of the jagged window with b, c shared by groups of heads."""

        @staticmethod
        def forward(ctx, x, a, b, c, block, group, residual=False, sigmoid_decay=False, sigmoid_pregate=False):
            ctx.block, ctx.group, ctx.residual = block, group, residual
            ctx.feat = dict(sigmoid_decay=sigmoid_decay, sigmoid_pregate=sigmoid_pregate)
            y, v = swr_forward_shared_gates(x, a, b, c, block, group, residual, save_carriers=True, **ctx.feat)
            ctx.save_for_backward(x, a, b, c, v)
            return y

        @staticmethod
        def backward(ctx, dy):
            x, a, b, c, v = ctx.saved_tensors
            dy = dy if dy.stride() == x.stride() else torch.empty_strided(
                x.shape, x.stride(), dtype=x.dtype, device=x.device).copy_(dy)
            dx, da, db, dc = swr_backward_shared_gates(x, a, b, c, dy, v, ctx.block, ctx.group, ctx.residual,
                                                       **ctx.feat)
            return dx, da.to(a.dtype), db, dc, None, None, None, None, None

    return _SWRFunction, _SWRUniformFunction, _SWRSharedGatesFunction


_FUNCTIONS = None


def __getattr__(name):
    global _FUNCTIONS
    names = ("SWRFunction", "SWRUniformFunction", "SWRSharedGatesFunction")
    if name in names:
        if _FUNCTIONS is None:
            _FUNCTIONS = dict(zip(names, _autograd_function()))
        return _FUNCTIONS[name]
    raise AttributeError(name)
