"""Double-precision CPU oracle for the Sliding Window Recurrence.

TEST INFRASTRUCTURE ONLY: the plain, slow, obviously correct checker the GPU
library is compared against.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import it.  It shares no code with the
HIP library (``paper_2512_13921_amd``) and never imports it.

The recurrence's arithmetic lives in ``swr_oracle.c`` (see its header for the
definition and the paper passages it follows); this module marshals numpy
arrays, and composes the Phalanx featurisation (Sec. 5, "Featurization": the
decay and the key-like pre-gate are sigmoids of projections) around it in
float64 when asked to: the forward evaluates the sigmoid of the given logits
and runs the recurrence on the results; the backward multiplies the
recurrence's da and db by the sigmoid's derivative (chain rule).

Tensor layout at this level is the library's: ``x, b, c, y, dy, ...`` are
``[B, T, H, D]``; ``a`` is ``[B, T, H]`` (decay shared by a head's D channels,
Sec. 5) or ``[B, T, H, D]`` (per-channel decay).  Inputs of any float dtype are
converted to float64 first.
"""
import ctypes
import os

import numpy as np

from . import build as _build

RESIDUAL = 1

_lib = None


def _load():
    global _lib
    if _lib is None:
        if _build.is_stale():
            _build.build()
        lib = ctypes.CDLL(_build.LIB)
        dp = ctypes.POINTER(ctypes.c_double)
        i64 = ctypes.c_int64
        ci = ctypes.c_int
        for name, nin, nout in (("swr_oracle_forward_slice", 4, 1),
                                ("swr_oracle_backward_slice", 5, 4),
                                ("swr_oracle_forward", 4, 1),
                                ("swr_oracle_backward", 5, 4)):
            fn = getattr(lib, name)
            lead = [i64] if not name.endswith("_slice") else []
            fn.argtypes = lead + [i64, i64, i64, ci, ci] + [dp] * (nin + nout)
            fn.restype = ci
        for name, lead in (("swr_oracle_exact_forward", [i64]), ("swr_oracle_exact_backward", [i64])):
            fn = getattr(lib, name)
            nptr = 6 if name.endswith("forward") else 12
            fn.argtypes = lead + [i64, i64, ci, ci] + [dp] * nptr
            fn.restype = ci
        for name, nptr in (("swr_oracle_uniform_forward", 5), ("swr_oracle_uniform_backward", 9)):
            fn = getattr(lib, name)
            fn.argtypes = [i64, i64, i64, i64, ci, ci] + [dp] * nptr
            fn.restype = ci
        lib.swr_oracle_step.argtypes = [i64, i64, i64, i64, i64, ci, ci] + [dp] * 6
        lib.swr_oracle_step.restype = ci
        lib.swr_oracle_max_threads.restype = ci
        lib.swr_oracle_set_threads.argtypes = [ci]
        lib.swr_oracle_set_threads.restype = None
        _lib = lib
    return _lib


def _ptr(arr):
    return arr.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _c64(arr):
    return np.ascontiguousarray(arr, dtype=np.float64)


def max_threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return int(_load().swr_oracle_max_threads())


def set_threads(n: int) -> None:
    """Sets the OpenMP threads of the oracle's later parallel loops."""
    _load().swr_oracle_set_threads(int(n))


def forward_slices(x, a, b, c, block, residual=False):
    """Forward on independent slices: x, b, c are [S, T, D]; a is [S, T] or [S, T, D]."""
    lib = _load()
    x, a, b, c = _c64(x), _c64(a), _c64(b), _c64(c)
    S, T, D = x.shape
    apc = int(a.ndim == 3)
    y = np.empty((S, T, D), np.float64)
    rc = lib.swr_oracle_forward(S, T, D, int(block), apc, RESIDUAL if residual else 0,
                                _ptr(x), _ptr(a), _ptr(b), _ptr(c), _ptr(y))
    if rc != 0:
        raise ValueError("oracle forward rejected its arguments")
    return y


def backward_slices(x, a, b, c, dy, block, residual=False):
    """Backward on independent slices; returns (dx, da, db, dc) with da shaped like a."""
    lib = _load()
    x, a, b, c, dy = _c64(x), _c64(a), _c64(b), _c64(c), _c64(dy)
    S, T, D = x.shape
    apc = int(a.ndim == 3)
    dx, db, dc = (np.empty((S, T, D), np.float64) for _ in range(3))
    da = np.empty(a.shape, np.float64)
    rc = lib.swr_oracle_backward(S, T, D, int(block), apc, RESIDUAL if residual else 0,
                                 _ptr(x), _ptr(a), _ptr(b), _ptr(c), _ptr(dy),
                                 _ptr(dx), _ptr(da), _ptr(db), _ptr(dc))
    if rc != 0:
        raise ValueError("oracle backward rejected its arguments")
    return dx, da, db, dc


def _to_slices(t):
    # [B, T, H, ...] -> [B*H, T, ...]
    t = np.asarray(t)
    B, T, H = t.shape[:3]
    return np.moveaxis(t, 2, 1).reshape((B * H, T) + t.shape[3:])


def _from_slices(t, B, H):
    S, T = t.shape[:2]
    return np.moveaxis(t.reshape((B, H, T) + t.shape[2:]), 1, 2)


def sigmoid(z):
    """Logistic sigmoid 1 / (1 + exp(-z)) in float64, as exp(-log(1 + exp(-z)))
    so that no intermediate overflows."""
    z = np.asarray(z, np.float64)
    return np.exp(-np.logaddexp(0.0, -z))


def dsigmoid(z):
    """Derivative of the sigmoid: sigmoid(z) * (1 - sigmoid(z)) = sigmoid(z) sigmoid(-z)."""
    return sigmoid(z) * sigmoid(-np.asarray(z, np.float64))


def forward(x, a, b, c, block, residual=False, sigmoid_decay=False, sigmoid_pregate=False):
    """y = SWR(x, a, b, c) for [B, T, H, D] tensors (a: [B, T, H] or [B, T, H, D]).
    With sigmoid_decay / sigmoid_pregate, a / b are logits and the recurrence
    uses their sigmoids."""
    B, T, H, D = np.shape(x)
    a = sigmoid(a) if sigmoid_decay else a
    b = sigmoid(b) if sigmoid_pregate else b
    y = forward_slices(_to_slices(x), _to_slices(a), _to_slices(b), _to_slices(c),
                       block, residual)
    return _from_slices(y, B, H)


def backward(x, a, b, c, dy, block, residual=False, sigmoid_decay=False, sigmoid_pregate=False):
    """(dx, da, db, dc) for [B, T, H, D] tensors; da has the shape of a.  With
    sigmoid_decay / sigmoid_pregate, da / db are the gradients with respect to
    the logits."""
    B, T, H, D = np.shape(x)
    av = sigmoid(a) if sigmoid_decay else a
    bv = sigmoid(b) if sigmoid_pregate else b
    outs = backward_slices(_to_slices(x), _to_slices(av), _to_slices(bv), _to_slices(c),
                           _to_slices(dy), block, residual)
    dx, da, db, dc = (_from_slices(o, B, H) for o in outs)
    if sigmoid_decay:
        da = da * dsigmoid(a)
    if sigmoid_pregate:
        db = db * dsigmoid(b)
    return dx, da, db, dc


# ----------------------------------------------------------------------------
# Exact (untruncated) recurrence with an initial state (Sec. 3, eq. (2.1); the
# result of Alg. "Hierarchical Block Parallel Inference", Sec. 3.2)
# ----------------------------------------------------------------------------

def _opt_ptr(arr):
    return None if arr is None else _ptr(arr)


def exact_forward_slices(x, a, b, c, h0=None, residual=False):
    """Exact recurrence on independent slices: x, b, c are [S, T, D]; a is
    [S, T] or [S, T, D]; h0 is [S, D] or None (zero).  Returns (y, h_last)
    with h_last = the state after the last token, [S, D]."""
    lib = _load()
    x, a, b, c = _c64(x), _c64(a), _c64(b), _c64(c)
    S, T, D = x.shape
    h0 = None if h0 is None else _c64(np.broadcast_to(h0, (S, D)))
    y = np.empty((S, T, D), np.float64)
    h_last = np.empty((S, D), np.float64)
    rc = lib.swr_oracle_exact_forward(S, T, D, int(a.ndim == 3), RESIDUAL if residual else 0,
                                      _ptr(x), _ptr(a), _ptr(b), _ptr(c), _opt_ptr(h0),
                                      _ptr(y), _ptr(h_last))
    if rc != 0:
        raise ValueError("oracle exact forward rejected its arguments")
    return y, h_last


def exact_backward_slices(x, a, b, c, dy, h0=None, dh_last=None, residual=False):
    """Gradients of sum(dy * y) + sum(dh_last * h_last) for the exact
    recurrence on slices; returns (dx, da, db, dc, dh0) with da shaped like a
    and dh0 = d/d h0, [S, D]."""
    lib = _load()
    x, a, b, c, dy = _c64(x), _c64(a), _c64(b), _c64(c), _c64(dy)
    S, T, D = x.shape
    h0 = None if h0 is None else _c64(np.broadcast_to(h0, (S, D)))
    dh_last = None if dh_last is None else _c64(np.broadcast_to(dh_last, (S, D)))
    dx, db, dc = (np.empty((S, T, D), np.float64) for _ in range(3))
    da = np.empty(a.shape, np.float64)
    dh0 = np.empty((S, D), np.float64)
    rc = lib.swr_oracle_exact_backward(S, T, D, int(a.ndim == 3), RESIDUAL if residual else 0,
                                       _ptr(x), _ptr(a), _ptr(b), _ptr(c), _opt_ptr(h0), _ptr(dy),
                                       _opt_ptr(dh_last), _ptr(dx), _ptr(da), _ptr(db), _ptr(dc),
                                       _ptr(dh0))
    if rc != 0:
        raise ValueError("oracle exact backward rejected its arguments")
    return dx, da, db, dc, dh0


def _state_to_slices(h, B, H):
    # [B, H, D] -> [B*H, D]
    return None if h is None else np.asarray(h, np.float64).reshape(B * H, -1)


def exact_forward(x, a, b, c, h0=None, residual=False, sigmoid_decay=False, sigmoid_pregate=False):
    """Exact recurrence for [B, T, H, D] tensors (a: [B, T, H] or [B, T, H, D]);
    h0 is [B, H, D] or None.  Returns (y, h_last) with h_last [B, H, D]."""
    B, T, H, D = np.shape(x)
    a = sigmoid(a) if sigmoid_decay else a
    b = sigmoid(b) if sigmoid_pregate else b
    y, hl = exact_forward_slices(_to_slices(x), _to_slices(a), _to_slices(b), _to_slices(c),
                                 _state_to_slices(h0, B, H), residual)
    return _from_slices(y, B, H), hl.reshape(B, H, D)


def exact_backward(x, a, b, c, dy, h0=None, dh_last=None, residual=False,
                   sigmoid_decay=False, sigmoid_pregate=False):
    """(dx, da, db, dc, dh0) of the exact recurrence for [B, T, H, D] tensors;
    dh_last and dh0 are [B, H, D]."""
    B, T, H, D = np.shape(x)
    av = sigmoid(a) if sigmoid_decay else a
    bv = sigmoid(b) if sigmoid_pregate else b
    outs = exact_backward_slices(_to_slices(x), _to_slices(av), _to_slices(bv), _to_slices(c),
                                 _to_slices(dy), _state_to_slices(h0, B, H),
                                 _state_to_slices(dh_last, B, H), residual)
    dx, da, db, dc = (_from_slices(o, B, H) for o in outs[:4])
    if sigmoid_decay:
        da = da * dsigmoid(a)
    if sigmoid_pregate:
        db = db * dsigmoid(b)
    return dx, da, db, dc, outs[4].reshape(B, H, D)


# ----------------------------------------------------------------------------
# Recurrent form of the jagged window (decoding with a carried state)
# ----------------------------------------------------------------------------

def step_slices(x, a, b, c, state, t0, block, residual=False):
    """K tokens at positions t0 .. t0+K-1 of independent slices: x, b, c are
    [S, K, D]; a is [S, K] or [S, K, D]; state is [S, 2, D] (e, s after token
    t0-1).  Returns (y, new_state)."""
    lib = _load()
    x, a, b, c = _c64(x), _c64(a), _c64(b), _c64(c)
    S, K, D = x.shape
    st = np.array(state, dtype=np.float64, copy=True).reshape(S, 2, D)
    y = np.empty((S, K, D), np.float64)
    rc = lib.swr_oracle_step(S, K, D, int(block), int(t0), int(a.ndim == 3), RESIDUAL if residual else 0,
                             _ptr(x), _ptr(a), _ptr(b), _ptr(c), _ptr(st), _ptr(y))
    if rc != 0:
        raise ValueError("oracle step rejected its arguments")
    return y, st


def step(x, a, b, c, state, t0, block, residual=False, sigmoid_decay=False, sigmoid_pregate=False):
    """Recurrent jagged-window step for [B, K, H, D] tensors (a: [B, K, H] or
    [B, K, H, D]) with state [B, H, 2, D] (None: zeros, i.e. t0 = 0).
    Returns (y, new_state)."""
    B, K, H, D = np.shape(x)
    a = sigmoid(a) if sigmoid_decay else a
    b = sigmoid(b) if sigmoid_pregate else b
    st = np.zeros((B * H, 2, D)) if state is None else np.asarray(state, np.float64).reshape(B * H, 2, D)
    y, st = step_slices(_to_slices(x), _to_slices(a), _to_slices(b), _to_slices(c), st, t0, block, residual)
    return _from_slices(y, B, H), st.reshape(B, H, 2, D)


# ----------------------------------------------------------------------------
# Uniform window (Sec. 4.1): the banded operator I + AZ + ... + (AZ)^{k-1}
# ----------------------------------------------------------------------------

def uniform_forward_slices(x, a, b, c, k, residual=False):
    """Uniform-window forward on independent slices (every token sees the k
    most recent tokens): x, b, c are [S, T, D]; a is [S, T] or [S, T, D]."""
    lib = _load()
    x, a, b, c = _c64(x), _c64(a), _c64(b), _c64(c)
    S, T, D = x.shape
    y = np.empty((S, T, D), np.float64)
    rc = lib.swr_oracle_uniform_forward(S, T, D, int(k), int(a.ndim == 3), RESIDUAL if residual else 0,
                                        _ptr(x), _ptr(a), _ptr(b), _ptr(c), _ptr(y))
    if rc != 0:
        raise ValueError("oracle uniform forward rejected its arguments")
    return y


def uniform_backward_slices(x, a, b, c, dy, k, residual=False):
    """Uniform-window backward on slices; returns (dx, da, db, dc)."""
    lib = _load()
    x, a, b, c, dy = _c64(x), _c64(a), _c64(b), _c64(c), _c64(dy)
    S, T, D = x.shape
    dx, db, dc = (np.empty((S, T, D), np.float64) for _ in range(3))
    da = np.empty(a.shape, np.float64)
    rc = lib.swr_oracle_uniform_backward(S, T, D, int(k), int(a.ndim == 3), RESIDUAL if residual else 0,
                                         _ptr(x), _ptr(a), _ptr(b), _ptr(c), _ptr(dy),
                                         _ptr(dx), _ptr(da), _ptr(db), _ptr(dc))
    if rc != 0:
        raise ValueError("oracle uniform backward rejected its arguments")
    return dx, da, db, dc


def uniform_forward(x, a, b, c, k, residual=False, sigmoid_decay=False, sigmoid_pregate=False):
    """Uniform-window y for [B, T, H, D] tensors (a: [B, T, H] or [B, T, H, D])."""
    B, T, H, D = np.shape(x)
    a = sigmoid(a) if sigmoid_decay else a
    b = sigmoid(b) if sigmoid_pregate else b
    y = uniform_forward_slices(_to_slices(x), _to_slices(a), _to_slices(b), _to_slices(c), k, residual)
    return _from_slices(y, B, H)


def uniform_backward(x, a, b, c, dy, k, residual=False, sigmoid_decay=False, sigmoid_pregate=False):
    """(dx, da, db, dc) of the uniform window for [B, T, H, D] tensors; with the
    sigmoid flags da / db are with respect to the logits."""
    B, T, H, D = np.shape(x)
    av = sigmoid(a) if sigmoid_decay else a
    bv = sigmoid(b) if sigmoid_pregate else b
    outs = uniform_backward_slices(_to_slices(x), _to_slices(av), _to_slices(bv), _to_slices(c),
                                   _to_slices(dy), k, residual)
    dx, da, db, dc = (_from_slices(o, B, H) for o in outs)
    if sigmoid_decay:
        da = da * dsigmoid(a)
    if sigmoid_pregate:
        db = db * dsigmoid(b)
    return dx, da, db, dc


# ----------------------------------------------------------------------------
# Gates shared by groups of heads (Sec. 5, "Gate sharing across heads")
# ----------------------------------------------------------------------------

def _expand_heads(g, group):
    # [B, T, G, D] -> [B, T, G * group, D]: head h reads group h // group
    return np.repeat(np.asarray(g, np.float64), group, axis=2)


def grouped_forward(x, a, b, c, block, group, residual=False, sigmoid_decay=False, sigmoid_pregate=False):
    """Jagged-window forward where heads g*group .. g*group+group-1 share the
    pre-gate b[:, :, g] and the post-gate c[:, :, g] ([B, T, H/group, D]):
    the plain recurrence on gates repeated over each group's heads."""
    return forward(x, a, _expand_heads(b, group), _expand_heads(c, group), block, residual,
                   sigmoid_decay, sigmoid_pregate)


def grouped_backward(x, a, b, c, dy, block, group, residual=False, sigmoid_decay=False,
                     sigmoid_pregate=False):
    """(dx, da, db, dc) for shared gates: db and dc ([B, T, H/group, D]) are
    the per-head gradients of the repeated gates summed over each group."""
    dx, da, db, dc = backward(x, a, _expand_heads(b, group), _expand_heads(c, group), dy, block,
                              residual, sigmoid_decay, sigmoid_pregate)
    B, T, H, D = db.shape

    def fold(t):
        return t.reshape(B, T, H // group, group, D).sum(axis=3)

    return dx, da, fold(db), fold(dc)
