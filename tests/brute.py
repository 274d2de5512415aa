"""Brute-force constructions used to pin the oracle (tiny inputs only).

Each function re-derives the Sliding Window Recurrence from a *different*
statement in the paper than the oracle's restarted loop, so that a mistake in
either shows up as a disagreement:

* ``dense_L``          -- the transfer operator entry by entry, L_ij = a_{i:j+1}
                          (Sec. 3, eqs. (2.2)-(2.3) and the entry formula after them).
* ``dense_L_neumann``  -- the same operator as the finite Neumann series
                          sum_k (AZ)^k (Sec. 3, eq. (2.3)).
* ``dense_Ltilde``     -- the jagged operator assembled from its hierarchical
                          pieces, calL + G Z_b R (Sec. 4.2, truncated
                          factorisation), with each L_t = (I - A_t Z)^{-1}
                          obtained by a linear solve (Sec. 3.2, intra-block
                          operator), g_t the block's cumulative products and
                          r_t^T = e_l^T L_t (Sec. 3.2, carrier definitions).
* ``dense_L_hierarchical`` -- the full operator from the exact hierarchical
                          decomposition calL + G Z_b T R (Sec. 3.2, Thm.
                          "Hierarchical Decomposition"), with the carrier
                          transfer operator T = (I_b - C Z_b)^{-1} obtained by
                          a linear solve.
* ``window_sum``       -- the explicit sum of decay products over each token's
                          window.
* ``torch_forward``    -- a differentiable float64 torch version of
                          ``window_sum`` whose autograd gradients pin the
                          oracle's backward.
* ``kogge_stone``      -- the Kogge-Stone scan in the paper's matrix form
                          (Sec. 3.1, Alg. "Kogge-Stone Parallel Algorithm":
                          v <- v + F v with F = diag(f) Z^s, then F <- F^2),
                          optionally stopped after a number of stages, which
                          is how Sec. 4.1 defines the uniform window.
* ``dense_L_banded``   -- the uniform window's banded operator
                          I + AZ + ... + (AZ)^{k-1} (Sec. 4.1) by matrix powers.
* ``uniform_window_sum`` / ``torch_uniform`` -- explicit sums over each
                          token's k most recent tokens, and a differentiable
                          torch version of them.
Everything is float64.  Sizes must be tiny (the dense builders are O(T^2)).
"""
import numpy as np


def decay_product(a, i, j):
    """a_{i:j+1} = a_i a_{i-1} ... a_{j+1}; 1 when j == i; 0 when j > i."""
    if j > i:
        return 0.0
    p = 1.0
    for m in range(j + 1, i + 1):
        p *= a[m]
    return p


def dense_L(a):
    """Full (untruncated) transfer operator, entry by entry."""
    a = np.asarray(a, np.float64)
    n = a.shape[0]
    L = np.zeros((n, n))
    for i in range(n):
        for j in range(i + 1):
            L[i, j] = decay_product(a, i, j)
    return L


def dense_L_neumann(a):
    """Full transfer operator as I + AZ + (AZ)^2 + ... + (AZ)^{n-1}."""
    a = np.asarray(a, np.float64)
    n = a.shape[0]
    AZ = np.diag(a) @ np.eye(n, k=-1)
    L = np.zeros((n, n))
    P = np.eye(n)
    for _ in range(n):
        L += P
        P = P @ AZ
    return L


def window_start(i, block):
    return block * max(i // block - 1, 0)


def dense_Ltilde(a, block):
    """Jagged-window operator calL + G Z_b R for a (1-D) decay sequence.

    A last block shorter than ``block`` is handled by zero-padding to a whole
    number of blocks and truncating the result (the padding sits after every
    real token, so it cannot reach them)."""
    a = np.asarray(a, np.float64)
    n = a.shape[0]
    nb = -(-n // block)
    N = nb * block
    ap = np.zeros(N)
    ap[:n] = a
    calL = np.zeros((N, N))
    G = np.zeros((N, nb))
    R = np.zeros((nb, N))
    Zl = np.eye(block, k=-1)
    for t in range(nb):
        sl = slice(t * block, (t + 1) * block)
        at = ap[sl]
        Lt = np.linalg.solve(np.eye(block) - np.diag(at) @ Zl, np.eye(block))
        calL[sl, sl] = Lt
        G[sl, t] = np.cumprod(at)            # (a_{t,1}, a_{t,2:1}, ..., a_{t,l:1})
        R[t, sl] = Lt[block - 1, :]          # e_l^T L_t
    Zb = np.eye(nb, k=-1)
    Lt_full = calL + G @ Zb @ R
    return Lt_full[:n, :n]


def window_sum(a, u, block):
    """h~_i = sum_{j=s(i)}^{i} a_{i:j+1} u_j for u of shape [T, D] and a of
    shape [T] (shared decay) or [T, D] (per-channel decay)."""
    a = np.asarray(a, np.float64)
    u = np.asarray(u, np.float64)
    T, D = u.shape
    h = np.zeros((T, D))
    for i in range(T):
        for j in range(window_start(i, block), i + 1):
            for mu in range(D):
                aa = a if a.ndim == 1 else a[:, mu]
                h[i, mu] += decay_product(aa, i, j) * u[j, mu]
    return h


def swr_slice(x, a, b, c, block, residual=False):
    """Forward of one slice through the explicit window sum."""
    x = np.asarray(x, np.float64)
    h = window_sum(a, np.asarray(b, np.float64) * x, block)
    y = np.asarray(c, np.float64) * h
    return y + x if residual else y


def torch_forward(x, a, b, c, block, residual=False, truncated=True):
    """Differentiable float64 forward of one slice (torch CPU), built from the
    explicit products.  ``truncated=False`` gives the untruncated recurrence."""
    import torch
    T, D = x.shape
    u = b * x
    rows = []
    for i in range(T):
        j0 = window_start(i, block) if truncated else 0
        acc = torch.zeros(D, dtype=torch.float64)
        for j in range(j0, i + 1):
            if a.dim() == 1:
                w = torch.prod(a[j + 1:i + 1]) if i > j else torch.ones((), dtype=torch.float64)
            else:
                w = torch.prod(a[j + 1:i + 1], dim=0) if i > j else torch.ones(D, dtype=torch.float64)
            acc = acc + w * u[j]
        rows.append(acc)
    h = torch.stack(rows)
    y = c * h
    return y + x if residual else y


def torch_grads(x, a, b, c, dy, block, residual=False, truncated=True):
    """(dx, da, db, dc) of sum(dy * forward) by torch autograd, as numpy."""
    import torch
    ts = [torch.tensor(np.asarray(v, np.float64), requires_grad=True) for v in (x, a, b, c)]
    y = torch_forward(*ts, block, residual=residual, truncated=truncated)
    (y * torch.tensor(np.asarray(dy, np.float64))).sum().backward()
    # a leaf that no product touched (T = 1) gets no .grad: its gradient is 0
    return tuple(t.grad.numpy() if t.grad is not None else np.zeros(t.shape) for t in ts)


def dense_L_hierarchical(a, block):
    """Full transfer operator assembled as calL + G Z_b T R, T = (I - C Z_b)^{-1}
    (the exact hierarchical decomposition; no truncation of T)."""
    a = np.asarray(a, np.float64)
    n = a.shape[0]
    nb = -(-n // block)
    N = nb * block
    ap = np.zeros(N)
    ap[:n] = a
    calL = np.zeros((N, N))
    G = np.zeros((N, nb))
    R = np.zeros((nb, N))
    Cd = np.zeros(nb)
    Zl = np.eye(block, k=-1)
    for t in range(nb):
        sl = slice(t * block, (t + 1) * block)
        at = ap[sl]
        Lt = np.linalg.solve(np.eye(block) - np.diag(at) @ Zl, np.eye(block))
        calL[sl, sl] = Lt
        G[sl, t] = np.cumprod(at)
        R[t, sl] = Lt[block - 1, :]
        Cd[t] = np.prod(at)                  # compound attenuation c_t = a_{t,l:1}
    Zb = np.eye(nb, k=-1)
    Tc = np.linalg.solve(np.eye(nb) - np.diag(Cd) @ Zb, np.eye(nb))
    return (calL + G @ Zb @ Tc @ R)[:n, :n]


def exact_states(a, u, h0=None):
    """h_i = sum_{j<=i} a_{i:j+1} u_j + a_{i:0} h0 by explicit products, for u
    [T, D] and a [T] or [T, D]."""
    a = np.asarray(a, np.float64)
    u = np.asarray(u, np.float64)
    T, D = u.shape
    h = np.zeros((T, D))
    for mu in range(D):
        aa = a if a.ndim == 1 else a[:, mu]
        for i in range(T):
            acc = 0.0
            for j in range(i + 1):
                acc += decay_product(aa, i, j) * u[j, mu]
            if h0 is not None:
                acc += decay_product(aa, i, -1) * h0[mu]
            h[i, mu] = acc
    return h


def torch_exact(x, a, b, c, h0, residual=False):
    """Differentiable float64 exact recurrence of one slice from explicit
    products; returns (y, h_last)."""
    import torch
    T, D = x.shape
    u = b * x
    rows = []
    for i in range(T):
        acc = torch.zeros(D, dtype=torch.float64)
        for j in range(-1, i + 1):
            src = h0 if j < 0 else u[j]
            if i > j:
                w = torch.prod(a[j + 1:i + 1], dim=0) if a.dim() == 2 else torch.prod(a[j + 1:i + 1])
            else:
                w = torch.ones((), dtype=torch.float64)
            acc = acc + w * src
        rows.append(acc)
    h = torch.stack(rows) if rows else torch.zeros((0, D), dtype=torch.float64)
    y = c * h
    h_last = h[-1] if T > 0 else h0
    return (y + x if residual else y), h_last


def kogge_stone(a, u, stages=None):
    """Kogge-Stone scan of x_i = a_i x_{i-1} + u_i in the matrix form of
    Sec. 3.1: the work vector v starts as u and f as a; stage t applies
    v <- v + diag(f) Z^s v and squares F = diag(f) Z^s (f_i <- f_i f_{i-s}),
    s = 2^t.  ``stages`` stops the loop early (all stages when None).
    u is [T, D]; a is [T] or [T, D]."""
    u = np.asarray(u, np.float64)
    T = u.shape[0]
    a = np.asarray(a, np.float64)
    f = (a[:, None] * np.ones_like(u)) if a.ndim == 1 else a.copy()
    v = u.copy()
    s, t = 1, 0
    while s <= T - 1 and (stages is None or t < stages):
        v_new = v.copy()
        v_new[s:] = v[s:] + f[s:] * v[:-s]
        f_new = f.copy()
        f_new[s:] = f[s:] * f[:-s]   # rows i <= s of F are zero: their f is never used
        v, f = v_new, f_new
        s, t = 2 * s, t + 1
    return v


def dense_L_banded(a, k):
    """Uniform-window operator I + AZ + ... + (AZ)^{k-1} (shared decay a [T])."""
    a = np.asarray(a, np.float64)
    n = a.shape[0]
    AZ = np.diag(a) @ np.eye(n, k=-1)
    L = np.zeros((n, n))
    P = np.eye(n)
    for _ in range(k):
        L += P
        P = P @ AZ
    return L


def uniform_window_sum(a, u, k):
    """h_i = sum_{j=max(0,i-k+1)}^{i} a_{i:j+1} u_j (u [T, D]; a [T] or [T, D])."""
    a = np.asarray(a, np.float64)
    u = np.asarray(u, np.float64)
    T, D = u.shape
    h = np.zeros((T, D))
    for i in range(T):
        for j in range(max(0, i - k + 1), i + 1):
            for mu in range(D):
                aa = a if a.ndim == 1 else a[:, mu]
                h[i, mu] += decay_product(aa, i, j) * u[j, mu]
    return h


def torch_uniform(x, a, b, c, k, residual=False):
    """Differentiable float64 uniform-window forward of one slice (explicit products)."""
    import torch
    T, D = x.shape
    u = b * x
    rows = []
    for i in range(T):
        acc = torch.zeros(D, dtype=torch.float64)
        for j in range(max(0, i - k + 1), i + 1):
            if a.dim() == 1:
                w = torch.prod(a[j + 1:i + 1]) if i > j else torch.ones((), dtype=torch.float64)
            else:
                w = torch.prod(a[j + 1:i + 1], dim=0) if i > j else torch.ones(D, dtype=torch.float64)
            acc = acc + w * u[j]
        rows.append(acc)
    h = torch.stack(rows)
    y = c * h
    return y + x if residual else y
