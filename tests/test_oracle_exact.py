"""Pins of the oracle's exact (untruncated) recurrence, Sec. 3 eq. (2.1) with
an initial state, against constructions that do not re-type its loop: the
transfer operator entry by entry, the exact hierarchical decomposition
calL + G Z_b T R (Thm. "Hierarchical Decomposition", the operator that
Alg. "Hierarchical Block Parallel Inference" applies), closed forms, the
window truncation's exactness on the first two blocks, torch autograd and
finite differences."""
import numpy as np
import pytest

import brute
import oracle

SHAPES = [(1, 1), (2, 3), (7, 2), (16, 3), (33, 2), (50, 1)]   # (T, D)


def _inputs(rng, T, D, per_channel=False, zeros=True):
    x = rng.standard_normal((T, D))
    b = rng.standard_normal((T, D))
    c = rng.standard_normal((T, D))
    a = rng.uniform(0.0, 1.0, (T, D) if per_channel else T)
    if zeros and T > 2:
        flat = a.reshape(-1)
        idx = rng.choice(flat.size, size=max(1, flat.size // 8), replace=False)
        flat[idx[: len(idx) // 2]] = 0.0
        flat[idx[len(idx) // 2:]] = 1.0
    h0 = rng.standard_normal(D)
    return x, a, b, c, h0


def _fwd(x, a, b, c, h0=None, residual=False):
    y, hl = oracle.exact_forward_slices(x[None], a[None], b[None], c[None],
                                        None if h0 is None else h0[None], residual)
    return y[0], hl[0]


def _bwd(x, a, b, c, dy, h0=None, dh_last=None, residual=False):
    outs = oracle.exact_backward_slices(x[None], a[None], b[None], c[None], dy[None],
                                        None if h0 is None else h0[None],
                                        None if dh_last is None else dh_last[None], residual)
    return tuple(o[0] for o in outs)


@pytest.mark.parametrize("T,D", SHAPES)
@pytest.mark.parametrize("per_channel", [False, True])
@pytest.mark.parametrize("with_h0", [False, True])
def test_exact_forward_equals_explicit_products(rng, T, D, per_channel, with_h0):
    x, a, b, c, h0 = _inputs(rng, T, D, per_channel)
    h0 = h0 if with_h0 else None
    h = brute.exact_states(a, b * x, h0)
    y, hl = _fwd(x, a, b, c, h0)
    np.testing.assert_allclose(y, c * h, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(hl, h[-1], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("T,block", [(16, 4), (23, 4), (40, 8), (37, 16), (9, 1), (12, 32)])
def test_exact_forward_equals_hierarchical_decomposition(rng, T, block):
    # L = calL + G Z_b T R with the carrier system solved exactly: the
    # operator that the three stages of the hierarchical algorithm apply.
    x, a, b, c, _ = _inputs(rng, T, 3)
    L = brute.dense_L_hierarchical(a, block)
    np.testing.assert_allclose(L, brute.dense_L(a), rtol=1e-12, atol=1e-13)
    y, _ = _fwd(x, a, b, c)
    np.testing.assert_allclose(y, c * (L @ (b * x)), rtol=1e-11, atol=1e-12)


def test_exact_forward_closed_forms(rng):
    T, D = 21, 3
    x, _, b, c, h0 = _inputs(rng, T, D)
    u = b * x
    y0, hl0 = _fwd(x, np.zeros(T), b, c, h0)          # a = 0: no memory at all
    np.testing.assert_array_equal(y0, c * u)
    np.testing.assert_array_equal(hl0, u[-1])
    y1, hl1 = _fwd(x, np.ones(T), b, c, h0)           # a = 1: running sum from h0
    h = h0 + np.cumsum(u, axis=0)
    np.testing.assert_allclose(y1, c * h, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(hl1, h[-1], rtol=1e-12, atol=1e-12)


def test_exact_residual_adds_x(rng):
    x, a, b, c, h0 = _inputs(rng, 13, 2)
    y, _ = _fwd(x, a, b, c, h0)
    yr, _ = _fwd(x, a, b, c, h0, residual=True)
    np.testing.assert_allclose(yr, y + x, rtol=0, atol=1e-15)


@pytest.mark.parametrize("block", [1, 2, 4, 8])
def test_truncated_equals_exact_on_first_two_blocks(rng, block):
    # The jagged window loses nothing on the first 2l tokens (Sec. 4.2); the
    # two oracles are independent loops, so this pins them against each other.
    T = 5 * block + 3
    x, a, b, c, _ = _inputs(rng, T, 3)
    y_exact, _ = _fwd(x, a, b, c)
    y_swr = oracle.forward_slices(x[None], a[None], b[None], c[None], block)[0]
    n = 2 * block
    np.testing.assert_allclose(y_swr[:n], y_exact[:n], rtol=1e-13, atol=1e-13)
    # ...and beyond them the truncation is visible (a is not identically 0).
    assert np.max(np.abs(y_swr[n:] - y_exact[n:])) > 1e-6


def test_exact_state_chaining(rng):
    # Splitting the sequence and passing h_last on as h0 reproduces one pass.
    T, D = 40, 3
    x, a, b, c, h0 = _inputs(rng, T, D)
    y, hl = _fwd(x, a, b, c, h0)
    for cut in (0, 1, 17, 39, 40):
        y1, h1 = _fwd(x[:cut], a[:cut], b[:cut], c[:cut], h0)
        y2, h2 = _fwd(x[cut:], a[cut:], b[cut:], c[cut:], h1)
        np.testing.assert_allclose(np.concatenate([y1, y2]), y, rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(h2, hl, rtol=1e-13, atol=1e-13)


def test_exact_empty_sequence_passes_state_through(rng):
    h0 = rng.standard_normal(4)
    e = np.zeros((0, 4))
    y, hl = _fwd(e, np.zeros(0), e, e, h0)
    assert y.shape == (0, 4)
    np.testing.assert_array_equal(hl, h0)
    dx, da, db, dc, dh0 = _bwd(e, np.zeros(0), e, e, e, h0, dh_last=np.arange(4.0))
    np.testing.assert_array_equal(dh0, np.arange(4.0))


# --------------------------------------------------------------------------- backward


@pytest.mark.parametrize("T,D", [(1, 2), (6, 2), (19, 3)])
@pytest.mark.parametrize("per_channel", [False, True])
@pytest.mark.parametrize("residual", [False, True])
def test_exact_backward_equals_autograd(rng, T, D, per_channel, residual):
    import torch
    x, a, b, c, h0 = _inputs(rng, T, D, per_channel)
    dy = rng.standard_normal((T, D))
    dhl = rng.standard_normal(D)
    ts = [torch.tensor(v, requires_grad=True) for v in (x, a, b, c, h0)]
    y, hl = brute.torch_exact(*ts, residual=residual)
    ((y * torch.tensor(dy)).sum() + (hl * torch.tensor(dhl)).sum()).backward()
    ref = [t.grad.numpy() if t.grad is not None else np.zeros(t.shape) for t in ts]
    got = _bwd(x, a, b, c, dy, h0, dhl, residual)
    for name, g, r in zip(("dx", "da", "db", "dc", "dh0"), got, ref):
        np.testing.assert_allclose(g, r, rtol=1e-11, atol=1e-11, err_msg=name)


def test_exact_backward_finite_differences(rng):
    T, D = 24, 3
    x, a, b, c, h0 = _inputs(rng, T, D, zeros=False)
    a = 0.5 + 0.45 * a
    dy = rng.standard_normal((T, D))
    dhl = rng.standard_normal(D)

    def loss(x_, a_, b_, c_, h0_):
        y, hl = _fwd(x_, a_, b_, c_, h0_)
        return float(np.sum(y * dy) + np.sum(hl * dhl))

    grads = _bwd(x, a, b, c, dy, h0, dhl)
    args = [x, a, b, c, h0]
    eps = 1e-6
    for k, g in zip((0, 1, 2, 3, 4), (grads[0], grads[1], grads[2], grads[3], grads[4])):
        v = args[k]
        for idx in [np.unravel_index(i, v.shape) for i in rng.choice(v.size, min(5, v.size), replace=False)]:
            p = [q.copy() for q in args]
            m = [q.copy() for q in args]
            p[k][idx] += eps
            m[k][idx] -= eps
            fd = (loss(*p) - loss(*m)) / (2 * eps)
            assert abs(fd - g[idx]) <= 1e-6 * max(1.0, abs(fd)), (k, idx, fd, g[idx])


def test_exact_backward_is_adjoint_in_u_and_h0(rng):
    # For fixed a and c the map (u, h0) -> (y, h_last) is linear; its adjoint,
    # (du, dh0) = J^T (dy, dh_last), must satisfy <J v, w> = <v, J^T w>.
    T, D = 30, 2
    x, a, b, c, h0 = _inputs(rng, T, D)
    ones = np.ones((T, D))
    dy = rng.standard_normal((T, D))
    dhl = rng.standard_normal(D)
    y, hl = _fwd(x, a, ones, c, h0)                 # u = x
    dx, _, _, _, dh0 = _bwd(x, a, ones, c, dy, h0, dhl)
    lhs = np.sum(y * dy) + np.sum(hl * dhl)
    rhs = np.sum(x * dx) + np.sum(h0 * dh0)
    assert abs(lhs - rhs) <= 1e-11 * max(1.0, abs(lhs))


def test_exact_backward_equals_truncated_when_T_le_2l(rng):
    block = 8
    x, a, b, c, _ = _inputs(rng, 2 * block, 3)
    dy = rng.standard_normal(x.shape)
    ex = _bwd(x, a, b, c, dy)
    tr = oracle.backward_slices(x[None], a[None], b[None], c[None], dy[None], block)
    for g, r in zip(ex[:4], tr):
        np.testing.assert_allclose(g, r[0], rtol=1e-12, atol=1e-12)


def test_exact_featurised_composition(rng):
    # Logit inputs: the wrapper's gradients w.r.t. the logits by finite differences.
    B, T, H, D = 1, 9, 2, 2
    x = rng.standard_normal((B, T, H, D))
    b = rng.standard_normal((B, T, H, D))
    c = rng.standard_normal((B, T, H, D))
    za = rng.standard_normal((B, T, H))
    h0 = rng.standard_normal((B, H, D))
    dy = rng.standard_normal((B, T, H, D))
    kw = dict(sigmoid_decay=True, sigmoid_pregate=True)
    _, dza, dzb, _, _ = oracle.exact_backward(x, za, b, c, dy, h0, **kw)

    def loss(za_, b_):
        return float(np.sum(oracle.exact_forward(x, za_, b_, c, h0, **kw)[0] * dy))

    eps = 1e-6
    for idx in [(0, 3, 1), (0, 8, 0)]:
        p, m = za.copy(), za.copy()
        p[idx] += eps
        m[idx] -= eps
        fd = (loss(p, b) - loss(m, b)) / (2 * eps)
        assert abs(fd - dza[idx]) <= 1e-6 * max(1.0, abs(fd))
    idx = (0, 4, 1, 0)
    p, m = b.copy(), b.copy()
    p[idx] += eps
    m[idx] -= eps
    fd = (loss(za, p) - loss(za, m)) / (2 * eps)
    assert abs(fd - dzb[idx]) <= 1e-6 * max(1.0, abs(fd))


def test_exact_batched_layout_matches_slices(rng):
    B, T, H, D = 2, 11, 3, 2
    x = rng.standard_normal((B, T, H, D))
    b = rng.standard_normal((B, T, H, D))
    c = rng.standard_normal((B, T, H, D))
    a = rng.uniform(size=(B, T, H))
    h0 = rng.standard_normal((B, H, D))
    y, hl = oracle.exact_forward(x, a, b, c, h0)
    for bi in range(B):
        for hi in range(H):
            ys, hs = _fwd(x[bi, :, hi], a[bi, :, hi], b[bi, :, hi], c[bi, :, hi], h0[bi, hi])
            np.testing.assert_array_equal(y[bi, :, hi], ys)
            np.testing.assert_array_equal(hl[bi, hi], hs)
