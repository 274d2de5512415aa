"""Pins of the oracle's uniform window (Sec. 4.1, "Uniform Window
Recurrences": the Kogge-Stone factorisation of Sec. 3.1 stopped after log2 k
stages, i.e. the banded operator I + AZ + ... + (AZ)^{k-1}) against
constructions that do not re-type its restarted loop: the Kogge-Stone scan
itself stopped early, the banded operator by matrix powers, explicit products,
closed forms, its relation to the untruncated recurrence and to the jagged
window of Sec. 4.2, torch autograd and finite differences."""
import numpy as np
import pytest

import brute
import oracle

SHAPES = [(1, 1), (2, 3), (9, 2), (16, 3), (33, 2), (50, 1)]   # (T, D)


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
    return x, a, b, c


def _fwd(x, a, b, c, k, residual=False):
    return oracle.uniform_forward_slices(x[None], a[None], b[None], c[None], k, residual)[0]


def _bwd(x, a, b, c, dy, k, residual=False):
    return tuple(o[0] for o in oracle.uniform_backward_slices(x[None], a[None], b[None], c[None],
                                                               dy[None], k, residual))


@pytest.mark.parametrize("T,D", SHAPES)
@pytest.mark.parametrize("k", [1, 2, 3, 4, 8, 16])
@pytest.mark.parametrize("per_channel", [False, True])
def test_uniform_forward_equals_explicit_products(rng, T, D, k, per_channel):
    x, a, b, c = _inputs(rng, T, D, per_channel)
    h = brute.uniform_window_sum(a, b * x, k)
    np.testing.assert_allclose(_fwd(x, a, b, c, k), c * h, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("T", [1, 5, 16, 37, 64])
@pytest.mark.parametrize("stages", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("per_channel", [False, True])
def test_uniform_window_is_kogge_stone_stopped_early(rng, T, stages, per_channel):
    # Sec. 4.1: stopping the scan after log2 k stages leaves lags 0 .. k-1.
    x, a, b, c = _inputs(rng, T, 3, per_channel)
    k = 2 ** stages
    ks = brute.kogge_stone(a, b * x, stages)
    np.testing.assert_allclose(_fwd(x, a, b, c, k), c * ks, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("T,k", [(12, 1), (12, 4), (23, 5), (30, 16), (7, 40)])
def test_uniform_forward_equals_banded_operator(rng, T, k):
    x, a, b, c = _inputs(rng, T, 2)
    Lk = brute.dense_L_banded(a, k)
    np.testing.assert_allclose(_fwd(x, a, b, c, k), c * (Lk @ (b * x)), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("per_channel", [False, True])
def test_uniform_wide_window_is_the_exact_recurrence(rng, per_channel):
    # k >= T keeps every lag: the untruncated recurrence from zero state; for
    # any k the first k tokens see all of their past.
    T, D = 40, 3
    x, a, b, c = _inputs(rng, T, D, per_channel, zeros=False)
    exact, _ = oracle.exact_forward_slices(x[None], a[None], b[None], c[None])
    np.testing.assert_allclose(_fwd(x, a, b, c, T), exact[0], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(_fwd(x, a, b, c, 100), exact[0], rtol=1e-13, atol=1e-13)
    for k in (1, 4, 16):
        np.testing.assert_allclose(_fwd(x, a, b, c, k)[:k], exact[0][:k], rtol=1e-13, atol=1e-13)
        assert not np.allclose(_fwd(x, a, b, c, k)[k:], exact[0][k:])


def test_uniform_closed_forms(rng):
    T, D = 30, 2
    x, a, b, c = _inputs(rng, T, D, zeros=False)
    u = b * x
    np.testing.assert_array_equal(_fwd(x, np.zeros(T), b, c, 8), c * u)     # a = 0: no memory
    np.testing.assert_array_equal(_fwd(x, a, b, c, 1), c * u)               # k = 1: lag 0 only
    k = 6                                                                   # a = 1: moving sums
    cs = np.vstack([np.zeros((1, D)), np.cumsum(u, axis=0)])
    mov = np.array([cs[i + 1] - cs[max(0, i - k + 1)] for i in range(T)])
    np.testing.assert_allclose(_fwd(x, np.ones(T), b, c, k), c * mov, rtol=1e-12, atol=1e-12)
    y = _fwd(x, a, b, c, 4, residual=True)
    np.testing.assert_allclose(y - x, _fwd(x, a, b, c, 4), rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("block", [1, 2, 4, 8])
def test_jagged_window_between_uniform_windows(rng, block):
    # Sec. 4.2: the jagged window keeps every lag up to l and some lags up to
    # 2l - 1, so with non-negative inputs it lies between the uniform windows
    # k = l and k = 2l; a block's first token sees exactly lags 0 .. l and
    # (past the first block) its last token lags 0 .. 2l - 1.
    T, D = 45, 2
    x = rng.uniform(0.0, 1.0, (T, D))
    b = rng.uniform(0.0, 1.0, (T, D))
    c = np.ones((T, D))
    a = rng.uniform(0.2, 1.0, T)
    jag = oracle.forward_slices(x[None], a[None], b[None], c[None], block)[0]
    lo, hi = _fwd(x, a, b, c, block), _fwd(x, a, b, c, 2 * block)
    assert np.all(lo <= jag * (1 + 1e-13)) and np.all(jag <= hi * (1 + 1e-13))
    first = np.arange(block, T, block)
    np.testing.assert_allclose(jag[first], _fwd(x, a, b, c, block + 1)[first], rtol=1e-13, atol=0)
    last = np.arange(2 * block - 1, T, block)
    np.testing.assert_allclose(jag[last], hi[last], rtol=1e-13, atol=0)


@pytest.mark.parametrize("T,D", [(1, 2), (6, 2), (17, 3), (24, 1)])
@pytest.mark.parametrize("k", [1, 2, 4, 8])
@pytest.mark.parametrize("per_channel", [False, True])
@pytest.mark.parametrize("residual", [False, True])
def test_uniform_backward_equals_autograd(rng, T, D, k, per_channel, residual):
    x, a, b, c = _inputs(rng, T, D, per_channel)
    dy = rng.standard_normal((T, D))
    import torch
    ts = [torch.tensor(v, requires_grad=True) for v in (x, a, b, c)]
    y = brute.torch_uniform(*ts, k, residual=residual)
    (y * torch.tensor(dy)).sum().backward()
    ref = [t.grad.numpy() if t.grad is not None else np.zeros(t.shape) for t in ts]
    got = _bwd(x, a, b, c, dy, k, residual)
    for name, g, r in zip(("dx", "da", "db", "dc"), got, ref):
        np.testing.assert_allclose(g, r, rtol=1e-11, atol=1e-11, err_msg=name)


def test_uniform_da_finite_differences(rng):
    T, D, k = 21, 3, 4
    x, a, b, c = _inputs(rng, T, D, zeros=False)
    dy = rng.standard_normal((T, D))
    _, da, _, _ = _bwd(x, a, b, c, dy, k)
    eps = 1e-6
    for m in (0, 1, 5, 12, 20):
        ap, am = a.copy(), a.copy()
        ap[m] += eps
        am[m] -= eps
        fd = (np.sum(dy * _fwd(x, ap, b, c, k)) - np.sum(dy * _fwd(x, am, b, c, k))) / (2 * eps)
        assert abs(fd - da[m]) <= 1e-7 * max(1.0, abs(fd)), (m, fd, da[m])


@pytest.mark.parametrize("k", [1, 2, 5])
def test_uniform_backward_at_zero_decay(rng, k):
    # a = 0: h_i = u_i, and a_m enters only output m, through the state at
    # m - 1 of its window, which is u_{m-1} when the window holds two tokens.
    T, D = 12, 3
    x, _, b, c = _inputs(rng, T, D, zeros=False)
    dy = rng.standard_normal((T, D))
    dx, da, db, dc = _bwd(x, np.zeros(T), b, c, dy, k)
    u, dh = b * x, c * dy
    np.testing.assert_array_equal(dc, dy * u)
    np.testing.assert_array_equal(dx, b * dh)
    np.testing.assert_array_equal(db, x * dh)
    ref = np.zeros(T)
    if k >= 2:
        ref[1:] = np.sum(dh[1:] * u[:-1], axis=1)
    np.testing.assert_allclose(da, ref, rtol=1e-14, atol=1e-14)


def test_uniform_featurisation_chain_rule(rng):
    B, T, H, D, k = 1, 13, 2, 2, 4
    x = rng.standard_normal((B, T, H, D))
    za = rng.standard_normal((B, T, H))
    zb = rng.standard_normal((B, T, H, D))
    c = rng.standard_normal((B, T, H, D))
    dy = rng.standard_normal((B, T, H, D))
    import torch
    ts = [torch.tensor(v, requires_grad=True) for v in (x, za, zb, c)]
    ys = []
    for h in range(H):
        ys.append(brute.torch_uniform(ts[0][0, :, h], torch.sigmoid(ts[1][0, :, h]),
                                      torch.sigmoid(ts[2][0, :, h]), ts[3][0, :, h], k))
    (torch.stack(ys, 1) * torch.tensor(dy[0])).sum().backward()
    y = oracle.uniform_forward(x, za, zb, c, k, sigmoid_decay=True, sigmoid_pregate=True)
    np.testing.assert_allclose(y[0], torch.stack(ys, 1).detach().numpy(), rtol=1e-12, atol=1e-12)
    got = oracle.uniform_backward(x, za, zb, c, dy, k, sigmoid_decay=True, sigmoid_pregate=True)
    for g, t in zip(got, ts):
        np.testing.assert_allclose(g, t.grad.numpy(), rtol=1e-10, atol=1e-11)


def test_uniform_rejects_bad_arguments():
    x = np.zeros((1, 4, 2))
    with pytest.raises(ValueError):
        oracle.uniform_forward_slices(x, np.zeros((1, 4)), x, x, 0)
