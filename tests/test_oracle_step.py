"""Pins of the oracle's recurrent (token-by-token, two-state) form of the
jagged window against the window's own definition: explicit decay-product
sums over each token's window (Sec. 4.2), the closed forms, and the state
carried across arbitrary split points (including inside a block)."""
import numpy as np
import pytest

import brute
import oracle


def _inputs(rng, T, D, per_channel=False):
    x = rng.standard_normal((T, D))
    b = rng.standard_normal((T, D))
    c = rng.standard_normal((T, D))
    a = rng.uniform(0.0, 1.0, (T, D) if per_channel else T)
    if T > 4:
        flat = a.reshape(-1)
        idx = rng.choice(flat.size, size=max(1, flat.size // 8), replace=False)
        flat[idx[: len(idx) // 2]] = 0.0
        flat[idx[len(idx) // 2:]] = 1.0
    return x, a, b, c


def _step(x, a, b, c, state, t0, block, residual=False):
    D = x.shape[1]
    st = np.zeros((1, 2, D)) if state is None else state[None]
    y, st = oracle.step_slices(x[None], a[None], b[None], c[None], st, t0, block, residual)
    return y[0], st[0]


def _restarted_state(a, u, start, i):
    """sum_{j=start}^{i} a_{i:j+1} u_j: the state at token i restarted at `start`."""
    D = u.shape[1]
    out = np.zeros(D)
    for mu in range(D):
        aa = a if a.ndim == 1 else a[:, mu]
        for j in range(start, i + 1):
            out[mu] += brute.decay_product(aa, i, j) * u[j, mu]
    return out


@pytest.mark.parametrize("T,D,block", [(1, 2, 4), (9, 2, 4), (33, 3, 8), (40, 2, 16), (7, 1, 1)])
@pytest.mark.parametrize("per_channel", [False, True])
@pytest.mark.parametrize("residual", [False, True])
def test_step_from_zero_equals_window_sums(rng, T, D, block, per_channel, residual):
    x, a, b, c = _inputs(rng, T, D, per_channel)
    y, st = _step(x, a, b, c, None, 0, block, residual)
    np.testing.assert_allclose(y, brute.swr_slice(x, a, b, c, block, residual), rtol=1e-12, atol=1e-12)
    # The state after the last token: e is that token's jagged-window state,
    # s its state restarted at the start of its own block.
    u = b * x
    last = T - 1
    e_ref = _restarted_state(a, u, brute.window_start(last, block), last)
    s_ref = _restarted_state(a, u, block * (last // block), last)
    np.testing.assert_allclose(st[0], e_ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(st[1], s_ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("block", [1, 4, 16])
def test_step_split_anywhere(rng, block):
    T, D = 50, 3
    x, a, b, c = _inputs(rng, T, D)
    y_full, st_full = _step(x, a, b, c, None, 0, block)
    for cuts in ((0, 50), (0, 1, 50), (0, 16, 50), (0, 7, 23, 24, 49, 50), tuple(range(51))):
        st = None
        parts = []
        for lo, hi in zip(cuts[:-1], cuts[1:]):
            yp, st = _step(x[lo:hi], a[lo:hi], b[lo:hi], c[lo:hi], st, lo, block)
            parts.append(yp)
        np.testing.assert_allclose(np.concatenate(parts), y_full, rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(st, st_full, rtol=1e-13, atol=1e-13)


def test_step_closed_forms(rng):
    T, D = 20, 2
    x, a, b, c = _inputs(rng, T, D)
    u = b * x
    y0, _ = _step(x, np.zeros(T), b, c, None, 0, 4)            # a = 0: no memory
    np.testing.assert_array_equal(y0, c * u)
    y1, _ = _step(x, a, b, c, None, 0, 1)                        # block 1: lag <= 1
    ref = u.copy()
    ref[1:] += a[1:, None] * u[:-1]
    np.testing.assert_allclose(y1, c * ref, rtol=1e-13, atol=1e-13)


def test_step_batched_layout(rng):
    B, K, H, D = 2, 5, 3, 2
    x = rng.standard_normal((B, K, H, D))
    b = rng.standard_normal((B, K, H, D))
    c = rng.standard_normal((B, K, H, D))
    a = rng.uniform(size=(B, K, H))
    st0 = rng.standard_normal((B, H, 2, D))
    y, st = oracle.step(x, a, b, c, st0, 6, 4)
    for bi in range(B):
        for hi in range(H):
            ys, ss = _step(x[bi, :, hi], a[bi, :, hi], b[bi, :, hi], c[bi, :, hi], st0[bi, hi], 6, 4)
            np.testing.assert_array_equal(y[bi, :, hi], ys)
            np.testing.assert_array_equal(st[bi, hi], ss)
