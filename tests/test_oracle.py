"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these re-types the oracle's loop: each compares it with a different
construction (explicit products, the hierarchical operator, the Neumann
series, closed forms, torch autograd, finite differences, adjoint identities).
"""
import numpy as np
import pytest

import brute
import oracle

SHAPES = [  # (T, D, block)
    (1, 1, 1), (5, 2, 1), (7, 3, 2), (16, 2, 4), (23, 3, 4), (33, 2, 8), (48, 3, 16),
    (37, 2, 16), (20, 1, 32),
]


def _inputs(rng, T, D, per_channel=False, zeros=True):
    x = rng.standard_normal((T, D))
    b = rng.standard_normal((T, D))
    c = rng.standard_normal((T, D))
    a = rng.uniform(0.0, 1.0, (T, D) if per_channel else T)
    if zeros and T > 2:
        flat = a.reshape(-1)
        idx = rng.choice(flat.size, size=max(1, flat.size // 8), replace=False)
        flat[idx[: len(idx) // 2]] = 0.0      # exact zeros must propagate
        flat[idx[len(idx) // 2:]] = 1.0       # and exact ones must not decay
    return x, a, b, c


def _fwd(x, a, b, c, block, residual=False):
    return oracle.forward_slices(x[None], a[None], b[None], c[None], block, residual)[0]


def _bwd(x, a, b, c, dy, block, residual=False):
    outs = oracle.backward_slices(x[None], a[None], b[None], c[None], dy[None], block, residual)
    return tuple(o[0] for o in outs)


# --------------------------------------------------------------------------- forward


@pytest.mark.parametrize("T,D,block", SHAPES)
@pytest.mark.parametrize("per_channel", [False, True])
@pytest.mark.parametrize("residual", [False, True])
def test_forward_equals_explicit_window_sum(rng, T, D, block, per_channel, residual):
    x, a, b, c = _inputs(rng, T, D, per_channel)
    ref = brute.swr_slice(x, a, b, c, block, residual)
    np.testing.assert_allclose(_fwd(x, a, b, c, block, residual), ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("T,D,block", SHAPES)
def test_forward_equals_hierarchical_operator(rng, T, D, block):
    # y = c * (L~ u) with L~ = calL + G Z_b R assembled from its pieces.
    x, a, b, c = _inputs(rng, T, D)
    Lt = brute.dense_Ltilde(a, block)
    ref = c * (Lt @ (b * x))
    np.testing.assert_allclose(_fwd(x, a, b, c, block), ref, rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("n", [1, 2, 5, 12])
def test_dense_operator_constructions_agree(rng, n):
    # Entry formula L_ij = a_{i:j+1} against the Neumann series (eq. (2.3)),
    # and against the linear solve (I - AZ) x = u (eq. (2.2)).
    a = rng.uniform(-1.5, 1.5, n)
    L = brute.dense_L(a)
    np.testing.assert_allclose(L, brute.dense_L_neumann(a), rtol=1e-12, atol=1e-14)
    u = rng.standard_normal(n)
    x = np.linalg.solve(np.eye(n) - np.diag(a) @ np.eye(n, k=-1), u)
    np.testing.assert_allclose(L @ u, x, rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("n,block", [(8, 2), (12, 4), (16, 4), (15, 4), (24, 8)])
def test_jagged_operator_is_block_bidiagonal_part_of_L(rng, n, block):
    # T ~ I_b keeps the diagonal blocks L_t and the first sub-diagonal blocks
    # F_{t,t-1} = g_t r_{t-1}^T of the exact operator unchanged, and drops the rest.
    a = rng.uniform(0.0, 1.0, n)
    L = brute.dense_L(a)
    Lt = brute.dense_Ltilde(a, block)
    blk = np.arange(n) // block
    keep = (blk[:, None] == blk[None, :]) | (blk[:, None] == blk[None, :] + 1)
    np.testing.assert_allclose(Lt, np.where(keep, L, 0.0), rtol=1e-12, atol=1e-14)


def test_block_identities(rng):
    # g_t = a_{t,1} L_t e_1 (remark after Alg. 2) and rank-one F_{t,t-1} (Thm. low-rank).
    block, nb = 6, 4
    a = rng.uniform(0.0, 1.0, block * nb)
    L = brute.dense_L(a)
    for t in range(1, nb):
        sl, pv = slice(t * block, (t + 1) * block), slice((t - 1) * block, t * block)
        Lt, Lp = L[sl, sl], L[pv, pv]
        g = np.cumprod(a[sl])
        np.testing.assert_allclose(g, a[t * block] * Lt[:, 0], rtol=1e-12)
        np.testing.assert_allclose(L[sl, pv], np.outer(g, Lp[-1, :]), rtol=1e-12, atol=1e-15)


def test_decay_zero_closed_form(rng):
    # a == 0: every state is just its own input, y = c * b * x.
    T, D = 40, 3
    x, _, b, c = _inputs(rng, T, D)
    np.testing.assert_allclose(_fwd(x, np.zeros(T), b, c, 8), c * b * x, rtol=1e-15)


@pytest.mark.parametrize("block", [1, 3, 8])
def test_decay_one_closed_form(rng, block):
    # a == 1: jagged box filter, h_i = sum_{j=s(i)}^{i} u_j = S_i - S_{s(i)-1}.
    T, D = 41, 2
    x, _, b, c = _inputs(rng, T, D)
    u = b * x
    S = np.vstack([np.zeros((1, D)), np.cumsum(u, axis=0)])
    starts = np.array([brute.window_start(i, block) for i in range(T)])
    h = S[np.arange(T) + 1] - S[starts]
    np.testing.assert_allclose(_fwd(x, np.ones(T), b, c, block), c * h, rtol=1e-10, atol=1e-12)


def test_block_one_closed_form(rng):
    # l = 1: each token sees itself and its predecessor, h_i = u_i + a_i u_{i-1}.
    T, D = 30, 3
    x, a, b, c = _inputs(rng, T, D)
    u = b * x
    h = u.copy()
    h[1:] += a[1:, None] * u[:-1]
    np.testing.assert_allclose(_fwd(x, a, b, c, 1), c * h, rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("block", [1, 2, 4, 8])
def test_first_two_blocks_equal_untruncated(rng, block):
    # "no error on the first 2l time steps" (Sec. 4.2): T <= 2l gives the exact
    # recurrence; at T = 2l + 1 the last token loses the first block's inputs.
    D = 2
    T = 2 * block + 1
    x, a, b, c = _inputs(rng, T, D, zeros=False)
    a = rng.uniform(0.3, 1.0, T)
    exact = c * (brute.dense_L(a) @ (b * x))
    y = _fwd(x, a, b, c, block)
    np.testing.assert_allclose(y[:2 * block], exact[:2 * block], rtol=1e-12, atol=1e-13)
    assert np.abs(y[2 * block] - exact[2 * block]).max() > 1e-6


def test_window_support(rng):
    # Output i depends on input j exactly when s(i) <= j <= i (lags up to l on
    # the block's first token and up to 2l - 1 on its last).
    T, D, block = 20, 1, 4
    x, a, b, c = _inputs(rng, T, D, zeros=False)
    a = rng.uniform(0.2, 0.9, T)
    base = _fwd(x, a, b, c, block)
    for j in range(T):
        xp = x.copy()
        xp[j] += 1.0
        changed = np.abs(_fwd(xp, a, b, c, block) - base)[:, 0] > 0
        expect = np.array([brute.window_start(i, block) <= j <= i for i in range(T)])
        assert np.array_equal(changed, expect), j


def test_batched_layout_matches_slices(rng):
    B, T, H, D, block = 2, 19, 3, 2, 4
    x, b, c, dy = (rng.standard_normal((B, T, H, D)) for _ in range(4))
    a = rng.uniform(0, 1, (B, T, H))
    y = oracle.forward(x, a, b, c, block)
    dx, da, db, dc = oracle.backward(x, a, b, c, dy, block)
    for bi in range(B):
        for h in range(H):
            ys = brute.swr_slice(x[bi, :, h], a[bi, :, h], b[bi, :, h], c[bi, :, h], block)
            np.testing.assert_allclose(y[bi, :, h], ys, rtol=1e-12, atol=1e-12)
            g = _bwd(x[bi, :, h], a[bi, :, h], b[bi, :, h], c[bi, :, h], dy[bi, :, h], block)
            for full, one in zip((dx, da, db, dc), g):
                np.testing.assert_array_equal(full[bi, :, h], one)


# --------------------------------------------------------------------------- backward


@pytest.mark.parametrize("T,D,block", [(1, 1, 1), (6, 2, 1), (9, 2, 2), (13, 3, 4), (20, 2, 8),
                                       (17, 1, 16)])
@pytest.mark.parametrize("per_channel", [False, True])
@pytest.mark.parametrize("residual", [False, True])
def test_backward_equals_autograd(rng, T, D, block, per_channel, residual):
    x, a, b, c = _inputs(rng, T, D, per_channel)
    dy = rng.standard_normal((T, D))
    got = _bwd(x, a, b, c, dy, block, residual)
    ref = brute.torch_grads(x, a, b, c, dy, block, residual)
    for name, g, r in zip(("dx", "da", "db", "dc"), got, ref):
        np.testing.assert_allclose(g, r, rtol=1e-11, atol=1e-12, err_msg=name)


def test_backward_finite_differences(rng):
    T, D, block = 14, 2, 4
    x, a, b, c = _inputs(rng, T, D, zeros=False)
    dy = rng.standard_normal((T, D))
    grads = dict(zip("xabc", _bwd(x, a, b, c, dy, block)))
    args = dict(x=x, a=a, b=b, c=c)
    eps = 1e-6

    def loss(**kw):
        v = {**args, **kw}
        return float(np.sum(dy * _fwd(v["x"], v["a"], v["b"], v["c"], block)))

    for name in "xabc":
        base = args[name]
        fd = np.zeros_like(base)
        for idx in np.ndindex(base.shape):
            p, m = base.copy(), base.copy()
            p[idx] += eps
            m[idx] -= eps
            fd[idx] = (loss(**{name: p}) - loss(**{name: m})) / (2 * eps)
        np.testing.assert_allclose(grads[name], fd, rtol=1e-6, atol=1e-7, err_msg=name)


def test_backward_adjoint_identities(rng):
    # y is linear in each of x, b and c separately, so <dy, y> = <dz, z> for z in {x, b, c}.
    T, D, block = 29, 3, 4
    x, a, b, c = _inputs(rng, T, D)
    dy = rng.standard_normal((T, D))
    dx, da, db, dc = _bwd(x, a, b, c, dy, block)
    ydy = np.sum(dy * _fwd(x, a, b, c, block))
    for g, z in ((dx, x), (db, b), (dc, c)):
        assert np.isclose(np.sum(g * z), ydy, rtol=1e-12, atol=1e-12)
    # and the u-adjoint is the transpose of the jagged operator.
    Lt = brute.dense_Ltilde(a, block)
    np.testing.assert_allclose(dx / np.where(b == 0, 1, b), Lt.T @ (c * dy), rtol=1e-9, atol=1e-10)


def test_backward_decay_zero_closed_form(rng):
    # a == 0: da_k = sum_mu c_k dy_k u_{k-1} (0 at k = 0); du = c * dy.
    T, D, block = 25, 3, 4
    x, _, b, c = _inputs(rng, T, D)
    dy = rng.standard_normal((T, D))
    dx, da, db, dc = _bwd(x, np.zeros(T), b, c, dy, block)
    u = b * x
    ref_da = np.zeros(T)
    ref_da[1:] = np.sum(c[1:] * dy[1:] * u[:-1], axis=1)
    np.testing.assert_allclose(da, ref_da, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(dx, b * c * dy, rtol=1e-15)
    np.testing.assert_allclose(dc, dy * u, rtol=1e-15)


@pytest.mark.parametrize("block", [2, 4])
def test_backward_equals_untruncated_when_T_le_2l(rng, block):
    T, D = 2 * block, 2
    x, a, b, c = _inputs(rng, T, D, zeros=False)
    dy = rng.standard_normal((T, D))
    got = _bwd(x, a, b, c, dy, block)
    ref = brute.torch_grads(x, a, b, c, dy, block, truncated=False)
    for g, r in zip(got, ref):
        np.testing.assert_allclose(g, r, rtol=1e-11, atol=1e-12)


def test_rejects_bad_arguments():
    x = np.zeros((1, 4, 2))
    with pytest.raises(ValueError):
        oracle.forward_slices(x, np.zeros((1, 4)), x, x, block=0)


def test_empty_sequence():
    x = np.zeros((2, 0, 3))
    assert oracle.forward_slices(x, np.zeros((2, 0)), x, x, block=4).shape == (2, 0, 3)


@pytest.mark.parametrize("T,D,block", [(37, 3, 8), (100, 5, 16), (64, 2, 64)])
def test_channel_constant_per_channel_decay_is_shared_decay(rng, T, D, block):
    # The per-channel recurrence with the same decay on every channel is the
    # shared-decay recurrence (eq. (2.1) with a scalar transition): identical
    # outputs and input gradients, and the shared decay's gradient is the sum
    # over channels of the per-channel one (chain rule through the broadcast).
    x, a, b, c = _inputs(rng, T, D)
    dy = rng.standard_normal((T, D))
    ab = np.repeat(a[:, None], D, axis=1)
    y1 = oracle.forward_slices(x[None], a[None], b[None], c[None], block)
    y2 = oracle.forward_slices(x[None], ab[None], b[None], c[None], block)
    np.testing.assert_allclose(y2, y1, rtol=1e-13, atol=1e-13)
    g1 = oracle.backward_slices(x[None], a[None], b[None], c[None], dy[None], block)
    g2 = oracle.backward_slices(x[None], ab[None], b[None], c[None], dy[None], block)
    for i in (0, 2, 3):
        np.testing.assert_allclose(g2[i], g1[i], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(g2[1].sum(axis=-1), g1[1], rtol=1e-12, atol=1e-12)


# ----------------------------------------------------------------------------- featurisation


def test_sigmoid_values():
    # closed forms and the symmetry sigma(-z) = 1 - sigma(z), including the tails
    z = np.array([-800.0, -40.0, -1.0, 0.0, 1.0, 40.0, 800.0])
    s = oracle.sigmoid(z)
    assert s[3] == 0.5 and s[0] == 0.0 and s[-1] == 1.0
    np.testing.assert_allclose(s[4], 1.0 / (1.0 + np.exp(-1.0)), rtol=1e-15)
    np.testing.assert_allclose(oracle.sigmoid(-z) + s, 1.0, rtol=0, atol=1e-15)
    np.testing.assert_allclose(oracle.dsigmoid(0.0), 0.25, rtol=1e-15)
    assert np.all(np.isfinite(oracle.dsigmoid(z)))


@pytest.mark.parametrize("sig_a,sig_b", [(True, False), (False, True), (True, True)])
@pytest.mark.parametrize("per_channel", [False, True])
def test_featurised_gradients_by_finite_differences(rng, sig_a, sig_b, per_channel):
    # d/dz of sum(dy * y(sigma(z_a), sigma(z_b))) by central differences on a few entries
    B, T, H, D, block = 1, 23, 2, 3, 8
    x, c, dy = (rng.standard_normal((B, T, H, D)) for _ in range(3))
    za = rng.standard_normal((B, T, H, D) if per_channel else (B, T, H)) * 2.0
    zb = rng.standard_normal((B, T, H, D)) * 2.0
    kw = dict(sigmoid_decay=sig_a, sigmoid_pregate=sig_b)
    dx, da, db, dc = oracle.backward(x, za, zb, c, dy, block, **kw)

    def loss(za_, zb_):
        return float(np.sum(dy * oracle.forward(x, za_, zb_, c, block, **kw)))

    h = 1e-6
    for idx in [(0, 0, 0), (0, 5, 1), (0, 22, 1)]:
        full = idx + ((1,) if per_channel else ())
        e = np.zeros_like(za); e[full] = h
        fd = (loss(za + e, zb) - loss(za - e, zb)) / (2 * h)
        np.testing.assert_allclose(da[full], fd, rtol=1e-6, atol=1e-8)
        e = np.zeros_like(zb); e[idx + (2,)] = h
        fd = (loss(za, zb + e) - loss(za, zb - e)) / (2 * h)
        np.testing.assert_allclose(db[idx + (2,)], fd, rtol=1e-6, atol=1e-8)


def test_featurised_equals_plain_on_sigmoid_values(rng):
    # the featurised call on logits z is the plain call on sigma(z); gradients
    # differ exactly by the factor sigma'(z)
    B, T, H, D, block = 2, 40, 2, 4, 16
    x, c, dy = (rng.standard_normal((B, T, H, D)) for _ in range(3))
    za, zb = rng.standard_normal((B, T, H)), rng.standard_normal((B, T, H, D))
    a, b = 1.0 / (1.0 + np.exp(-za)), 1.0 / (1.0 + np.exp(-zb))
    y1 = oracle.forward(x, za, zb, c, block, sigmoid_decay=True, sigmoid_pregate=True)
    np.testing.assert_allclose(y1, oracle.forward(x, a, b, c, block), rtol=1e-13, atol=1e-13)
    g1 = oracle.backward(x, za, zb, c, dy, block, sigmoid_decay=True, sigmoid_pregate=True)
    g0 = oracle.backward(x, a, b, c, dy, block)
    np.testing.assert_allclose(g1[1], g0[1] * a * (1 - a), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(g1[2], g0[2] * b * (1 - b), rtol=1e-12, atol=1e-13)
    for i in (0, 3):
        np.testing.assert_allclose(g1[i], g0[i], rtol=1e-13, atol=1e-13)
