"""Pins of the oracle's shared gates (Sec. 5, "Gate sharing across heads":
heads of a group share the pre-gate b and the post-gate c): the forward
against the window sums of every head with its group's gates, and the
gradients of the shared gates against torch autograd through one shared
leaf per group (float64)."""
import numpy as np
import pytest

import brute
import oracle


def _inputs(rng, B, T, H, D, group):
    G = H // group
    x = rng.standard_normal((B, T, H, D))
    a = rng.uniform(0.0, 1.0, (B, T, H))
    b = rng.standard_normal((B, T, G, D))
    c = rng.standard_normal((B, T, G, D))
    dy = rng.standard_normal((B, T, H, D))
    return x, a, b, c, dy


@pytest.mark.parametrize("H,group", [(4, 1), (4, 2), (6, 3), (4, 4)])
@pytest.mark.parametrize("block", [2, 4])
def test_grouped_forward_equals_window_sums(rng, H, group, block):
    B, T, D = 2, 11, 3
    x, a, b, c, _ = _inputs(rng, B, T, H, D, group)
    y = oracle.grouped_forward(x, a, b, c, block, group)
    for bi in range(B):
        for h in range(H):
            g = h // group
            ref = brute.swr_slice(x[bi, :, h], a[bi, :, h], b[bi, :, g], c[bi, :, g], block)
            np.testing.assert_allclose(y[bi, :, h], ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("H,group", [(4, 2), (6, 3), (2, 2)])
@pytest.mark.parametrize("sigmoid", [False, True])
@pytest.mark.parametrize("residual", [False, True])
def test_grouped_backward_equals_autograd(rng, H, group, sigmoid, residual):
    import torch
    B, T, D, block = 1, 9, 2, 4
    x, a, b, c, dy = _inputs(rng, B, T, H, D, group)
    tx, ta, tb, tc = (torch.tensor(v, requires_grad=True) for v in (x, a, b, c))
    ys = []
    for h in range(H):
        g = h // group
        av = torch.sigmoid(ta[0, :, h]) if sigmoid else ta[0, :, h]
        bv = torch.sigmoid(tb[0, :, g]) if sigmoid else tb[0, :, g]
        ys.append(brute.torch_forward(tx[0, :, h], av, bv, tc[0, :, g], block, residual))
    y = torch.stack(ys, 1)[None]
    (y * torch.tensor(dy)).sum().backward()
    feat = dict(sigmoid_decay=sigmoid, sigmoid_pregate=sigmoid)
    np.testing.assert_allclose(oracle.grouped_forward(x, a, b, c, block, group, residual, **feat),
                               y.detach().numpy(), rtol=1e-12, atol=1e-12)
    got = oracle.grouped_backward(x, a, b, c, dy, block, group, residual, **feat)
    for name, g_, t in zip(("dx", "da", "db", "dc"), got, (tx, ta, tb, tc)):
        np.testing.assert_allclose(g_, t.grad.numpy(), rtol=1e-10, atol=1e-11, err_msg=name)


def test_group_of_one_is_the_plain_recurrence(rng):
    x, a, b, c, dy = _inputs(rng, 1, 20, 3, 2, 1)
    np.testing.assert_array_equal(oracle.grouped_forward(x, a, b, c, 4, 1), oracle.forward(x, a, b, c, 4))
    for g_, r in zip(oracle.grouped_backward(x, a, b, c, dy, 4, 1), oracle.backward(x, a, b, c, dy, 4)):
        np.testing.assert_array_equal(g_, r)
