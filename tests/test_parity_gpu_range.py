"""GPU parity at the ends of the floating-point range.

Two regimes, each made by scaling seeded N(0, 1) draws by powers of two (exact
in both I/O dtypes):

* small: x and b scaled by 2^-62, so u = b * x is about 2^-124, next to the
  smallest normal float32 (2^-126).  The low halves of the split-bf16 MFMA
  operands of u are then bf16 denormals, outputs reach the denormal range of
  the I/O dtype, and the decays are small (sigmoid(N(-4, 1)) ~ 0.02), so
  products of decays underflow to zero within a block.
* large: x and b scaled by 2^60 and c by 2^-2, with decays near 1
  (sigmoid(N(3, 1))), so that the states (and dc) reach about 2^126, y about
  2^123 and da about 2^126: a few binades below the largest finite bf16 /
  float32 value (about 2^128).

Each case first checks on the oracle's result that it really sits in its
regime (finite, below 2^127.5, and for the large regime above 2^120), then
compares every output with the oracle under the usual scaled metric.
"""
import sys

import numpy as np
import pytest

import oracle
import workloads as W
from parity import assert_close, to_device, to_host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

REGIMES = {
    # name: (log2 scale of x and b, log2 scale of c, mean of the decay's logit)
    "small": (-62, 0, -4.0),
    "large": (60, -2, 3.0),
}
TOP = 2.0 ** 127.5


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def swr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2512_13921_amd as lib
    lib.load()
    return lib


def _problem(regime, seed, B, T, H, D, block, dtype, per_channel=False, group=1):
    sx, sc, mu = REGIMES[regime]
    p = W.random_problem(seed, B, T, H, D, block, dtype, "sigmoid", mu, per_channel=per_channel)
    fx, fc = np.float32(2.0 ** sx), np.float32(2.0 ** sc)
    b = p.b[:, :, ::group] if group > 1 else p.b
    c = p.c[:, :, ::group] if group > 1 else p.c
    # powers of two: the scaled values are still exactly representable
    return W.Problem(p.cfg, p.x * fx, p.a, np.ascontiguousarray(b * fx), np.ascontiguousarray(c * fc), p.dy)


def _check_regime(regime, refs):
    for name, r in refs.items():
        r = np.asarray(r)
        assert np.isfinite(r).all(), name
        assert np.abs(r).max() < TOP, (name, np.log2(np.abs(r).max()))
    if regime == "large":
        assert np.abs(np.asarray(refs["y"])).max() > 2.0 ** 120
    else:
        assert np.abs(np.asarray(refs["y"])).max() < 2.0 ** -100


def _compare(regime, dtype, outs, refs, what):
    _check_regime(regime, refs)
    for name, t in outs.items():
        st = assert_close(to_host(t), refs[name], dtype, f"{what} {name}")
        _say(f"[range] {what} {name}: max_e={st['max_e']:.2e} mean_e={st['mean_e']:.2e}")


def _dev(prob, dt, names):
    return [to_device(getattr(prob, n), dt) for n in names]


@pytest.mark.parametrize("regime", sorted(REGIMES))
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("D,block", [(64, 64), (128, 128), (16, 16)])
def test_jagged_window_range(swr, regime, dtype, D, block):
    prob = _problem(regime, 31, 2, 1000, 2, D, block, dtype)
    _say(f"[range] jagged {regime} {dtype} D={D} l={block}")
    x, a, b, c, dy = _dev(prob, dtype, "x a b c dy".split())
    y, v = swr.swr_forward(x, a, b, c, block, save_carriers=True)
    grads = swr.swr_backward(x, a, b, c, dy, v, block)
    torch.cuda.synchronize()
    refs = dict(y=oracle.forward(prob.x, prob.a, prob.b, prob.c, block))
    refs.update(zip(("dx", "da", "db", "dc"), oracle.backward(prob.x, prob.a, prob.b, prob.c, prob.dy, block)))
    _compare(regime, dtype, dict(zip(("y", "dx", "da", "db", "dc"), (y,) + tuple(grads))), refs,
             f"jagged {regime} {dtype} D={D}")


@pytest.mark.parametrize("regime", sorted(REGIMES))
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_per_channel_decay_range(swr, regime, dtype):
    prob = _problem(regime, 32, 2, 700, 2, 128, 128, dtype, per_channel=True)
    _say(f"[range] per-channel {regime} {dtype}")
    x, a, b, c, dy = _dev(prob, dtype, "x a b c dy".split())
    y, v = swr.swr_forward(x, a, b, c, 128, save_carriers=True)
    grads = swr.swr_backward(x, a, b, c, dy, v, 128)
    torch.cuda.synchronize()
    refs = dict(y=oracle.forward(prob.x, prob.a, prob.b, prob.c, 128))
    refs.update(zip(("dx", "da", "db", "dc"), oracle.backward(prob.x, prob.a, prob.b, prob.c, prob.dy, 128)))
    _compare(regime, dtype, dict(zip(("y", "dx", "da", "db", "dc"), (y,) + tuple(grads))), refs,
             f"per-channel {regime} {dtype}")


@pytest.mark.parametrize("regime", sorted(REGIMES))
@pytest.mark.parametrize("dtype,D,k", [("bf16", 128, 128), ("f32", 64, 64)])
def test_uniform_window_range(swr, regime, dtype, D, k):
    prob = _problem(regime, 33, 2, 700, 2, D, k, dtype)
    _say(f"[range] uniform {regime} {dtype} D={D} k={k}")
    x, a, b, c, dy = _dev(prob, dtype, "x a b c dy".split())
    y = swr.swr_uniform_forward(x, a, b, c, k)
    grads = swr.swr_uniform_backward(x, a, b, c, dy, k)
    torch.cuda.synchronize()
    refs = dict(y=oracle.uniform_forward(prob.x, prob.a, prob.b, prob.c, k))
    refs.update(zip(("dx", "da", "db", "dc"),
                    oracle.uniform_backward(prob.x, prob.a, prob.b, prob.c, prob.dy, k)))
    _compare(regime, dtype, dict(zip(("y", "dx", "da", "db", "dc"), (y,) + tuple(grads))), refs,
             f"uniform {regime} {dtype} D={D}")


@pytest.mark.parametrize("regime", sorted(REGIMES))
def test_exact_recurrence_range(swr, regime):
    prob = _problem(regime, 34, 2, 1000, 2, 128, 128, "bf16")
    sx, _, _ = REGIMES[regime]
    rng = np.random.default_rng(34)
    # initial state at the scale of u = b * x
    h0 = (rng.standard_normal((2, 2, 128)) * 2.0 ** (2 * sx)).astype(np.float32)
    dhl = rng.standard_normal((2, 2, 128)).astype(np.float32)
    _say(f"[range] exact {regime}")
    x, a, b, c, dy = _dev(prob, "bf16", "x a b c dy".split())
    h0_t, dhl_t = torch.from_numpy(h0).cuda(), torch.from_numpy(dhl).cuda()
    y, v, hl = swr.swr_exact_forward(x, a, b, c, 128, h0=h0_t, save_carriers=True, want_h_last=True)
    grads = swr.swr_exact_backward(x, a, b, c, dy, v, 128, h0=h0_t, dh_last=dhl_t, want_dh0=True)
    torch.cuda.synchronize()
    ry, rhl = oracle.exact_forward(prob.x, prob.a, prob.b, prob.c, h0)
    refs = dict(y=ry, h_last=rhl)
    refs.update(zip(("dx", "da", "db", "dc", "dh0"),
                    oracle.exact_backward(prob.x, prob.a, prob.b, prob.c, prob.dy, h0, dhl)))
    outs = dict(zip(("y", "h_last", "dx", "da", "db", "dc", "dh0"), (y, hl) + tuple(grads)))
    _compare(regime, "bf16", outs, refs, f"exact {regime}")


@pytest.mark.parametrize("regime", sorted(REGIMES))
def test_shared_gates_range(swr, regime):
    group = 2
    prob = _problem(regime, 35, 2, 900, 4, 128, 128, "bf16", group=group)
    _say(f"[range] shared gates {regime}")
    x, a, b, c, dy = _dev(prob, "bf16", "x a b c dy".split())
    y, v = swr.swr_forward_shared_gates(x, a, b, c, 128, group, save_carriers=True)
    grads = swr.swr_backward_shared_gates(x, a, b, c, dy, v, 128, group)
    torch.cuda.synchronize()
    refs = dict(y=oracle.grouped_forward(prob.x, prob.a, prob.b, prob.c, 128, group))
    refs.update(zip(("dx", "da", "db", "dc"),
                    oracle.grouped_backward(prob.x, prob.a, prob.b, prob.c, prob.dy, 128, group)))
    _compare(regime, "bf16", dict(zip(("y", "dx", "da", "db", "dc"), (y,) + tuple(grads))), refs,
             f"shared gates {regime}")
