"""GPU parity of the per-channel-decay path (a and da of shape [B, T, H, D],
SWR_FLAG_PER_CHANNEL_DECAY) against the double-precision oracle."""
import sys

import numpy as np
import pytest

import oracle
import workloads as W
from parity import assert_close, check_full, compare_whole, run_gpu, to_device, to_host, workload

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


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


def _problem(seed, B, T, H, D, block, dtype, **kw):
    return W.random_problem(seed, B, T, H, D, block, dtype, per_channel=True, **kw)


SMALL = [
    # (B, T, H, D, block, dtype)
    (1, 64, 1, 16, 16, "f32"),
    (2, 1000, 3, 64, 64, "f32"),
    (1, 333, 2, 128, 128, "f32"),     # D = 128: two 64-channel halves per head
    (2, 517, 2, 32, 32, "bf16"),
    (1, 777, 2, 128, 128, "bf16"),
    (2, 300, 2, 16, 16, "bf16"),
    (1, 1024, 2, 128, 64, "bf16"),
    (1, 640, 3, 64, 128, "bf16"),
    (1, 1, 1, 64, 64, "bf16"),        # a single token
    (1, 17, 1, 128, 128, "bf16"),     # shorter than one sub-block
    (2, 700, 3, 128, 32, "f32"),
]


@pytest.mark.parametrize("B,T,H,D,block,dtype", SMALL)
@pytest.mark.parametrize("run_len", [0, "min"])
def test_small_against_oracle(swr, B, T, H, D, block, dtype, run_len):
    rl = max(64, block) if run_len == "min" else 0     # "min": every step its own run
    prob = _problem(31 + T + D, B, T, H, D, block, dtype, a_mu=1.5)
    _say(f"[per-channel small] B={B} T={T} H={H} D={D} l={block} {dtype} run_len={rl}")
    y, grads = run_gpu(swr, prob, run_len=rl)
    assert grads[1].shape == y.shape and grads[1].dtype == torch.float32
    check_full(prob, y, grads, what=f"pc {B}x{T}x{H}x{D} l{block} {dtype}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_residual_and_strided_layout(swr, dtype):
    prob = _problem(3, 2, 400, 2, 128, 64, dtype)
    y, grads = run_gpu(swr, prob, residual=True, layout="bhtd")
    assert y.stride() != y.contiguous().stride()
    check_full(prob, y, grads, residual=True, what="pc residual bhtd")


@pytest.mark.parametrize("value", [0.0, 1.0])
def test_decay_closed_forms(swr, value):
    prob = _problem(11, 1, 500, 2, 64, 128, "f32")
    prob.a[...] = value
    y, grads = run_gpu(swr, prob)
    check_full(prob, y, grads, what=f"pc a={value}")
    if value == 0.0:
        np.testing.assert_allclose(to_host(y), (prob.c * prob.b * prob.x).astype(np.float64),
                                   rtol=1e-6, atol=1e-6)


def test_zero_and_unit_decays_mixed(swr):
    prob = _problem(12, 2, 700, 2, 128, 128, "bf16")
    mask = np.random.default_rng(0).random(prob.a.shape)
    prob.a[mask < 0.05] = 0.0
    prob.a[mask > 0.95] = 1.0
    y, grads = run_gpu(swr, prob)
    check_full(prob, y, grads, what="pc mixed zeros/ones")


def test_channel_constant_decay_matches_shared_decay(swr):
    # A per-channel decay that is the same on every channel is the shared
    # decay: y and dx/db/dc agree, and the shared da is the channel sum.
    shared = W.random_problem(41, 2, 600, 2, 64, 64, "f32")
    x, b, c, dy = (to_device(getattr(shared, n), "f32") for n in ("x", "b", "c", "dy"))
    a1 = to_device(shared.a, "f32")
    a2 = a1[..., None].expand(x.shape).contiguous()
    y1, v1 = swr.swr_forward(x, a1, b, c, 64, save_carriers=True)
    y2, v2 = swr.swr_forward(x, a2, b, c, 64, save_carriers=True)
    g1 = swr.swr_backward(x, a1, b, c, dy, v1, 64)
    g2 = swr.swr_backward(x, a2, b, c, dy, v2, 64)
    torch.cuda.synchronize()
    ref_y = oracle.forward(shared.x, shared.a, shared.b, shared.c, 64)
    ref = oracle.backward(shared.x, shared.a, shared.b, shared.c, shared.dy, 64)
    assert_close(to_host(y2), ref_y, "f32", "pc-constant y")
    assert_close(to_host(v2), to_host(v1), "f32", "pc-constant carriers")
    for name, i in (("dx", 0), ("db", 2), ("dc", 3)):
        assert_close(to_host(g2[i]), ref[i], "f32", f"pc-constant {name}")
    assert_close(to_host(g2[1]).sum(axis=-1), ref[1], "f32", "pc-constant da summed")


def _carriers_by_definition(prob):
    """v_t per channel: state at the end of block t of the recurrence restarted
    at the block's start (float64 loop)."""
    cfg = prob.cfg
    l, T = cfg.block, cfg.T
    nb = -(-T // l)
    u = prob.b.astype(np.float64) * prob.x.astype(np.float64)
    a = prob.a.astype(np.float64)
    v = np.zeros((cfg.B, cfg.H, nb, cfg.D))
    for t in range(nb):
        s = np.zeros((cfg.B, cfg.H, cfg.D))
        for m in range(t * l, min((t + 1) * l, T)):
            s = a[:, m] * s + u[:, m]
        v[:, :, t] = s
    return v


@pytest.mark.parametrize("dtype,D,block", [("bf16", 128, 128), ("f32", 64, 32), ("bf16", 16, 16)])
def test_block_carriers(swr, dtype, D, block):
    prob = _problem(21, 2, 517, 3, D, block, dtype)
    x, a, b, c = (to_device(getattr(prob, n), dtype) for n in "xabc")
    _, v1 = swr.swr_forward(x, a, b, c, block, save_carriers=True, run_len=max(64, block))
    v2 = swr.swr_carriers(x, a, b, block)
    torch.cuda.synchronize()
    assert torch.equal(v1, v2)
    ref = _carriers_by_definition(prob)
    scale = np.sqrt(np.mean(ref * ref))
    err = np.abs(to_host(v1) - ref) / np.maximum(np.abs(ref), scale)
    assert err.max() < 1e-4, err.max()


def test_deterministic(swr):
    prob = _problem(13, 2, 2048, 4, 128, 128, "bf16")
    y1, g1 = run_gpu(swr, prob)
    y2, g2 = run_gpu(swr, prob)
    assert torch.equal(y1, y2)
    for p_, q_ in zip(g1, g2):
        assert torch.equal(p_, q_)


def test_autograd_function(swr):
    prob = _problem(15, 1, 256, 2, 64, 64, "f32")
    x, a, b, c = (to_device(getattr(prob, n), "f32").requires_grad_() for n in "xabc")
    y = swr.SWRFunction.apply(x, a, b, c, 64)
    (y * to_device(prob.dy, "f32")).sum().backward()
    ref = oracle.backward(prob.x, prob.a, prob.b, prob.c, prob.dy, 64)
    for t, r, n in zip((x, a, b, c), ref, "xabc"):
        assert_close(to_host(t.grad), r, "f32", "pc autograd d" + n)


def test_tiny_workload_per_channel(swr):
    cfg = W.PER_CHANNEL[1]
    prob = W.generate(cfg, with_dy=True)
    _say(f"[per-channel] {cfg.name}")
    y, grads = run_gpu(swr, prob)
    check_full(prob, y, grads, what=cfg.name)


def test_headline_shape_per_channel_whole_tensors(swr):
    """B=8, T=16384, H=16, d=128, block 128 with per-channel decay, in the
    default launch configuration; every element of every output is compared
    with the oracle."""
    cfg = W.PER_CHANNEL[3]
    _say(f"[per-channel] {cfg.name}: generating inputs")
    prob = workload(cfg)
    y, grads = run_gpu(swr, prob)

    def ref_chunk(b, h0, h1):
        args = [np.asarray(getattr(prob, n))[b:b + 1, :, h0:h1] for n in ("x", "a", "b", "c")]
        ref = dict(y=oracle.forward(*args, cfg.block))
        ref.update(zip(("dx", "da", "db", "dc"),
                       oracle.backward(*args, prob.dy[b:b + 1, :, h0:h1], cfg.block)))
        return ref

    outs = [("y", y, 2, 1)] + [(n, g, 2, 1) for n, g in zip(("dx", "da", "db", "dc"), grads)]
    _say("[per-channel] comparing whole tensors with the oracle")
    compare_whole(f"per-channel {cfg.name}", cfg.dtype, cfg.B, cfg.H, outs, ref_chunk)
