"""GPU parity for head widths other than the kernels' own (16, 32, 64, 128):
any D that is a multiple of 16 up to 256.  A head narrower than the kernel
width leaves lanes idle; a head wider than 128 channels (64 with a
per-channel decay) runs as two (four) virtual heads whose decay-gradient
shares meet in two atomic adds onto a zeroed da.  Forward, carriers and
backward (with and without saved carriers) against the oracle."""
import sys

import numpy as np
import pytest

import workloads as W
from parity import check_full, run_gpu, to_device, to_host

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


def _both(swr, prob, **kw):
    y, with_v = run_gpu(swr, prob, **kw)
    _, without_v = run_gpu(swr, prob, carriers=False, **kw)
    for name, g1, g2 in zip(("dx", "da", "db", "dc"), with_v, without_v):
        assert torch.equal(g1, g2), f"{name} differs without carriers"
    return y, without_v


SHARED = [
    # (B, T, H, D, block, dtype)
    (2, 517, 3, 48, 64, "bf16"),
    (1, 333, 2, 48, 16, "f32"),
    (2, 300, 2, 80, 128, "bf16"),
    (1, 700, 2, 96, 32, "f32"),
    (2, 400, 2, 112, 64, "bf16"),
    (1, 300, 2, 144, 128, "bf16"),
    (1, 257, 3, 192, 16, "f32"),
    (2, 500, 2, 208, 64, "bf16"),
    (1, 640, 2, 256, 128, "bf16"),
    (1, 200, 2, 256, 32, "f32"),
    (1, 1, 1, 240, 64, "bf16"),
]


@pytest.mark.parametrize("B,T,H,D,block,dtype", SHARED)
@pytest.mark.parametrize("run_len", [0, "min"])
def test_widths_shared_decay(swr, B, T, H, D, block, dtype, run_len):
    rl = max(64, block) if run_len == "min" else 0
    prob = W.random_problem(41 + T + D, B, T, H, D, block, dtype, "sigmoid", 1.5)
    _say(f"[width] B={B} T={T} H={H} D={D} l={block} {dtype} run_len={rl}")
    y, grads = _both(swr, prob, run_len=rl)
    check_full(prob, y, grads, what=f"width {B}x{T}x{H}x{D} l{block} {dtype}")


PER_CHANNEL = [
    (2, 400, 2, 48, 64, "bf16"),
    (1, 300, 2, 80, 32, "f32"),
    (1, 500, 2, 144, 128, "bf16"),
    (2, 300, 2, 256, 16, "bf16"),
    (1, 129, 3, 208, 64, "f32"),
]


@pytest.mark.parametrize("B,T,H,D,block,dtype", PER_CHANNEL)
def test_widths_per_channel_decay(swr, B, T, H, D, block, dtype):
    prob = W.random_problem(42 + T + D, B, T, H, D, block, dtype, per_channel=True)
    _say(f"[width, per channel] B={B} T={T} H={H} D={D} l={block} {dtype}")
    y, grads = _both(swr, prob, run_len=max(64, block))
    check_full(prob, y, grads, what=f"width pc {B}x{T}x{H}x{D} l{block} {dtype}")


@pytest.mark.parametrize("D", [96, 256])
def test_widths_flags_and_strided_layout(swr, D):
    prob = W.random_problem(43 + D, 2, 384, 2, D, 64, "bf16", logits=True)
    feat = dict(sigmoid_decay=True, sigmoid_pregate=True)
    y, grads = _both(swr, prob, residual=True, layout="bhtd", **feat)
    check_full(prob, y, grads, residual=True, what=f"width {D} residual bhtd featurised", **feat)


@pytest.mark.parametrize("D,block,dtype", [(96, 64, "bf16"), (144, 32, "f32"), (256, 128, "bf16")])
def test_widths_block_carriers(swr, D, block, dtype):
    # every block's carrier against its definition (the block's local solve
    # from zero, in float64)
    prob = W.random_problem(44 + D, 2, 517, 3, D, block, dtype)
    x, a, b, c = (to_device(getattr(prob, n), dtype) for n in "xabc")
    _, v1 = swr.swr_forward(x, a, b, c, block, save_carriers=True, run_len=max(64, block))
    v2 = swr.swr_carriers(x, a, b, block)
    torch.cuda.synchronize()
    assert torch.equal(v1, v2)
    cfg = prob.cfg
    nb = -(-cfg.T // block)
    u = prob.b.astype(np.float64) * prob.x.astype(np.float64)
    av = prob.a.astype(np.float64)
    ref = np.zeros((cfg.B, cfg.H, nb, cfg.D))
    for t in range(nb):
        s = np.zeros((cfg.B, cfg.H, cfg.D))
        for m in range(t * block, min((t + 1) * block, cfg.T)):
            s = av[:, m, :, None] * s + u[:, m]
        ref[:, :, t] = s
    scale = np.sqrt(np.mean(ref * ref))
    err = np.abs(to_host(v1) - ref) / np.maximum(np.abs(ref), scale)
    assert err.max() < 1e-4, err.max()


def test_split_heads_deterministic(swr):
    # the two virtual heads' decay-gradient shares meet in atomic adds onto
    # zero: two addends give the same sum in either order
    prob = W.random_problem(45, 2, 4096, 4, 256, 128, "bf16")
    _, g1 = run_gpu(swr, prob)
    _, g2 = run_gpu(swr, prob)
    for p_, q in zip(g1, g2):
        assert torch.equal(p_, q)


def test_wide_heads_medium_size(swr):
    # several thousand tokens per sequence, many runs per sequence
    prob = W.random_problem(46, 2, 8192, 4, 192, 128, "bf16", "exp_softplus")
    _say("[width] medium B=2 T=8192 H=4 D=192 l=128 bf16")
    y, grads = run_gpu(swr, prob)
    check_full(prob, y, grads, what="width 192 medium")
