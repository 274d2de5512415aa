"""GPU parity of the backward called as the paper's problem statement has it
(inputs and coefficients only, Alg. "Block Two-Pass"): swr_backward without
the forward's block carriers, which the kernels then recompute from the
previous block's x, b and a.  The gradients must equal those of the call
with saved carriers bit for bit (the same local solves and sub-block walk
as the forward), and match the oracle."""
import sys

import numpy as np
import pytest

import workloads as W
from parity import check_full, run_gpu, to_device, workload

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


CASES = [
    # (B, T, H, D, block, dtype)
    (1, 64, 1, 16, 16, "f32"),
    (2, 1000, 3, 64, 64, "f32"),
    (1, 333, 2, 128, 128, "f32"),
    (2, 517, 2, 32, 32, "f32"),
    (2, 1000, 3, 64, 64, "bf16"),
    (1, 777, 2, 128, 128, "bf16"),
    (2, 300, 3, 16, 16, "bf16"),
    (1, 513, 3, 32, 32, "bf16"),
    (1, 1024, 2, 128, 64, "bf16"),
    (1, 640, 2, 64, 128, "bf16"),
    (1, 1, 1, 64, 64, "bf16"),
    (1, 17, 1, 128, 128, "bf16"),
    (1, 130, 1, 16, 128, "f32"),
    (3, 300, 6, 128, 32, "f32"),
]


@pytest.mark.parametrize("B,T,H,D,block,dtype", CASES)
@pytest.mark.parametrize("run_len", [0, "min"])
def test_without_carriers_small(swr, B, T, H, D, block, dtype, run_len):
    rl = max(64, block) if run_len == "min" else 0   # "min": every step its own run
    prob = W.random_problem(31 + T + D, B, T, H, D, block, dtype, "sigmoid", 1.5)
    _say(f"[no carriers] B={B} T={T} H={H} D={D} l={block} {dtype} run_len={rl}")
    y, grads = _both(swr, prob, run_len=rl)
    check_full(prob, y, grads, what=f"no carriers {B}x{T}x{H}x{D} l{block} {dtype}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_without_carriers_residual_strided(swr, dtype):
    prob = W.random_problem(32, 2, 384, 3, 64, 64, dtype)
    y, grads = _both(swr, prob, residual=True, layout="bhtd")
    check_full(prob, y, grads, residual=True, what="no carriers residual bhtd")


@pytest.mark.parametrize("D,block", [(128, 128), (64, 64), (32, 16)])
def test_without_carriers_featurised(swr, D, block):
    prob = W.random_problem(33, 2, 700, 2, D, block, "bf16", logits=True)
    feat = dict(sigmoid_decay=True, sigmoid_pregate=True)
    y, grads = _both(swr, prob, **feat)
    check_full(prob, y, grads, what="no carriers featurised", **feat)


@pytest.mark.parametrize("D,block,dtype", [(128, 128, "bf16"), (64, 32, "f32"), (16, 16, "bf16")])
def test_without_carriers_per_channel(swr, D, block, dtype):
    prob = W.random_problem(34, 2, 600, 2, D, block, dtype, per_channel=True)
    y, grads = _both(swr, prob, run_len=max(64, block))
    check_full(prob, y, grads, what="no carriers per-channel")


@pytest.mark.parametrize("D", [16, 32])
def test_without_carriers_packed_small_heads(swr, D):
    # adjacent heads of 16 / 32 channels run packed on the per-channel kernels
    prob = W.random_problem(35, 2, 500, 8, D, 16, "bf16")
    y, grads = _both(swr, prob)
    check_full(prob, y, grads, what=f"no carriers packed d={D}")


def test_without_carriers_closed_forms(swr):
    prob = W.random_problem(36, 1, 700, 2, 128, 128, "bf16")
    rng = np.random.default_rng(0)
    mask = rng.random(prob.a.shape)
    prob.a[mask < 0.05] = 0.0
    prob.a[mask > 0.95] = 1.0
    y, grads = _both(swr, prob)
    check_full(prob, y, grads, what="no carriers mixed zeros/ones")


def test_without_carriers_autograd(swr):
    # the autograd wrapper with save_carriers=False keeps only the inputs
    prob = W.random_problem(37, 1, 300, 2, 64, 64, "f32")
    x, a, b, c = (to_device(getattr(prob, n), "f32").requires_grad_() for n in "xabc")
    y = swr.SWRFunction.apply(x, a, b, c, 64, False, False, False, False)   # save_carriers=False
    (y * to_device(prob.dy, "f32")).sum().backward()
    _, ref = run_gpu(swr, prob)
    for t, r, n in zip((x, a, b, c), ref, "xabc"):
        assert torch.equal(t.grad, r), n


@pytest.mark.parametrize("cid", [3, 5])
def test_without_carriers_full_size(swr, cid):
    """Full size, default launch configuration: bit-identical to the backward
    with saved carriers (which the whole-tensor oracle comparison covers)."""
    cfg = W.CONFIGS[cid]
    _say(f"[no carriers, config {cid}] {cfg.name}")
    prob = workload(cfg)
    dt = cfg.dtype
    x, a, b, c, dy = (to_device(getattr(prob, n), dt) for n in ("x", "a", "b", "c", "dy"))
    _, v = swr.swr_forward(x, a, b, c, cfg.block, save_carriers=True)
    g1 = swr.swr_backward(x, a, b, c, dy, v, cfg.block)
    g2 = swr.swr_backward(x, a, b, c, dy, None, cfg.block)
    torch.cuda.synchronize()
    for name, p, q in zip(("dx", "da", "db", "dc"), g1, g2):
        assert torch.equal(p, q), f"config {cid}: {name} differs without carriers"
