"""GPU parity of the fused Phalanx featurisation (SWR_FLAG_SIGMOID_DECAY,
SWR_FLAG_SIGMOID_PREGATE): a and/or b are logits, the kernels apply the
sigmoid, and the backward returns gradients with respect to the logits."""
import sys

import numpy as np
import pytest

import oracle
import workloads as W
from parity import assert_close, check_full, compare_whole, run_gpu, to_device, to_host, workload

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

FEATS = [dict(sigmoid_decay=True, sigmoid_pregate=False),
         dict(sigmoid_decay=False, sigmoid_pregate=True),
         dict(sigmoid_decay=True, sigmoid_pregate=True)]


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


SMALL = [
    # (B, T, H, D, block, dtype, per_channel)
    (2, 1000, 3, 64, 64, "f32", False),
    (1, 333, 2, 128, 128, "f32", False),
    (1, 777, 2, 128, 128, "bf16", False),
    (2, 300, 2, 16, 16, "bf16", False),
    (1, 640, 3, 64, 128, "bf16", True),
    (2, 517, 2, 128, 32, "f32", True),
    (1, 17, 1, 128, 128, "bf16", True),
]


@pytest.mark.parametrize("B,T,H,D,block,dtype,per_channel", SMALL)
@pytest.mark.parametrize("feat", range(len(FEATS)))
def test_small_against_oracle(swr, B, T, H, D, block, dtype, per_channel, feat):
    kw = FEATS[feat]
    prob = W.random_problem(51 + T + D, B, T, H, D, block, dtype, a_mu=2.0,
                            per_channel=per_channel, logits=True)
    if not kw["sigmoid_decay"]:      # the kernels take the decay itself: hand them sigma(z)
        prob.a[...] = W.round_to(oracle.sigmoid(prob.a).astype(np.float32), dtype)
    _say(f"[feat] B={B} T={T} H={H} D={D} l={block} {dtype} pc={per_channel} {kw}")
    rl = max(64, block) if feat == 2 else 0      # one case per shape with minimal runs
    y, grads = run_gpu(swr, prob, run_len=rl, **kw)
    check_full(prob, y, grads, what=f"feat {kw}", **kw)


@pytest.mark.parametrize("per_channel", [False, True])
def test_extreme_logits(swr, per_channel):
    # saturated sigmoids (decay exactly 0 or 1 in float32) stay finite and exact
    prob = W.random_problem(61, 1, 400, 2, 64, 64, "f32", per_channel=per_channel, logits=True)
    rng = np.random.default_rng(1)
    pick = rng.random(prob.a.shape)
    prob.a[pick < 0.2] = -120.0
    prob.a[pick > 0.8] = 120.0
    prob.b[rng.random(prob.b.shape) < 0.1] = -120.0
    kw = FEATS[2]
    y, grads = run_gpu(swr, prob, **kw)
    check_full(prob, y, grads, what="extreme logits", **kw)


def test_featurised_matches_plain_kernels(swr):
    # sigmoid inside the kernel vs sigmoid applied beforehand (float32 on the
    # device): same outputs to float32 rounding, gradients related by sigma'
    prob = W.random_problem(62, 2, 512, 2, 64, 64, "f32", logits=True)
    x, za, zb, c, dy = (to_device(getattr(prob, n), "f32") for n in ("x", "a", "b", "c", "dy"))
    a, b = torch.sigmoid(za), torch.sigmoid(zb)
    y1, v1 = swr.swr_forward(x, za, zb, c, 64, save_carriers=True, **FEATS[2])
    y0, v0 = swr.swr_forward(x, a, b, c, 64, save_carriers=True)
    g1 = swr.swr_backward(x, za, zb, c, dy, v1, 64, **FEATS[2])
    g0 = swr.swr_backward(x, a, b, c, dy, v0, 64)
    torch.cuda.synchronize()
    assert_close(to_host(y1), to_host(y0), "f32", "y")
    assert_close(to_host(v1), to_host(v0), "f32", "carriers")
    assert_close(to_host(g1[0]), to_host(g0[0]), "f32", "dx")
    assert_close(to_host(g1[1]), to_host(g0[1] * a * (1 - a)), "f32", "da")
    assert_close(to_host(g1[2]), to_host(g0[2] * b * (1 - b)), "f32", "db")


def test_autograd_function(swr):
    prob = W.random_problem(63, 1, 256, 2, 64, 64, "f32", logits=True)
    x, a, b, c = (to_device(getattr(prob, n), "f32").requires_grad_() for n in "xabc")
    y = swr.SWRFunction.apply(x, a, b, c, 64, False, True, True)
    (y * to_device(prob.dy, "f32")).sum().backward()
    ref = oracle.backward(prob.x, prob.a, prob.b, prob.c, prob.dy, 64, **FEATS[2])
    for t, r, n in zip((x, a, b, c), ref, "xabc"):
        assert_close(to_host(t.grad), r, "f32", "feat autograd d" + n)


def test_full_size_whole_tensors_with_logits(swr):
    """B=8, T=4096, H=16, d=128, block 64 with the decay's logits N(3, 1) and
    pre-gate logits, both through the kernels' sigmoid; every element of every
    output is compared with the oracle."""
    cfg = W.CONFIGS[2].with_(logits=True)
    _say(f"[feat] {cfg.name} (logits): generating inputs")
    prob = workload(cfg)
    kw = FEATS[2]
    y, grads = run_gpu(swr, prob, **kw)

    def ref_chunk(b, h0, h1):
        args = [np.asarray(getattr(prob, n))[b:b + 1, :, h0:h1] for n in ("x", "a", "b", "c")]
        ref = dict(y=oracle.forward(*args, cfg.block, **kw))
        ref.update(zip(("dx", "da", "db", "dc"),
                       oracle.backward(*args, prob.dy[b:b + 1, :, h0:h1], cfg.block, **kw)))
        return ref

    outs = [("y", y, 2, 1)] + [(n, g, 2, 1) for n, g in zip(("dx", "da", "db", "dc"), grads)]
    _say("[feat] comparing whole tensors with the oracle")
    compare_whole(f"featurised {cfg.name} (logits)", cfg.dtype, cfg.B, cfg.H, outs, ref_chunk)
