"""GPU parity of the uniform window (Sec. 4.1: every token sees its k most
recent tokens, k = block): the HIP library through its C ABI binding against
the double-precision oracle on the same seeded, rounded inputs."""
import sys

import numpy as np
import pytest

import oracle
import workloads as W
from parity import assert_close, compare_whole, to_device, to_host, workload

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


def _run(swr, prob, residual=False, run_len=0, layout="bthd", backward=True, **feat):
    cfg = prob.cfg
    dt = cfg.dtype
    x, b, c, a = (to_device(getattr(prob, n), dt) for n in ("x", "b", "c", "a"))
    dy = to_device(prob.dy, dt) if backward else None
    if layout == "bhtd":
        def bhtd(t):
            if t.dim() == 4:
                return t.permute(0, 2, 1, 3).contiguous().permute(0, 2, 1, 3)
            return t.permute(0, 2, 1).contiguous().permute(0, 2, 1)
        x, b, c, a = (bhtd(t) for t in (x, b, c, a))
        dy = bhtd(dy) if dy is not None else None
    y = swr.swr_uniform_forward(x, a, b, c, cfg.block, residual=residual, run_len=run_len, **feat)
    grads = (swr.swr_uniform_backward(x, a, b, c, dy, cfg.block, residual=residual, run_len=run_len, **feat)
             if backward else None)
    torch.cuda.synchronize()
    return y, grads


def _check(prob, y, grads, residual=False, what="", **feat):
    cfg = prob.cfg
    ref_y = oracle.uniform_forward(prob.x, prob.a, prob.b, prob.c, cfg.block, residual, **feat)
    assert_close(to_host(y), ref_y, cfg.dtype, what + " y")
    if grads is not None:
        ref = oracle.uniform_backward(prob.x, prob.a, prob.b, prob.c, prob.dy, cfg.block, residual, **feat)
        for name, g, r in zip(("dx", "da", "db", "dc"), grads, ref):
            assert_close(to_host(g), r, cfg.dtype, f"{what} {name}")


SMALL = [
    # (B, T, H, D, block, dtype)
    (1, 64, 1, 16, 16, "f32"),
    (2, 1000, 3, 64, 64, "f32"),
    (1, 333, 2, 128, 128, "f32"),
    (2, 517, 3, 32, 32, "f32"),
    (2, 1000, 3, 64, 64, "bf16"),
    (1, 777, 2, 128, 128, "bf16"),
    (2, 300, 5, 16, 16, "bf16"),
    (1, 513, 3, 32, 32, "bf16"),
    (1, 1024, 2, 128, 64, "bf16"),
    (1, 640, 2, 64, 128, "bf16"),
    (1, 1, 1, 64, 64, "bf16"),      # a single token
    (1, 17, 1, 128, 128, "bf16"),   # shorter than a sub-block ... a block
    (1, 130, 1, 16, 128, "f32"),
    (3, 300, 6, 128, 32, "f32"),
    (2, 450, 3, 128, 16, "bf16"),   # 16 tokens per window, padded head groups
]


@pytest.mark.parametrize("B,T,H,D,block,dtype", SMALL)
@pytest.mark.parametrize("run_len", [0, "min"])
def test_uniform_small_against_oracle(swr, B, T, H, D, block, dtype, run_len):
    rl = max(64, block) if run_len == "min" else 0    # "min": many runs, each with its halo
    prob = W.random_problem(11 + T + D, B, T, H, D, block, dtype, "sigmoid", 1.5)
    _say(f"[uniform] B={B} T={T} H={H} D={D} k={block} {dtype} run_len={rl}")
    y, grads = _run(swr, prob, run_len=rl)
    _check(prob, y, grads, what=f"uniform {B}x{T}x{H}x{D} k{block} {dtype}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_uniform_residual_and_layout(swr, dtype):
    prob = W.random_problem(3, 2, 400, 3, 128, 64, dtype)
    y, grads = _run(swr, prob, residual=True, layout="bhtd")
    assert y.stride() != y.contiguous().stride()
    _check(prob, y, grads, residual=True, what="uniform residual bhtd")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("block", [32, 128])
@pytest.mark.parametrize("flags", ["both", "decay", "pregate"])
def test_uniform_featurisation(swr, dtype, block, flags):
    prob = W.random_problem(4, 2, 500, 2, 64, block, dtype, logits=True)
    feat = dict(sigmoid_decay=flags != "pregate", sigmoid_pregate=flags != "decay")
    if not feat["sigmoid_decay"]:      # the kernels take the decay itself: hand them sigma(z)
        prob.a[...] = W.round_to(oracle.sigmoid(prob.a).astype(np.float32), dtype)
    y, grads = _run(swr, prob, **feat)
    _check(prob, y, grads, what=f"uniform featurised ({flags})", **feat)


def test_uniform_featurised_headline_width(swr):
    # 128 channels as two 64-channel halves, several runs of several steps:
    # the pre-gate's e^-z carried from step to step.
    prob = W.random_problem(5, 1, 1536, 2, 128, 128, "bf16", logits=True)
    feat = dict(sigmoid_decay=True, sigmoid_pregate=True)
    y, grads = _run(swr, prob, run_len=512, **feat)
    _check(prob, y, grads, what="uniform featurised d128 runs", **feat)


@pytest.mark.parametrize("value", [0.0, 1.0])
@pytest.mark.parametrize("block", [16, 64, 128])
def test_uniform_decay_closed_forms(swr, value, block):
    prob = W.random_problem(5, 1, 300, 2, 64, block, "f32")
    prob.a[...] = value
    y, grads = _run(swr, prob)
    _check(prob, y, grads, what=f"uniform a={value}")
    u = prob.b.astype(np.float64) * prob.x
    if value == 0.0:       # no memory: h = u
        np.testing.assert_allclose(to_host(y), prob.c * u, rtol=1e-6, atol=1e-6)


def test_uniform_zero_and_one_decays_mixed(swr):
    prob = W.random_problem(6, 2, 700, 2, 128, 64, "f32")
    rng = np.random.default_rng(0)
    mask = rng.uniform(size=prob.a.shape)
    prob.a[mask < 0.05] = 0.0
    prob.a[mask > 0.95] = 1.0
    y, grads = _run(swr, prob)
    _check(prob, y, grads, what="uniform mixed zeros and ones")


def test_uniform_deterministic(swr):
    # D = 128 adds the decay gradient of two 64-channel halves: still bitwise reproducible
    prob = W.random_problem(8, 2, 1500, 3, 128, 128, "bf16")
    y1, g1 = _run(swr, prob)
    y2, g2 = _run(swr, prob)
    assert torch.equal(y1, y2)
    for p_, q_ in zip(g1, g2):
        assert torch.equal(p_, q_)


def test_uniform_run_length_does_not_change_results_beyond_rounding(swr):
    prob = W.random_problem(9, 1, 2048, 2, 64, 64, "f32")
    ya, ga = _run(swr, prob, run_len=64)
    yb, gb = _run(swr, prob, run_len=1024)
    assert_close(to_host(ya), to_host(yb).astype(np.float64), "f32", "run length y")
    for p_, q_ in zip(ga, gb):
        assert_close(to_host(p_), to_host(q_), "f32", "run length grads")


def test_uniform_empty_inputs(swr):
    x = torch.zeros((0, 16, 2, 64), device="cuda", dtype=torch.bfloat16)
    a = torch.zeros((0, 16, 2), device="cuda", dtype=torch.bfloat16)
    y = swr.swr_uniform_forward(x, a, x, x, 64)
    assert y.shape == x.shape
    g = swr.swr_uniform_backward(x, a, x, x, x, 64)
    assert g[1].shape == a.shape


def test_uniform_wide_window_matches_exact_on_short_sequences(swr):
    # T <= k: nothing is truncated, the uniform window is the exact recurrence
    prob = W.random_problem(10, 2, 128, 2, 64, 128, "f32")
    y, _ = _run(swr, prob, backward=False)
    ref, _ = oracle.exact_forward(prob.x, prob.a, prob.b, prob.c)
    assert_close(to_host(y), ref, "f32", "uniform T <= k")


def test_uniform_headline_shape_whole_tensors(swr):
    """The headline shape (B=8, T=16384, H=16, d=128, k=128) in the default
    launch configuration; every element of every output is compared with the
    oracle."""
    cfg = W.CONFIGS[3]
    _say(f"[uniform headline] {cfg.name}: generating inputs")
    prob = workload(cfg)
    y, grads = _run(swr, prob)

    def ref_chunk(b, h0, h1):
        args = [np.asarray(getattr(prob, n))[b:b + 1, :, h0:h1] for n in ("x", "a", "b", "c")]
        ref = dict(y=oracle.uniform_forward(*args, cfg.block))
        ref.update(zip(("dx", "da", "db", "dc"),
                       oracle.uniform_backward(*args, prob.dy[b:b + 1, :, h0:h1], cfg.block)))
        return ref

    outs = [("y", y, 2, 1)] + [(n, g, 2, 1) for n, g in zip(("dx", "da", "db", "dc"), grads)]
    _say("[uniform headline] comparing whole tensors with the oracle")
    compare_whole(f"uniform k={cfg.block} {cfg.name}", cfg.dtype, cfg.B, cfg.H, outs, ref_chunk)


def test_uniform_autograd_function(swr):
    prob = W.random_problem(12, 2, 300, 2, 64, 32, "f32")
    x, a, b, c = (to_device(getattr(prob, n), "f32").requires_grad_(True) for n in ("x", "a", "b", "c"))
    y = swr.SWRUniformFunction.apply(x, a, b, c, 32)
    y.backward(to_device(prob.dy, "f32"))
    torch.cuda.synchronize()
    assert_close(to_host(y), oracle.uniform_forward(prob.x, prob.a, prob.b, prob.c, 32), "f32", "autograd y")
    ref = oracle.uniform_backward(prob.x, prob.a, prob.b, prob.c, prob.dy, 32)
    for name, t, r in zip(("dx", "da", "db", "dc"), (x, a, b, c), ref):
        assert_close(to_host(t.grad), r, "f32", f"autograd {name}")


def test_uniform_in_a_captured_graph(swr):
    # Forward and backward (d = 128: a zero fill of da, then two halves adding
    # to it) captured once in a HIP graph: every replay, with eager work and
    # synchronisations between replays, reproduces the eager results bit for bit.
    prob = W.random_problem(14, 2, 700, 2, 128, 64, "bf16")
    x, a, b, c, dy = (to_device(getattr(prob, n), "bf16") for n in ("x", "a", "b", "c", "dy"))
    y_e = swr.swr_uniform_forward(x, a, b, c, 64)
    g_e = swr.swr_uniform_backward(x, a, b, c, dy, 64)
    torch.cuda.synchronize()
    y = torch.empty_like(y_e)
    outs = tuple(torch.empty_like(t) for t in g_e)
    graph = torch.cuda.CUDAGraph()
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        with torch.cuda.graph(graph, stream=stream):
            swr.swr_uniform_forward(x, a, b, c, 64, y=y)
            swr.swr_uniform_backward(x, a, b, c, dy, 64, outputs=outs)
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()
    for rep in range(3):
        for t in (y,) + outs:
            t.fill_(7.0)                  # eager work between the replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y_e), rep
        for p_, q_ in zip(outs, g_e):
            assert torch.equal(p_, q_), rep
