"""GPU parity of the gates shared by groups of heads (Sec. 5, "Gate sharing
across heads"): the HIP library through its C ABI binding against the
double-precision oracle on the same seeded, rounded inputs."""
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


def _gated(prob, group):
    # the gates of each group: those the problem drew for the group's first head
    return (np.ascontiguousarray(prob.b[:, :, ::group]), np.ascontiguousarray(prob.c[:, :, ::group]))


def _run(swr, prob, group, residual=False, run_len=0, gate_layout="btgd", backward=True, **feat):
    cfg = prob.cfg
    dt = cfg.dtype
    bg, cg = _gated(prob, group)
    x, a = to_device(prob.x, dt), to_device(prob.a, dt)
    b, c = to_device(bg, dt), to_device(cg, dt)
    if gate_layout == "bgtd":    # gates stored [B, G, T, D], handed over as a strided view
        b, c = (t.permute(0, 2, 1, 3).contiguous().permute(0, 2, 1, 3) for t in (b, c))
    y, v = swr.swr_forward_shared_gates(x, a, b, c, cfg.block, group, residual=residual, run_len=run_len,
                                        save_carriers=True, **feat)
    grads = None
    if backward:
        dy = to_device(prob.dy, dt)
        grads = swr.swr_backward_shared_gates(x, a, b, c, dy, v, cfg.block, group, residual=residual,
                                              run_len=run_len, **feat)
    torch.cuda.synchronize()
    return y, grads


def _check(prob, group, y, grads, residual=False, what="", **feat):
    cfg = prob.cfg
    bg, cg = _gated(prob, group)
    assert_close(to_host(y), oracle.grouped_forward(prob.x, prob.a, bg, cg, cfg.block, group, residual, **feat),
                 cfg.dtype, what + " y")
    if grads is not None:
        ref = oracle.grouped_backward(prob.x, prob.a, bg, cg, prob.dy, cfg.block, group, residual, **feat)
        for name, g, r in zip(("dx", "da", "db", "dc"), grads, ref):
            assert_close(to_host(g), r, cfg.dtype, f"{what} {name}")


SMALL = [
    # (B, T, H, D, block, dtype, group)
    (1, 64, 2, 16, 16, "f32", 2),
    (2, 1000, 4, 64, 64, "f32", 2),
    (1, 333, 4, 128, 128, "f32", 4),
    (2, 517, 6, 32, 32, "f32", 3),
    (2, 1000, 4, 64, 64, "bf16", 4),
    (1, 777, 4, 128, 128, "bf16", 2),
    (2, 300, 8, 16, 16, "bf16", 8),
    (1, 1024, 6, 128, 64, "bf16", 2),
    (1, 1, 2, 64, 64, "bf16", 2),      # a single token
    (3, 300, 4, 128, 32, "f32", 1),
    (1, 300, 32, 64, 64, "bf16", 16),  # the largest group summed inside the backward
    (1, 300, 32, 64, 64, "bf16", 32),  # larger groups: float32 shares in a workspace, then summed
    (1, 200, 32, 128, 128, "f32", 32),
]


@pytest.mark.parametrize("B,T,H,D,block,dtype,group", SMALL)
@pytest.mark.parametrize("run_len", [0, "min"])
def test_shared_gates_small_against_oracle(swr, B, T, H, D, block, dtype, group, run_len):
    rl = max(64, block) if run_len == "min" else 0
    prob = W.random_problem(13 + T + D, B, T, H, D, block, dtype, "sigmoid", 1.5)
    _say(f"[groups] B={B} T={T} H={H} D={D} l={block} {dtype} group={group} run_len={rl}")
    y, grads = _run(swr, prob, group, run_len=rl)
    _check(prob, group, y, grads, what=f"groups {B}x{T}x{H}x{D} l{block} {dtype} g{group}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_shared_gates_flags_and_layout(swr, dtype):
    prob = W.random_problem(21, 2, 500, 4, 128, 128, dtype, logits=True)
    feat = dict(sigmoid_decay=True, sigmoid_pregate=True)
    y, grads = _run(swr, prob, 2, residual=True, gate_layout="bgtd", **feat)
    _check(prob, 2, y, grads, residual=True, what="groups flags bgtd", **feat)


def test_group_of_one_matches_the_plain_calls(swr):
    prob = W.random_problem(22, 2, 700, 3, 128, 64, "bf16")
    y1, g1 = _run(swr, prob, 1)
    x, a, b, c, dy = (to_device(getattr(prob, n), "bf16") for n in ("x", "a", "b", "c", "dy"))
    y2, v = swr.swr_forward(x, a, b, c, 64, save_carriers=True)
    g2 = swr.swr_backward(x, a, b, c, dy, v, 64)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    for name, p_, q_ in zip(("dx", "da", "db", "dc"), g1, g2):
        if name == "da":   # a 128-channel head's da is summed as two halves here: rounding order only
            np.testing.assert_allclose(to_host(p_), to_host(q_), rtol=1e-5, atol=1e-5 * float(q_.abs().max()))
        else:
            assert torch.equal(p_, q_), name


@pytest.mark.parametrize("D", [64, 128])
def test_shared_gates_deterministic(swr, D):
    prob = W.random_problem(23, 2, 1500, 8, D, 128, "bf16")
    y1, g1 = _run(swr, prob, 4)
    y2, g2 = _run(swr, prob, 4)
    assert torch.equal(y1, y2)
    for p_, q_ in zip(g1, g2):
        assert torch.equal(p_, q_)


def test_shared_gates_headline_shape_whole_tensors(swr):
    """The headline shape (B=8, T=16384, H=16, d=128, l=128) with 8 gate groups
    of 2 heads; every element of y, dx, da and of the groups' db, dc is
    compared with the oracle."""
    cfg = W.CONFIGS[3]
    group = 2
    _say(f"[groups headline] {cfg.name}: generating inputs")
    prob = workload(cfg)
    y, grads = _run(swr, prob, group)
    bg, cg = _gated(prob, group)

    def ref_chunk(b, h0, h1):
        per_head = [np.asarray(getattr(prob, n))[b:b + 1, :, h0:h1] for n in ("x", "a", "dy")]
        bs, cs = bg[b:b + 1, :, h0 // group:h1 // group], cg[b:b + 1, :, h0 // group:h1 // group]
        xs, as_, dys = per_head
        ref = dict(y=oracle.grouped_forward(xs, as_, bs, cs, cfg.block, group))
        ref.update(zip(("dx", "da", "db", "dc"),
                       oracle.grouped_backward(xs, as_, bs, cs, dys, cfg.block, group)))
        return ref

    outs = [("y", y, 2, 1), ("dx", grads[0], 2, 1), ("da", grads[1], 2, 1),
            ("db", grads[2], 2, group), ("dc", grads[3], 2, group)]
    _say("[groups headline] comparing whole tensors with the oracle")
    compare_whole(f"shared gates {cfg.H // group}x{group} {cfg.name}", cfg.dtype, cfg.B, cfg.H, outs,
                  ref_chunk, quantum=group)


def test_shared_gates_autograd_function(swr):
    prob = W.random_problem(24, 2, 300, 4, 64, 64, "f32")
    group = 2
    bg, cg = _gated(prob, group)
    x, a = (to_device(getattr(prob, n), "f32").requires_grad_(True) for n in ("x", "a"))
    b, c = (to_device(v, "f32").requires_grad_(True) for v in (bg, cg))
    y = swr.SWRSharedGatesFunction.apply(x, a, b, c, 64, group)
    y.backward(to_device(prob.dy, "f32"))
    torch.cuda.synchronize()
    assert_close(to_host(y), oracle.grouped_forward(prob.x, prob.a, bg, cg, 64, group), "f32", "autograd y")
    ref = oracle.grouped_backward(prob.x, prob.a, bg, cg, prob.dy, 64, group)
    for name, t, r in zip(("dx", "da", "db", "dc"), (x, a, b, c), ref):
        assert_close(to_host(t.grad), r, "f32", f"autograd {name}")


def test_shared_gates_in_a_captured_graph(swr):
    prob = W.random_problem(25, 2, 600, 4, 128, 128, "bf16")
    group = 2
    bg, cg = _gated(prob, group)
    x, a, dy = (to_device(getattr(prob, n), "bf16") for n in ("x", "a", "dy"))
    b, c = to_device(bg, "bf16"), to_device(cg, "bf16")
    y_e, v = swr.swr_forward_shared_gates(x, a, b, c, 128, group, save_carriers=True)
    g_e = swr.swr_backward_shared_gates(x, a, b, c, dy, v, 128, group)
    torch.cuda.synchronize()
    y, v2 = torch.empty_like(y_e), torch.empty_like(v)
    outs = tuple(torch.empty_like(t) for t in g_e)
    graph = torch.cuda.CUDAGraph()
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        with torch.cuda.graph(graph, stream=stream):
            swr.swr_forward_shared_gates(x, a, b, c, 128, group, y=y, carriers=v2)
            swr.swr_backward_shared_gates(x, a, b, c, dy, v2, 128, group, outputs=outs)
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()
    for rep in range(3):
        for t in (y, v2) + outs:
            t.fill_(7.0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y_e), rep
        for p_, q_ in zip(outs, g_e):
            assert torch.equal(p_, q_), rep
