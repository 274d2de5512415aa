"""The allocation-free exact forward, swr_exact_forward_noalloc (its workspace
is the library's static device array), against swr_exact_forward with a
caller-provided workspace, both called through the C ABI on the same inputs:
consecutive calls, each smaller than the one before, whose outputs start out
as NaN; every call must give the same results bit for bit, and match the
oracle."""
import numpy as np
import pytest

import oracle
import workloads as W
from parity import assert_close, to_device, to_host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def swr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2512_13921_amd as lib
    lib.load()
    return lib


# (B, T, H, D, block, dtype, per-channel decay): each call smaller than the one before
CALLS = [
    (2, 3000, 4, 128, 128, "bf16", False),
    (1, 700, 2, 64, 64, "bf16", False),
    (1, 333, 3, 32, 32, "f32", True),
]


def _run_both(swr, seed, B, T, H, D, block, dtype, per_channel):
    prob = W.random_problem(seed, B, T, H, D, block, dtype, "sigmoid", 3.0, per_channel=per_channel)
    x, a, b, c = (to_device(getattr(prob, n), dtype) for n in "xabc")
    h0 = np.random.default_rng(seed).standard_normal((B, H, D)).astype(np.float32)
    h0_t = torch.from_numpy(h0).cuda()
    nb = -(-T // block)
    y = torch.full_like(x, float("nan"))
    v = torch.full((B, H, nb, D), float("nan"), dtype=torch.float32, device="cuda")
    hl = torch.full((B, H, D), float("nan"), dtype=torch.float32, device="cuda")
    out = swr.swr_exact_forward_noalloc(x, a, b, c, block, h0=h0_t, y=y, carriers=v, h_last=hl)
    assert out[0] is y and out[1] is v and out[2] is hl
    y2, v2, hl2 = swr.swr_exact_forward(x, a, b, c, block, h0=h0_t, save_carriers=True, want_h_last=True)
    torch.cuda.synchronize()
    return prob, h0, (y, v, hl), (y2, v2, hl2)


def test_noalloc_matches_the_workspace_call_on_consecutive_calls(swr):
    for i, call in enumerate(CALLS):
        B, T, H, D, block, dtype, pc = call
        print(f"[noalloc] call {i}: B={B} T={T} H={H} D={D} l={block} {dtype} per_channel={pc}", flush=True)
        prob, h0, got, ref = _run_both(swr, 70 + i, *call)
        for name, p_, q_ in zip(("y", "carriers", "h_last"), got, ref):
            assert torch.equal(p_, q_), (i, name)
        ry, rhl = oracle.exact_forward(prob.x, prob.a, prob.b, prob.c, h0)
        assert_close(to_host(got[0]), ry, dtype, f"noalloc call {i} y")
        assert_close(to_host(got[2]), rhl, dtype, f"noalloc call {i} h_last")


def test_noalloc_after_a_larger_call_on_another_stream(swr):
    # calls ordered through one stream after work on another stream that the
    # caller synchronised with: the array's contents from the earlier call do
    # not leak into the later one
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        _run_both(swr, 80, *CALLS[0])
    torch.cuda.current_stream().wait_stream(side)
    prob, h0, got, ref = _run_both(swr, 81, *CALLS[1])
    for name, p_, q_ in zip(("y", "carriers", "h_last"), got, ref):
        assert torch.equal(p_, q_), name


def test_noalloc_refuses_problems_beyond_the_static_array(swr):
    # refused during validation, before any HIP call: 65536 (batch, head)
    # sequences need more than the array for the one pass and the three stages
    x = torch.zeros((512, 64, 128, 128), dtype=torch.bfloat16, device="cuda")
    a = torch.zeros((512, 64, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(swr.SwrError) as err:
        swr.swr_exact_forward_noalloc(x, a, x, x, 128, y=torch.empty_like(x))
    assert err.value.code == swr.SWR_ERR_SCRATCH
    assert "SWR_NOALLOC_SCRATCH_BYTES" in str(err.value)


def test_noalloc_falls_back_to_the_three_stages(swr):
    # B16 T16384 H16 d128: the one pass needs 33.8 MB of workspace, more than
    # the static array, the three stages about 4 MB; the allocation-free call
    # runs the three stages and agrees with the one pass up to rounding
    g = torch.Generator(device="cuda").manual_seed(92)
    shape = (16, 16384, 16, 128)
    x, b, c = (torch.randn(shape, generator=g, device="cuda").to(torch.bfloat16) for _ in range(3))
    a = torch.sigmoid(2.0 + torch.randn(shape[:3], generator=g, device="cuda")).to(torch.bfloat16)
    y1, hl1 = swr.swr_exact_forward(x, a, b, c, 128, want_h_last=True)
    y2, hl2 = swr.swr_exact_forward_noalloc(x, a, b, c, 128, want_h_last=True)
    torch.cuda.synchronize()
    for name, u, w in (("y", y2, y1), ("h_last", hl2, hl1)):
        assert torch.isfinite(u).all(), name
        assert_close(to_host(u[:1]) if u.dim() == 4 else to_host(u), to_host(w[:1]) if w.dim() == 4 else to_host(w),
                     "bf16", "fallback " + name)
    del x, b, c, y1, y2


def test_noalloc_in_a_captured_graph(swr):
    # the allocation-free exact forward captured once in a HIP graph (its
    # flags are cleared by a kernel, not a memset) and replayed, with an eager
    # call of another size between replays that leaves other contents in the
    # static array: every replay gives the eager result bit for bit
    prob = W.random_problem(90, 2, 2600, 2, 128, 128, "bf16", "sigmoid", 3.0)
    x, a, b, c = (to_device(getattr(prob, n), "bf16") for n in "xabc")
    other = W.random_problem(91, 1, 5000, 3, 64, 64, "bf16", "sigmoid", 3.0)
    xo, ao, bo, co = (to_device(getattr(other, n), "bf16") for n in "xabc")
    y_e, v_e, hl_e = swr.swr_exact_forward(x, a, b, c, 128, save_carriers=True, want_h_last=True)
    torch.cuda.synchronize()
    y, v, hl = torch.empty_like(y_e), torch.empty_like(v_e), torch.empty_like(hl_e)
    graph = torch.cuda.CUDAGraph()
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        with torch.cuda.graph(graph, stream=stream):
            swr.swr_exact_forward_noalloc(x, a, b, c, 128, y=y, carriers=v, h_last=hl)
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()
    for rep in range(3):
        for t in (y, v, hl):
            t.fill_(7.0)
        swr.swr_exact_forward_noalloc(xo, ao, bo, co, 64)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y_e) and torch.equal(v, v_e) and torch.equal(hl, hl_e), rep
