"""GPU parity of recurrent decoding: swr_step (jagged window, two states),
swr_decode_state (the state after a prompt processed by swr_forward) and
swr_exact_step (exact recurrence), against the oracle on the same seeded,
rounded inputs."""
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


def _dev(prob):
    dt = prob.cfg.dtype
    return [to_device(getattr(prob, n), dt) for n in "xabc"]


CASES = [
    # (B, T, H, D, block, dtype, prompt lengths)
    (2, 200, 3, 64, 64, "f32", (0, 64, 100, 199)),
    (1, 300, 2, 128, 128, "bf16", (128, 131, 257)),
    (2, 90, 2, 16, 16, "bf16", (1, 16, 47)),
    (1, 150, 4, 32, 32, "f32", (96, 149)),
]


@pytest.mark.parametrize("B,T,H,D,block,dtype,prompts", CASES)
@pytest.mark.parametrize("per_channel", [False, True])
def test_prefill_then_decode_matches_full_forward(swr, B, T, H, D, block, dtype, prompts, per_channel):
    prob = W.random_problem(51 + T, B, T, H, D, block, dtype, "sigmoid", 2.0, with_dy=False,
                            per_channel=per_channel)
    x, a, b, c = _dev(prob)
    ref = oracle.forward(prob.x, prob.a, prob.b, prob.c, block)
    for T0 in prompts:
        sl = slice(0, T0)
        y0, v = swr.swr_forward(x[:, sl], a[:, sl], b[:, sl], c[:, sl], block, save_carriers=True)
        st = swr.swr_decode_state(x[:, sl], a[:, sl], v, block)
        outs = [y0]
        for t in range(T0, T):
            s1 = slice(t, t + 1)
            yt, st = swr.swr_step(x[:, s1], a[:, s1], b[:, s1], c[:, s1], block, t, st)
            outs.append(yt)
        torch.cuda.synchronize()
        assert_close(to_host(torch.cat(outs, dim=1)), ref, dtype, f"prompt {T0}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_decode_state_against_oracle(swr, dtype):
    prob = W.random_problem(61, 2, 333, 3, 128, 64, dtype, "sigmoid", 2.0, with_dy=False)
    x, a, b, c = _dev(prob)
    _, v = swr.swr_forward(x, a, b, c, 64, save_carriers=True)
    st = swr.swr_decode_state(x, a, v, 64)
    torch.cuda.synchronize()
    _, ref = oracle.step(prob.x, prob.a, prob.b, prob.c, None, 0, 64)
    assert_close(to_host(st), ref, dtype, "decode state")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("residual", [False, True])
def test_step_chunks_against_oracle(swr, dtype, residual):
    # multi-token calls at arbitrary positions, starting from a nonzero state
    prob = W.random_problem(62, 2, 120, 2, 64, 32, dtype, "sigmoid", 2.0, with_dy=False)
    x, a, b, c = _dev(prob)
    rng = np.random.default_rng(5)
    st0 = rng.standard_normal((2, 2, 2, 64)).astype(np.float32)
    st = torch.from_numpy(st0).cuda()
    ref_state = st0.astype(np.float64)
    for lo, hi in ((0, 5), (5, 32), (32, 33), (33, 100), (100, 120)):
        sl = slice(lo, hi)
        t0 = 1000 + lo        # positions inside a longer sequence (1000 is not a block multiple)
        y, st = swr.swr_step(x[:, sl], a[:, sl], b[:, sl], c[:, sl], 32, t0, st, residual=residual)
        ry, ref_state = oracle.step(prob.x[:, sl], prob.a[:, sl], prob.b[:, sl], prob.c[:, sl], ref_state,
                                    t0, 32, residual)
        torch.cuda.synchronize()
        assert_close(to_host(y), ry, dtype, f"chunk {lo}:{hi} y")
        assert_close(to_host(st), ref_state, dtype, f"chunk {lo}:{hi} state")


def test_step_featurised(swr):
    prob = W.random_problem(63, 1, 80, 2, 32, 16, "bf16", "sigmoid", 3.0, with_dy=False, logits=True)
    x, a, b, c = _dev(prob)
    feat = dict(sigmoid_decay=True, sigmoid_pregate=True)
    y, st = swr.swr_step(x, a, b, c, 16, 0, **feat)
    ry, rst = oracle.step(prob.x, prob.a, prob.b, prob.c, None, 0, 16, **feat)
    torch.cuda.synchronize()
    assert_close(to_host(y), ry, "bf16", "featurised step y")
    assert_close(to_host(st), rst, "bf16", "featurised step state")
    # the decode state of a featurised prompt
    _, v = swr.swr_forward(x, a, b, c, 16, save_carriers=True, **feat)
    st2 = swr.swr_decode_state(x, a, v, 16, sigmoid_decay=True)
    torch.cuda.synchronize()
    assert_close(to_host(st2), rst, "bf16", "featurised decode state")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("per_channel", [False, True])
def test_exact_step_chain(swr, dtype, per_channel):
    # exact prefill (h_last) then token-by-token exact steps = one exact pass
    prob = W.random_problem(64, 2, 260, 2, 64, 64, dtype, "sigmoid", 3.0, with_dy=False,
                            per_channel=per_channel)
    x, a, b, c = _dev(prob)
    rng = np.random.default_rng(6)
    h0 = rng.standard_normal((2, 2, 64)).astype(np.float32)
    ref_y, ref_h = oracle.exact_forward(prob.x, prob.a, prob.b, prob.c, h0)
    T0 = 200
    st = torch.from_numpy(h0).cuda()
    if per_channel:       # the exact forward takes a per-head decay only: prefill by steps
        y0, st = swr.swr_exact_step(x[:, :T0], a[:, :T0], b[:, :T0], c[:, :T0], st)
    else:
        y0, st = swr.swr_exact_forward(x[:, :T0], a[:, :T0], b[:, :T0], c[:, :T0], 64, h0=st,
                                       want_h_last=True)
    outs = [y0]
    for t in range(T0, 260):
        s1 = slice(t, t + 1)
        yt, st = swr.swr_exact_step(x[:, s1], a[:, s1], b[:, s1], c[:, s1], st)
        outs.append(yt)
    torch.cuda.synchronize()
    assert_close(to_host(torch.cat(outs, dim=1)), ref_y, dtype, "exact decode y")
    assert_close(to_host(st), ref_h, dtype, "exact decode state")


def test_step_empty_calls_keep_state(swr):
    x = torch.empty((2, 0, 3, 64), dtype=torch.bfloat16, device="cuda")
    a = torch.empty((2, 0, 3), dtype=torch.bfloat16, device="cuda")
    st = torch.randn(2, 3, 2, 64, device="cuda")
    keep = st.clone()
    swr.swr_step(x, a, x, x, 64, 7, st)
    h = torch.randn(2, 3, 64, device="cuda")
    hk = h.clone()
    swr.swr_exact_step(x, a, x, x, h)
    z = swr.swr_decode_state(x, a, torch.empty((2, 3, 0, 64), device="cuda"), 64)
    torch.cuda.synchronize()
    assert torch.equal(st, keep) and torch.equal(h, hk) and torch.count_nonzero(z) == 0


def test_step_in_a_captured_graph(swr):
    # Decoding steps captured once in a HIP graph and replayed: every replay
    # (from the same starting state) reproduces the eager calls bit for bit.
    prob = W.random_problem(65, 2, 24, 2, 128, 16, "bf16", "sigmoid", 2.0, with_dy=False)
    x, a, b, c = _dev(prob)
    st0 = torch.randn(2, 2, 2, 128, device="cuda")
    st = st0.clone()
    y_eager = torch.empty_like(x)
    for t in range(24):
        s = slice(t, t + 1)
        swr.swr_step(x[:, s], a[:, s], b[:, s], c[:, s], 16, 40 + t, st, y=y_eager[:, s])
    torch.cuda.synchronize()
    st_eager = st.clone()

    st.copy_(st0)
    y = torch.zeros_like(x)
    g = torch.cuda.CUDAGraph()
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        with torch.cuda.graph(g, stream=stream):
            for t in range(24):
                s = slice(t, t + 1)
                swr.swr_step(x[:, s], a[:, s], b[:, s], c[:, s], 16, 40 + t, st, y=y[:, s])
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()
    for rep in range(3):
        st.copy_(st0)
        y.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y_eager), rep
        assert torch.equal(st, st_eager), rep
