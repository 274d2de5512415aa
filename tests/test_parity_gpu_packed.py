"""GPU parity of small heads (d = 16 or 32, the paper's own head size is 16)
with one decay per head: such heads, stored next to each other, run packed
four (d = 16) or two (d = 32) to a 64-channel virtual head on the per-channel
kernels.  Checked against the oracle on every path (jagged window, exact
recurrence, flags), and against the one-head-at-a-time path where packing is
not possible (heads not adjacent, misaligned pointers)."""
import numpy as np
import pytest

import oracle
import workloads as W
from parity import assert_close, check_full, run_gpu, to_device, to_host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def swr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2512_13921_amd as lib
    lib.load()
    return lib


CASES = [
    # (B, T, H, D, block, dtype)
    (2, 300, 4, 16, 16, "bf16"),
    (1, 1000, 8, 16, 16, "f32"),
    (2, 517, 8, 16, 64, "bf16"),
    (1, 700, 4, 32, 32, "bf16"),
    (2, 333, 6, 32, 128, "f32"),
    (1, 64, 128, 16, 16, "bf16"),     # the paper's layer: 128 heads of 16
    (1, 1, 4, 16, 16, "bf16"),
    (1, 17, 2, 32, 16, "f32"),
]


@pytest.mark.parametrize("B,T,H,D,block,dtype", CASES)
@pytest.mark.parametrize("run_len", [0, "min"])
def test_packed_heads_against_oracle(swr, B, T, H, D, block, dtype, run_len):
    rl = max(64, block) if run_len == "min" else 0
    prob = W.random_problem(81 + T + H, B, T, H, D, block, dtype, "sigmoid", 2.0)
    y, grads = run_gpu(swr, prob, run_len=rl)
    check_full(prob, y, grads, what=f"packed {B}x{T}x{H}x{D} l{block} {dtype}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_packed_heads_flags(swr, dtype):
    prob = W.random_problem(82, 2, 400, 8, 16, 16, dtype, "sigmoid", 3.0, logits=True)
    feat = dict(sigmoid_decay=True, sigmoid_pregate=True)
    y, grads = run_gpu(swr, prob, residual=True, **feat)
    check_full(prob, y, grads, residual=True, what="packed residual+sigmoid", **feat)


def test_packed_heads_block_carriers(swr):
    # carriers are per real head, [B, H, blocks, D], whatever the launch plan
    prob = W.random_problem(83, 2, 300, 8, 16, 32, "f32")
    x, a, b, c = (to_device(getattr(prob, n), "f32") for n in "xabc")
    _, v = swr.swr_forward(x, a, b, c, 32, save_carriers=True)
    v2 = swr.swr_carriers(x, a, b, 32)
    torch.cuda.synchronize()
    u = prob.b.astype(np.float64) * prob.x.astype(np.float64)
    av = prob.a.astype(np.float64)
    nb = -(-300 // 32)
    ref = np.zeros((2, 8, nb, 16))
    for t in range(nb):
        s = np.zeros((2, 8, 16))
        for m in range(t * 32, min((t + 1) * 32, 300)):
            s = av[:, m, :, None] * s + u[:, m]
        ref[:, :, t] = s
    assert torch.equal(v, v2)
    assert_close(to_host(v), ref, "f32", "packed carriers")


def test_packed_and_unpacked_plans_agree(swr):
    # the same heads stored [B, H, T, D] (not adjacent: one head at a time) and
    # [B, T, H, D] (adjacent: packed) give the same results
    prob = W.random_problem(84, 1, 500, 8, 16, 16, "f32", "sigmoid", 2.0)
    y1, g1 = run_gpu(swr, prob)
    y2, g2 = run_gpu(swr, prob, layout="bhtd")
    assert_close(to_host(y1), to_host(y2), "f32", "packed vs one head y")
    for name, p_, q_ in zip(("dx", "da", "db", "dc"), g1, g2):
        assert_close(to_host(p_), to_host(q_), "f32", "packed vs one head " + name)


def test_misaligned_small_heads_fall_back(swr):
    # a view starting one element into a buffer: 2-byte aligned only, so the
    # heads run one at a time (and still match the oracle)
    prob = W.random_problem(85, 1, 200, 4, 16, 16, "bf16")
    full = [torch.zeros(1 * 200 * 4 * 16 + 1, dtype=torch.bfloat16, device="cuda") for _ in range(4)]
    ts = []
    for buf, name in zip(full, ("x", "b", "c", "dy")):
        t = buf[1:].view(1, 200, 4, 16)
        t.copy_(to_device(getattr(prob, name), "bf16"))
        ts.append(t)
    x, b, c, dy = ts
    a = to_device(prob.a, "bf16")
    ybuf = torch.zeros(1 * 200 * 4 * 16 + 1, dtype=torch.bfloat16, device="cuda")
    y = ybuf[1:].view(1, 200, 4, 16)
    _, v = swr.swr_forward(x, a, b, c, 16, y=y, save_carriers=True)
    grads = swr.swr_backward(x, a, b, c, dy, v, 16)
    torch.cuda.synchronize()
    check_full(prob, y, grads, what="misaligned small heads")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_packed_heads_exact(swr, dtype):
    prob = W.random_problem(86, 2, 600, 8, 16, 16, dtype, "sigmoid", 3.0)
    x, a, b, c, dy = (to_device(getattr(prob, n), dtype) for n in ("x", "a", "b", "c", "dy"))
    rng = np.random.default_rng(4)
    h0 = rng.standard_normal((2, 8, 16)).astype(np.float32)
    dhl = rng.standard_normal((2, 8, 16)).astype(np.float32)
    h0_t, dhl_t = torch.from_numpy(h0).cuda(), torch.from_numpy(dhl).cuda()
    y, v, hl = swr.swr_exact_forward(x, a, b, c, 16, h0=h0_t, save_carriers=True, want_h_last=True, run_len=64)
    grads = swr.swr_exact_backward(x, a, b, c, dy, v, 16, h0=h0_t, dh_last=dhl_t, want_dh0=True, run_len=64)
    torch.cuda.synchronize()
    ref_y, ref_hl = oracle.exact_forward(prob.x, prob.a, prob.b, prob.c, h0)
    assert_close(to_host(y), ref_y, dtype, "packed exact y")
    assert_close(to_host(hl), ref_hl, dtype, "packed exact h_last")
    ref = oracle.exact_backward(prob.x, prob.a, prob.b, prob.c, prob.dy, h0, dhl)
    for name, g, r in zip(("dx", "da", "db", "dc", "dh0"), grads, ref):
        assert_close(to_host(g), r, dtype, "packed exact " + name)


def test_paper_shape_sampled(swr):
    # the paper's mixer shape (128 heads of 16, block 16) at T = 16K, B = 1;
    # whole sampled heads against the oracle
    prob = W.random_problem(87, 1, 16384, 128, 16, 16, "bf16", "sigmoid", 3.0)
    y, grads = run_gpu(swr, prob)
    picks = [0, 37, 127]
    hi = np.array(picks)
    take = lambda t: np.ascontiguousarray(np.asarray(t)[0][:, hi].transpose(1, 0, *range(2, np.asarray(t).ndim - 1)))
    xs, as_, bs, cs, dys = (take(getattr(prob, n)) for n in ("x", "a", "b", "c", "dy"))
    ref_y = oracle.forward_slices(xs, as_, bs, cs, 16)
    ref = oracle.backward_slices(xs, as_, bs, cs, dys, 16)
    assert_close(np.stack([to_host(y[0, :, h]) for h in picks]), ref_y, "bf16", "paper shape y")
    for name, g, r in zip(("dx", "da", "db", "dc"), grads, ref):
        got = np.stack([to_host(g[0, :, h]) for h in picks])
        assert_close(got, r, "bf16", "paper shape " + name)
