"""GPU parity: the HIP library (called through its C ABI binding) against the
double-precision oracle on the same seeded, rounded inputs."""
import sys

import numpy as np
import pytest

import oracle
import workloads as W
from parity import assert_close, check_full, compare_whole, run_gpu, to_device, to_host, workload

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def swr():
    _need_gpu()
    import paper_2512_13921_amd as lib
    lib.load()
    return lib


# ----------------------------------------------------------------------------- small shapes

SMALL = [
    # (B, T, H, D, block, dtype)
    (1, 64, 1, 16, 16, "f32"),
    (2, 1000, 3, 64, 64, "f32"),
    (1, 333, 2, 128, 128, "f32"),
    (2, 517, 2, 32, 32, "f32"),
    (2, 1000, 3, 64, 64, "bf16"),
    (1, 777, 2, 128, 128, "bf16"),
    (2, 300, 2, 16, 16, "bf16"),
    (1, 513, 3, 32, 32, "bf16"),
    (1, 1024, 2, 128, 64, "bf16"),
    (1, 640, 2, 64, 128, "bf16"),
    (1, 1, 1, 64, 64, "bf16"),      # a single token
    (1, 17, 1, 128, 128, "bf16"),   # shorter than one sub-block ... one block
    (1, 130, 1, 16, 128, "f32"),
    (2, 700, 4, 64, 64, "bf16"),    # several head pairs per batch entry
    (3, 300, 6, 128, 32, "f32"),
]


@pytest.mark.parametrize("B,T,H,D,block,dtype", SMALL)
@pytest.mark.parametrize("run_len", [0, "min"])
def test_small_against_oracle(swr, B, T, H, D, block, dtype, run_len):
    step = max(64, block)
    rl = step if run_len == "min" else 0     # "min": every step is its own run (many halos)
    prob = W.random_problem(7 + T + D, B, T, H, D, block, dtype, "sigmoid", 1.5)
    _say(f"[small] B={B} T={T} H={H} D={D} l={block} {dtype} run_len={rl}")
    y, grads = run_gpu(swr, prob, run_len=rl)
    check_full(prob, y, grads, what=f"{B}x{T}x{H}x{D} l{block} {dtype}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_residual_flag(swr, dtype):
    prob = W.random_problem(3, 2, 400, 2, 64, 64, dtype)
    y, grads = run_gpu(swr, prob, residual=True)
    check_full(prob, y, grads, residual=True, what="residual")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_strided_bhtd_layout(swr, dtype):
    prob = W.random_problem(5, 2, 384, 3, 64, 64, dtype)
    y, grads = run_gpu(swr, prob, layout="bhtd")
    assert y.stride() != y.contiguous().stride()
    check_full(prob, y, grads, what="bhtd")


@pytest.mark.parametrize("value", [0.0, 1.0])
@pytest.mark.parametrize("block", [16, 128])
def test_decay_closed_forms(swr, value, block):
    # a == 0: y = c*b*x; a == 1: a jagged box filter.  Both exact special cases.
    prob = W.random_problem(11, 1, 500, 2, 64, block, "f32")
    prob.a[...] = value
    y, grads = run_gpu(swr, prob)
    check_full(prob, y, grads, what=f"a={value}")
    if value == 0.0:
        np.testing.assert_allclose(to_host(y), (prob.c * prob.b * prob.x).astype(np.float64),
                                   rtol=1e-6, atol=1e-6)


def test_zero_decays_mixed(swr):
    prob = W.random_problem(12, 2, 700, 2, 128, 128, "bf16")
    rng = np.random.default_rng(0)
    mask = rng.random(prob.a.shape)
    prob.a[mask < 0.05] = 0.0
    prob.a[mask > 0.95] = 1.0
    y, grads = run_gpu(swr, prob)
    check_full(prob, y, grads, what="mixed zeros/ones")


def test_deterministic(swr):
    prob = W.random_problem(13, 2, 2048, 4, 128, 128, "bf16")
    y1, g1 = run_gpu(swr, prob)
    y2, g2 = run_gpu(swr, prob)
    assert torch.equal(y1, y2)
    for a, b in zip(g1, g2):
        assert torch.equal(a, b)


def test_inputs_may_alias(swr):
    # b and c may be the same tensor as x (only outputs must not overlap anything)
    prob = W.random_problem(14, 1, 256, 2, 64, 64, "bf16")
    x = to_device(prob.x, "bf16")
    a = to_device(prob.a, "bf16")
    y, v = swr.swr_forward(x, a, x, x, 64, save_carriers=True)
    dx, da, db, dc = swr.swr_backward(x, a, x, x, x, v, 64)
    torch.cuda.synchronize()
    ref = oracle.forward(prob.x, prob.a, prob.x, prob.x, 64)
    assert_close(to_host(y), ref, "bf16", "aliased inputs")
    rdx, rda, rdb, rdc = oracle.backward(prob.x, prob.a, prob.x, prob.x, prob.x, 64)
    assert_close(to_host(dx), rdx, "bf16", "aliased dx")
    assert_close(to_host(da), rda, "bf16", "aliased da")


def test_empty_inputs(swr):
    x = torch.empty((2, 0, 3, 64), dtype=torch.bfloat16, device="cuda")
    a = torch.empty((2, 0, 3), dtype=torch.bfloat16, device="cuda")
    y, v = swr.swr_forward(x, a, x, x, 64, save_carriers=True)
    dx, da, db, dc = swr.swr_backward(x, a, x, x, x, v, 64)
    assert y.shape == x.shape and da.shape == a.shape and v.shape == (2, 3, 0, 64)


def _carriers_by_definition(prob):
    """v_t: state at the end of block t of the recurrence restarted at the block's
    start (float64 loop, the carrier definition of Alg. "Block Two-Pass")."""
    cfg = prob.cfg
    l, T = cfg.block, cfg.T
    nb = -(-T // l)
    u = prob.b.astype(np.float64) * prob.x.astype(np.float64)     # [B, T, H, D]
    a = prob.a.astype(np.float64)
    v = np.zeros((cfg.B, cfg.H, nb, cfg.D))
    for t in range(nb):
        s = np.zeros((cfg.B, cfg.H, cfg.D))
        for m in range(t * l, min((t + 1) * l, T)):
            s = a[:, m, :, None] * s + u[:, m]
        v[:, :, t] = s
    return v


@pytest.mark.parametrize("dtype,D,block", [("bf16", 128, 128), ("f32", 64, 32), ("bf16", 16, 16)])
def test_block_carriers(swr, dtype, D, block):
    prob = W.random_problem(21, 2, 517, 3, D, block, dtype)
    x, a, b, c = (to_device(getattr(prob, n), dtype) for n in "xabc")
    _, v1 = swr.swr_forward(x, a, b, c, block, save_carriers=True, run_len=max(64, block))
    v2 = swr.swr_carriers(x, a, b, block)
    torch.cuda.synchronize()
    assert torch.equal(v1, v2)          # the same kernel path, bit for bit
    ref = _carriers_by_definition(prob)
    scale = np.sqrt(np.mean(ref * ref))
    err = np.abs(to_host(v1) - ref) / np.maximum(np.abs(ref), scale)
    assert err.max() < 1e-4, err.max()




def test_autograd_function(swr):
    prob = W.random_problem(15, 1, 256, 2, 64, 64, "f32")
    x, a, b, c = (to_device(getattr(prob, n), "f32").requires_grad_() for n in "xabc")
    y = swr.SWRFunction.apply(x, a, b, c, 64)
    dy = to_device(prob.dy, "f32")
    (y * dy).sum().backward()
    ref = oracle.backward(prob.x, prob.a, prob.b, prob.c, prob.dy, 64)
    for t, r, n in zip((x, a, b, c), (ref[0], ref[1], ref[2], ref[3]), "xabc"):
        assert_close(to_host(t.grad), r, "f32", "autograd d" + n)


# ----------------------------------------------------------------------------- the five workloads


def test_config1_full(swr):
    cfg = W.CONFIGS[1]
    prob = W.generate(cfg, with_dy=True)      # forward workload; the backward is checked too
    _say(f"[config 1] {cfg.name}")
    y, grads = run_gpu(swr, prob)
    check_full(prob, y, grads, what="config 1")


def _heads(t, b, h0, h1):
    """tensor[b:b+1, :, h0:h1] of a host array in [B, T, H, ...] layout."""
    return np.asarray(t)[b:b + 1, :, h0:h1]


@pytest.mark.parametrize("cid", [2, 3, 4, 5])
def test_full_size_whole_tensors(swr, cid):
    """Full-size run in the default launch configuration; every element of y,
    dx, da, db and dc is compared with the oracle (streamed over chunks of
    heads), and the whole-tensor error figures are reported."""
    cfg = W.CONFIGS[cid]
    _say(f"[config {cid}] {cfg.name}: generating inputs")
    prob = workload(cfg)
    _say(f"[config {cid}] running on the GPU")
    y, grads = run_gpu(swr, prob)

    def ref_chunk(b, h0, h1):
        args = [_heads(getattr(prob, n), b, h0, h1) for n in ("x", "a", "b", "c")]
        ref = dict(y=oracle.forward(*args, cfg.block))
        ref.update(zip(("dx", "da", "db", "dc"),
                       oracle.backward(*args, _heads(prob.dy, b, h0, h1), cfg.block)))
        return ref

    outs = [("y", y, 2, 1)] + [(n, g, 2, 1) for n, g in zip(("dx", "da", "db", "dc"), grads)]
    _say(f"[config {cid}] comparing whole tensors with the oracle")
    compare_whole(f"config {cid} {cfg.name}", cfg.dtype, cfg.B, cfg.H, outs, ref_chunk)
