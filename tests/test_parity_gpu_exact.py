"""GPU parity of the exact (untruncated) recurrence -- the three-stage
hierarchical algorithm (Alg. "Hierarchical Block Parallel Inference") behind
swr_exact_forward / swr_exact_backward -- against the oracle's exact loop on
the same seeded, rounded inputs, with initial states and final-state
gradients."""
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


def _state(rng, cfg, scale=1.0):
    return (scale * rng.standard_normal((cfg.B, cfg.H, cfg.D))).astype(np.float32)


def _exact_states(prob, h0, **feat):
    """h at every token (float64 oracle run with c = 1), [B, T, H, D]."""
    ones = np.ones_like(prob.c, dtype=np.float64)
    h, _ = oracle.exact_forward(prob.x, prob.a, prob.b, ones, h0, **feat)
    return h


def _block_end_states(prob, h):
    cfg = prob.cfg
    nb = -(-cfg.T // cfg.block)
    ends = [min((t + 1) * cfg.block, cfg.T) - 1 for t in range(nb)]
    return np.transpose(h[:, ends], (0, 2, 1, 3))          # [B, H, nb, D]


def run_exact(swr, prob, h0, dh_last, residual=False, run_len=0, backward=True, **feat):
    cfg = prob.cfg
    dt = cfg.dtype
    x, a, b, c = (to_device(getattr(prob, n), dt) for n in "xabc")
    h0_t = None if h0 is None else torch.from_numpy(h0).cuda()
    dhl_t = None if dh_last is None else torch.from_numpy(dh_last).cuda()
    y, v, hl = swr.swr_exact_forward(x, a, b, c, cfg.block, h0=h0_t, residual=residual, save_carriers=True,
                                     want_h_last=True, run_len=run_len, **feat)
    grads = None
    if backward:
        dy = to_device(prob.dy, dt)
        grads = swr.swr_exact_backward(x, a, b, c, dy, v, cfg.block, h0=h0_t, dh_last=dhl_t,
                                       residual=residual, want_dh0=True, run_len=run_len, **feat)
    torch.cuda.synchronize()
    return y, v, hl, grads


def check_exact(prob, h0, dh_last, y, v, hl, grads, residual=False, what="", **feat):
    cfg = prob.cfg
    ref_y, ref_hl = oracle.exact_forward(prob.x, prob.a, prob.b, prob.c, h0, residual, **feat)
    assert_close(to_host(y), ref_y, cfg.dtype, what + " y")
    # The final state and the block carriers are float32 on every path.
    assert_close(to_host(hl), ref_hl, "bf16" if cfg.dtype == "bf16" else "f32", what + " h_last")
    ref_v = _block_end_states(prob, _exact_states(prob, h0, **feat))
    assert_close(to_host(v), ref_v, cfg.dtype, what + " carriers")
    if grads is not None:
        ref = oracle.exact_backward(prob.x, prob.a, prob.b, prob.c, prob.dy, h0, dh_last, residual, **feat)
        for name, g, r in zip(("dx", "da", "db", "dc", "dh0"), grads, ref):
            assert_close(to_host(g), r, cfg.dtype, f"{what} {name}")


SMALL = [
    # (B, T, H, D, block, dtype)
    (1, 64, 1, 16, 16, "f32"),
    (2, 1000, 3, 64, 64, "f32"),
    (1, 333, 2, 128, 128, "f32"),
    (2, 517, 2, 32, 32, "f32"),
    (2, 1000, 3, 64, 64, "bf16"),
    (1, 777, 2, 128, 128, "bf16"),
    (2, 300, 2, 16, 16, "bf16"),
    (1, 1, 1, 64, 64, "bf16"),      # a single token: the recurrent decoding step
    (1, 17, 1, 128, 128, "bf16"),
    (2, 700, 4, 64, 64, "bf16"),
    (1, 700, 2, 64, 128, "bf16"),   # 8-wave groups of 64 channels (inputs fetched a step ahead)
    (3, 300, 6, 128, 32, "f32"),
]


@pytest.mark.parametrize("B,T,H,D,block,dtype", SMALL)
@pytest.mark.parametrize("run_len", [0, "min"])
def test_exact_small_against_oracle(swr, B, T, H, D, block, dtype, run_len):
    rl = max(64, block) if run_len == "min" else 0    # "min": many runs, a long carrier chain
    prob = W.random_problem(31 + T + D, B, T, H, D, block, dtype, "sigmoid", 2.0)
    rng = np.random.default_rng(T)
    h0, dhl = _state(rng, prob.cfg), _state(rng, prob.cfg)
    _say(f"[exact] B={B} T={T} H={H} D={D} l={block} {dtype} run_len={rl}")
    y, v, hl, grads = run_exact(swr, prob, h0, dhl, run_len=rl)
    check_exact(prob, h0, dhl, y, v, hl, grads, what=f"exact {B}x{T}x{H}x{D} l{block} {dtype}")


PC = [
    # (B, T, H, D, block, dtype): per-channel decay; D = 128 runs as two 64-channel halves
    (1, 64, 1, 16, 16, "f32"),
    (2, 1000, 3, 64, 64, "f32"),
    (1, 777, 2, 128, 128, "bf16"),
    (2, 300, 2, 32, 32, "bf16"),
    (1, 1, 1, 64, 64, "bf16"),
]


@pytest.mark.parametrize("B,T,H,D,block,dtype", PC)
@pytest.mark.parametrize("run_len", [0, "min"])
def test_exact_per_channel_against_oracle(swr, B, T, H, D, block, dtype, run_len):
    rl = max(64, block) if run_len == "min" else 0
    prob = W.random_problem(71 + T + D, B, T, H, D, block, dtype, "sigmoid", 2.0, per_channel=True)
    rng = np.random.default_rng(T + 1)
    h0, dhl = _state(rng, prob.cfg), _state(rng, prob.cfg)
    y, v, hl, grads = run_exact(swr, prob, h0, dhl, run_len=rl)
    check_exact(prob, h0, dhl, y, v, hl, grads, what=f"exact pc {B}x{T}x{H}x{D} l{block} {dtype}")


def test_exact_per_channel_featurised_residual(swr):
    prob = W.random_problem(72, 2, 300, 2, 128, 64, "bf16", "sigmoid", 3.0, per_channel=True, logits=True)
    rng = np.random.default_rng(9)
    h0, dhl = _state(rng, prob.cfg), _state(rng, prob.cfg)
    feat = dict(sigmoid_decay=True, sigmoid_pregate=True)
    y, v, hl, grads = run_exact(swr, prob, h0, dhl, residual=True, run_len=128, **feat)
    check_exact(prob, h0, dhl, y, v, hl, grads, residual=True, what="pc residual+sigmoid", **feat)


def test_exact_per_channel_constant_equals_shared(swr):
    # a decay constant across channels: the per-channel path gives the shared
    # path's outputs, and its da summed over channels is the shared da.
    prob = W.random_problem(73, 1, 500, 2, 64, 64, "f32", "sigmoid", 2.0)
    x, a, b, c, dy = (to_device(getattr(prob, n), "f32") for n in ("x", "a", "b", "c", "dy"))
    apc = a[..., None].expand(-1, -1, -1, 64).contiguous()
    y1, v1 = swr.swr_exact_forward(x, a, b, c, 64, save_carriers=True)
    y2, v2 = swr.swr_exact_forward(x, apc, b, c, 64, save_carriers=True)
    g1 = swr.swr_exact_backward(x, a, b, c, dy, v1, 64)
    g2 = swr.swr_exact_backward(x, apc, b, c, dy, v2, 64)
    torch.cuda.synchronize()
    assert_close(to_host(y2), to_host(y1), "f32", "pc vs shared y")
    for name, u, w in zip(("dx", "db", "dc"), (g2[0], g2[2], g2[3]), (g1[0], g1[2], g1[3])):
        assert_close(to_host(u), to_host(w), "f32", "pc vs shared " + name)
    assert_close(to_host(g2[1]).sum(-1), to_host(g1[1]), "f32", "pc vs shared da")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_exact_without_states(swr, dtype):
    prob = W.random_problem(41, 2, 640, 2, 64, 64, dtype, "sigmoid", 3.0)
    y, v, hl, grads = run_exact(swr, prob, None, None, run_len=64)
    check_exact(prob, None, None, y, v, hl, grads, what="no h0")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_exact_residual_and_featurisation(swr, dtype):
    prob = W.random_problem(42, 2, 400, 2, 128, 64, dtype, "sigmoid", 3.0, logits=True)
    rng = np.random.default_rng(1)
    h0, dhl = _state(rng, prob.cfg), _state(rng, prob.cfg)
    feat = dict(sigmoid_decay=True, sigmoid_pregate=True)
    y, v, hl, grads = run_exact(swr, prob, h0, dhl, residual=True, run_len=64, **feat)
    check_exact(prob, h0, dhl, y, v, hl, grads, residual=True, what="residual+sigmoid", **feat)


@pytest.mark.parametrize("value", [0.0, 1.0])
@pytest.mark.parametrize("T", [300, 5000])
def test_exact_decay_closed_forms(swr, value, T):
    # a == 0: y = c*b*x (h0 forgotten at once); a == 1: a running sum from h0
    # (T = 5000: 40 chunks, so the one-pass forward chains through boundaries)
    prob = W.random_problem(43, 1, T, 2, 64, 64, "f32")
    prob.a[...] = value
    rng = np.random.default_rng(2)
    h0, dhl = _state(rng, prob.cfg), _state(rng, prob.cfg)
    y, v, hl, grads = run_exact(swr, prob, h0, dhl, run_len=64)
    check_exact(prob, h0, dhl, y, v, hl, grads, what=f"a={value}")


def test_exact_equals_jagged_window_on_two_blocks(swr):
    # T <= 2l: the window truncation drops nothing, so both paths agree.
    prob = W.random_problem(44, 2, 256, 2, 128, 128, "f32")
    x, a, b, c, dy = (to_device(getattr(prob, n), "f32") for n in ("x", "a", "b", "c", "dy"))
    y_ex, v_ex = swr.swr_exact_forward(x, a, b, c, 128, save_carriers=True)
    y_sw, v_sw = swr.swr_forward(x, a, b, c, 128, save_carriers=True)
    g_ex = swr.swr_exact_backward(x, a, b, c, dy, v_ex, 128)
    g_sw = swr.swr_backward(x, a, b, c, dy, v_sw, 128)
    torch.cuda.synchronize()
    assert_close(to_host(y_ex), to_host(y_sw).astype(np.float64), "f32", "exact vs window y")
    for name, ge, gs in zip(("dx", "da", "db", "dc"), g_ex, g_sw):
        assert_close(to_host(ge), to_host(gs), "f32", "exact vs window " + name)


def test_exact_chunked_equals_one_pass(swr):
    # Processing the sequence in pieces, passing h_last on as h0, is the same
    # computation as one pass (recurrent prefill / decoding).
    prob = W.random_problem(45, 2, 1000, 2, 64, 64, "f32", "sigmoid", 3.0)
    x, a, b, c = (to_device(getattr(prob, n), "f32") for n in "xabc")
    y_full = swr.swr_exact_forward(x, a, b, c, 64)
    h = None
    parts = []
    for lo, hi in ((0, 333), (333, 334), (334, 640), (640, 1000)):
        sl = slice(lo, hi)
        yp, h = swr.swr_exact_forward(x[:, sl], a[:, sl], b[:, sl], c[:, sl], 64, h0=h, want_h_last=True)
        parts.append(yp)
    torch.cuda.synchronize()
    assert_close(to_host(torch.cat(parts, dim=1)), to_host(y_full), "f32", "chunked")


def test_exact_empty_sequence_passes_states(swr):
    x = torch.empty((2, 0, 3, 64), dtype=torch.bfloat16, device="cuda")
    a = torch.empty((2, 0, 3), dtype=torch.bfloat16, device="cuda")
    h0 = torch.randn(2, 3, 64, device="cuda")
    dhl = torch.randn(2, 3, 64, device="cuda")
    y, v, hl = swr.swr_exact_forward(x, a, x, x, 64, h0=h0, save_carriers=True, want_h_last=True)
    *_, dh0 = swr.swr_exact_backward(x, a, x, x, x, v, 64, h0=h0, dh_last=dhl, want_dh0=True)
    torch.cuda.synchronize()
    assert torch.equal(hl, h0) and torch.equal(dh0, dhl)
    _, hz = swr.swr_exact_forward(x, a, x, x, 64, want_h_last=True)
    torch.cuda.synchronize()
    assert torch.count_nonzero(hz) == 0


def test_exact_deterministic(swr):
    prob = W.random_problem(46, 2, 2048, 4, 128, 128, "bf16")
    rng = np.random.default_rng(3)
    h0, dhl = _state(rng, prob.cfg), _state(rng, prob.cfg)
    r1 = run_exact(swr, prob, h0, dhl)
    r2 = run_exact(swr, prob, h0, dhl)
    for t1, t2 in zip(r1[:3] + tuple(r1[3]), r2[:3] + tuple(r2[3])):
        assert torch.equal(t1, t2)


@pytest.mark.parametrize("cid", [3, 4, 5])
def test_exact_full_size_whole_tensors(swr, cid):
    """Full-size exact forward and backward in the default launch
    configuration, with an initial state and a final-state gradient; every
    element of y, h_last, dx, da, db, dc and dh0 is compared with the oracle."""
    cfg = W.CONFIGS[cid]
    _say(f"[exact config {cid}] {cfg.name}: generating inputs")
    prob = workload(cfg)
    rng = np.random.default_rng(cid)
    h0, dhl = _state(rng, cfg), _state(rng, cfg)
    _say(f"[exact config {cid}] running on the GPU")
    y, v, hl, grads = run_exact(swr, prob, h0, dhl)

    def ref_chunk(b, h0_, h1_):
        args = [np.asarray(getattr(prob, n))[b:b + 1, :, h0_:h1_] for n in ("x", "a", "b", "c")]
        st0, dst = h0[b:b + 1, h0_:h1_], dhl[b:b + 1, h0_:h1_]
        ref = dict(zip(("y", "h_last"), oracle.exact_forward(*args, st0)))
        ref.update(zip(("dx", "da", "db", "dc", "dh0"),
                       oracle.exact_backward(*args, prob.dy[b:b + 1, :, h0_:h1_], st0, dst)))
        states, _ = oracle.exact_forward(args[0], args[1], args[2], np.ones_like(args[3]), st0)
        nb = -(-cfg.T // cfg.block)
        ends = [min((t + 1) * cfg.block, cfg.T) - 1 for t in range(nb)]
        ref["carriers"] = np.transpose(states[:, ends], (0, 2, 1, 3))     # [1, heads, nb, D]
        return ref

    outs = [("y", y, 2, 1), ("h_last", hl, 1, 1)]
    outs += [(n, g, 2, 1) for n, g in zip(("dx", "da", "db", "dc"), grads[:4])]
    outs += [("dh0", grads[4], 1, 1), ("carriers", v, 1, 1)]
    _say(f"[exact config {cid}] comparing whole tensors with the oracle")
    compare_whole(f"exact config {cid} {cfg.name}", cfg.dtype, cfg.B, cfg.H, outs, ref_chunk)

CHAINED = [
    # (B, T, H, D, block, dtype): sequences of more than 16 chunks of 128 tokens,
    # so that the one-pass forward's boundary chunks (every 16th; every 8th for
    # bf16 heads of 64 on sequences of fewer than 256 chunks) publish inclusive
    # states that the chunks after them start from
    (1, 5000, 2, 128, 128, "f32"),   # ragged tail; float32 heads of 128 as two halves of 64
    (2, 4500, 3, 64, 64, "bf16"),
    (1, 4096, 1, 128, 128, "bf16"),  # the last chunk is a boundary chunk
    (1, 3072, 2, 64, 64, "bf16"),    # the same with boundaries every 8th chunk
    (1, 2049, 2, 32, 32, "bf16"),    # the last chunk starts right after the first boundary
    (1, 1025, 2, 64, 128, "bf16"),   # the same with boundaries every 8th chunk
    (1, 6000, 1, 16, 16, "f32"),
]


@pytest.mark.parametrize("B,T,H,D,block,dtype", CHAINED)
def test_exact_forward_across_boundary_chunks(swr, B, T, H, D, block, dtype):
    prob = W.random_problem(91 + T + D, B, T, H, D, block, dtype, "sigmoid", 3.0)
    rng = np.random.default_rng(T + 7)
    h0 = _state(rng, prob.cfg)
    _say(f"[exact chained] B={B} T={T} H={H} D={D} l={block} {dtype}")
    y, v, hl, _ = run_exact(swr, prob, h0, None, backward=False)
    check_exact(prob, h0, None, y, v, hl, None, what=f"chained {B}x{T}x{H}x{D} l{block} {dtype}")


@pytest.mark.parametrize("B,T,H,D,block,dtype", [(1, 65536, 2, 64, 128, "bf16"), (1, 20000, 2, 128, 128, "f32"),
                                                 (2, 16384, 2, 128, 64, "bf16")])
def test_exact_forward_is_deterministic(swr, B, T, H, D, block, dtype):
    # the chunks compose their predecessors in a fixed pattern, whatever order
    # the workgroups reach them in: repeated calls agree bit for bit
    prob = W.random_problem(95, B, T, H, D, block, dtype, "sigmoid", 4.0)
    x, a, b, c = (to_device(getattr(prob, n), dtype) for n in "xabc")
    h0 = torch.from_numpy(_state(np.random.default_rng(5), prob.cfg)).cuda()
    _say(f"[exact determinism] B={B} T={T} H={H} D={D} l={block} {dtype}")
    first = swr.swr_exact_forward(x, a, b, c, block, h0=h0, save_carriers=True, want_h_last=True)
    for _ in range(3):
        again = swr.swr_exact_forward(x, a, b, c, block, h0=h0, save_carriers=True, want_h_last=True)
        torch.cuda.synchronize()
        for name, u, w in zip(("y", "carriers", "h_last"), again, first):
            assert torch.equal(u, w), name
    ref_y, ref_hl = oracle.exact_forward(prob.x, prob.a, prob.b, prob.c, to_host(h0))
    assert_close(to_host(first[2]), ref_hl, "bf16" if dtype == "bf16" else "f32", "determinism h_last")


def _bhtd(t):
    # stored as [B, H, T, ...], handed over as a strided [B, T, H, ...] view
    if t.dim() == 4:
        return t.permute(0, 2, 1, 3).contiguous().permute(0, 2, 1, 3)
    return t.permute(0, 2, 1).contiguous().permute(0, 2, 1)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_exact_forward_chained_strided_featurised_residual(swr, dtype):
    # more than 16 chunks of 128 tokens, a [B, H, T, d] layout, the fused
    # sigmoids and the residual, on the one-pass forward
    prob = W.random_problem(97, 2, 2500, 3, 128, 64, dtype, "sigmoid", 3.0, logits=True)
    feat = dict(sigmoid_decay=True, sigmoid_pregate=True)
    x, a, b, c = (_bhtd(to_device(getattr(prob, n), dtype)) for n in "xabc")
    assert x.stride() != x.contiguous().stride()
    h0 = _state(np.random.default_rng(11), prob.cfg)
    _say(f"[exact chained strided] 2x2500x3x128 l64 {dtype}")
    y, v, hl = swr.swr_exact_forward(x, a, b, c, 64, h0=torch.from_numpy(h0).cuda(), residual=True,
                                     save_carriers=True, want_h_last=True, **feat)
    torch.cuda.synchronize()
    check_exact(prob, h0, None, y, v, hl, None, residual=True, what=f"chained strided {dtype}", **feat)


def test_exact_forward_chained_optional_outputs(swr):
    # y alone, then y with h_last alone: the same y bits as with every output
    prob = W.random_problem(98, 1, 3000, 2, 64, 128, "bf16", "sigmoid", 3.0)
    x, a, b, c = (to_device(getattr(prob, n), "bf16") for n in "xabc")
    y_all, v, hl = swr.swr_exact_forward(x, a, b, c, 128, save_carriers=True, want_h_last=True)
    y_only = swr.swr_exact_forward(x, a, b, c, 128)
    y_hl, hl2 = swr.swr_exact_forward(x, a, b, c, 128, want_h_last=True)
    torch.cuda.synchronize()
    assert torch.equal(y_only, y_all) and torch.equal(y_hl, y_all) and torch.equal(hl2, hl)
    check_exact(prob, None, None, y_all, v, hl, None, what="chained all outputs")


def test_exact_in_a_captured_graph(swr):
    # forward (one pass) and backward captured once in a HIP graph, replayed
    # with eager work between replays: every replay gives the eager results
    prob = W.random_problem(99, 2, 2300, 2, 64, 64, "bf16", "sigmoid", 3.0)
    x, a, b, c, dy = (to_device(getattr(prob, n), "bf16") for n in ("x", "a", "b", "c", "dy"))
    h0 = torch.from_numpy(_state(np.random.default_rng(3), prob.cfg)).cuda()
    y_e, v_e, hl_e = swr.swr_exact_forward(x, a, b, c, 64, h0=h0, save_carriers=True, want_h_last=True)
    g_e = swr.swr_exact_backward(x, a, b, c, dy, v_e, 64, h0=h0, dh_last=hl_e, want_dh0=True)
    torch.cuda.synchronize()
    y, v, hl = torch.empty_like(y_e), torch.empty_like(v_e), torch.empty_like(hl_e)
    outs = tuple(torch.empty_like(t) for t in g_e[:4])
    graph = torch.cuda.CUDAGraph()
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        with torch.cuda.graph(graph, stream=stream):
            swr.swr_exact_forward(x, a, b, c, 64, h0=h0, y=y, carriers=v, h_last=hl)
            swr.swr_exact_backward(x, a, b, c, dy, v, 64, h0=h0, dh_last=hl, outputs=outs)
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()
    for rep in range(3):
        for t in (y, v, hl) + outs:
            t.fill_(7.0)
        swr.swr_exact_forward(c, a, b, x, 64)   # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y_e) and torch.equal(v, v_e) and torch.equal(hl, hl_e), rep
        for p_, q_ in zip(outs, g_e[:4]):
            assert torch.equal(p_, q_), rep


@pytest.mark.parametrize("B,T,H,D,block,dtype", [(1, 40000, 2, 64, 128, "bf16"), (1, 33000, 1, 32, 32, "f32"),
                                                 (1, 32768, 1, 16, 16, "bf16")])
def test_exact_backward_one_pass_long_sequences(swr, B, T, H, D, block, dtype):
    # long sequences (256 chunks and more) through the one-pass backward
    # (chunks taken from the end, chained by the look-back): against the
    # oracle, and repeated calls agree bit for bit
    prob = W.random_problem(101 + D, B, T, H, D, block, dtype, "sigmoid", 4.0)
    rng = np.random.default_rng(D)
    h0, dhl = _state(rng, prob.cfg), _state(rng, prob.cfg)
    _say(f"[exact one-pass backward] B={B} T={T} H={H} D={D} l={block} {dtype}")
    y, v, hl, grads = run_exact(swr, prob, h0, dhl)
    check_exact(prob, h0, dhl, y, v, hl, grads, what=f"one-pass bwd {B}x{T}x{H}x{D} {dtype}")
    x, a, b, c, dy = (to_device(getattr(prob, n), dtype) for n in ("x", "a", "b", "c", "dy"))
    h0_t, dhl_t = torch.from_numpy(h0).cuda(), torch.from_numpy(dhl).cuda()
    again = swr.swr_exact_backward(x, a, b, c, dy, v, block, h0=h0_t, dh_last=dhl_t, want_dh0=True)
    torch.cuda.synchronize()
    for name, u, w in zip(("dx", "da", "db", "dc", "dh0"), again, grads):
        assert torch.equal(u, w), name


CHAINED_PC = [
    # (B, T, H, D, block, dtype, per-channel decay): the one-pass forward with a
    # decay product per channel (a decay per channel) on sequences of more than
    # 16 chunks; small heads stored next to each other (packed four or two to a
    # 64-channel group) run the three stages, checked the same way
    (1, 3000, 2, 128, 128, "bf16", True),   # heads of 128 as two halves of 64
    (1, 2500, 3, 64, 64, "f32", True),
    (2, 2049, 2, 32, 32, "bf16", True),
    (1, 2300, 1, 16, 16, "f32", True),
    (1, 3000, 4, 16, 16, "bf16", False),     # packed four to a group
    (2, 2600, 2, 32, 32, "f32", False),      # packed two to a group
    (1, 33000, 1, 64, 64, "bf16", True),     # 258 chunks: boundaries every 16
]


@pytest.mark.parametrize("B,T,H,D,block,dtype,pc", CHAINED_PC)
def test_exact_forward_chained_per_channel_products(swr, B, T, H, D, block, dtype, pc):
    prob = W.random_problem(111 + T + D, B, T, H, D, block, dtype, "sigmoid", 3.0, per_channel=pc)
    rng = np.random.default_rng(T + 9)
    h0 = _state(rng, prob.cfg)
    _say(f"[exact chained pc] B={B} T={T} H={H} D={D} l={block} {dtype} per_channel={pc}")
    y, v, hl, _ = run_exact(swr, prob, h0, None, backward=False)
    check_exact(prob, h0, None, y, v, hl, None, what=f"chained pc {B}x{T}x{H}x{D} {dtype} pc={pc}")
    x, a, b, c = (to_device(getattr(prob, n), dtype) for n in "xabc")
    again = swr.swr_exact_forward(x, a, b, c, block, h0=torch.from_numpy(h0).cuda(), save_carriers=True,
                                  want_h_last=True)
    torch.cuda.synchronize()
    for name, u, w in zip(("y", "carriers", "h_last"), again, (y, v, hl)):
        assert torch.equal(u, w), name


def test_exact_forward_chained_per_channel_featurised_residual(swr):
    prob = W.random_problem(113, 2, 2200, 2, 128, 64, "bf16", "sigmoid", 3.0, per_channel=True, logits=True)
    rng = np.random.default_rng(13)
    h0 = _state(rng, prob.cfg)
    feat = dict(sigmoid_decay=True, sigmoid_pregate=True)
    y, v, hl, _ = run_exact(swr, prob, h0, None, residual=True, backward=False, **feat)
    check_exact(prob, h0, None, y, v, hl, None, residual=True, what="chained pc residual+sigmoid", **feat)


def test_exact_forward_many_chained_sequences(swr):
    # 512 sequences of 18 chunks (9216 chunks, several per workgroup): repeated
    # calls agree bit for bit, and sampled sequences match the oracle
    prob = W.random_problem(121, 16, 2200, 32, 64, 64, "bf16", "sigmoid", 3.0, with_dy=False)
    x, a, b, c = (to_device(getattr(prob, n), "bf16") for n in "xabc")
    h0 = _state(np.random.default_rng(17), prob.cfg)
    h0_t = torch.from_numpy(h0).cuda()
    first = swr.swr_exact_forward(x, a, b, c, 64, h0=h0_t, save_carriers=True, want_h_last=True)
    for _ in range(2):
        again = swr.swr_exact_forward(x, a, b, c, 64, h0=h0_t, save_carriers=True, want_h_last=True)
        torch.cuda.synchronize()
        for name, u, w in zip(("y", "carriers", "h_last"), again, first):
            assert torch.equal(u, w), name
    y = to_host(first[0])
    hl = to_host(first[2])
    for bi, hi in ((0, 0), (15, 31), (7, 13), (3, 30)):
        sl = lambda t: t[bi:bi + 1, :, hi:hi + 1]
        ref_y, ref_hl = oracle.exact_forward(sl(prob.x), sl(prob.a), sl(prob.b), sl(prob.c), h0[bi:bi + 1, hi:hi + 1])
        assert_close(sl(y), ref_y, "bf16", f"many chains y ({bi}, {hi})")
        assert_close(hl[bi:bi + 1, hi:hi + 1], ref_hl, "bf16", f"many chains h_last ({bi}, {hi})")


@pytest.mark.parametrize("layout", ["bthd", "bhtd"])
def test_exact_forward_paired_heads(swr, layout):
    # bf16 heads of 64 channels run two at a time in the one-pass forward
    # (lanes 0-7 one head, 8-15 the other), with the fused sigmoids, the
    # residual and h0, in both layouts, on sequences of more than 16 chunks
    prob = W.random_problem(131, 2, 2300, 4, 64, 64, "bf16", "sigmoid", 3.0, logits=True)
    feat = dict(sigmoid_decay=True, sigmoid_pregate=True)
    x, a, b, c = (to_device(getattr(prob, n), "bf16") for n in "xabc")
    if layout == "bhtd":
        x, a, b, c = (_bhtd(t) for t in (x, a, b, c))
    h0 = _state(np.random.default_rng(19), prob.cfg)
    _say(f"[exact paired] 2x2300x4x64 l64 {layout}")
    y, v, hl = swr.swr_exact_forward(x, a, b, c, 64, h0=torch.from_numpy(h0).cuda(), residual=True,
                                     save_carriers=True, want_h_last=True, **feat)
    torch.cuda.synchronize()
    check_exact(prob, h0, None, y, v, hl, None, residual=True, what=f"paired {layout}", **feat)


@pytest.mark.parametrize("D", [128, 64])
def test_exact_one_pass_time_out_path(swr, monkeypatch, D):
    # The look-back's failure path, forced from the host: with
    # SWR_CHAIN_SPIN_LIMIT=0 a chunk gives up at its first poll that finds a
    # publication missing.  Every kernel still ends; each wait that gave up is
    # counted in the workspace's second int32, and the outputs that depend on
    # it are NaN; every finite output equals the normal call's bit for bit;
    # the next call with the default limit counts nothing and gives the
    # normal results.  Two long sequences (128 chunks each, one workgroup per
    # chunk), so that chunks are waiting while their predecessors compute.
    # d = 64 runs the paired-head forward and the one-pass backward.
    prob = W.random_problem(131 + D, 1, 128 * 128, 2, D, 128, "bf16", "sigmoid", 3.0)
    x, a, b, c, dy = (to_device(getattr(prob, n), "bf16") for n in ("x", "a", "b", "c", "dy"))
    ws = torch.zeros(8 << 20, dtype=torch.int32, device="cuda")

    def forward():
        out = swr.swr_exact_forward(x, a, b, c, 128, save_carriers=True, want_h_last=True, workspace=ws)
        torch.cuda.synchronize()
        return out, int(ws[1].item())

    def backward(v):
        out = swr.swr_exact_backward(x, a, b, c, dy, v, 128, workspace=ws)
        torch.cuda.synchronize()
        return out, int(ws[1].item())

    def check(name, got, ref, count):
        for i, (u, w) in enumerate(zip(got, ref)):
            fin = torch.isfinite(u)
            assert torch.equal(u[fin], w[fin]), (name, i)
            if count == 0:
                assert bool(fin.all()), (name, i)

    _say(f"[exact time-out path] D={D} normal")
    ref_f, n0 = forward()
    assert n0 == 0
    ref_b, n0 = backward(ref_f[1]) if D <= 64 else (None, 0)
    assert n0 == 0
    monkeypatch.setenv("SWR_CHAIN_SPIN_LIMIT", "0")
    _say(f"[exact time-out path] D={D} spin limit 0")
    got_f, nf = forward()
    _say(f"[exact time-out path] forward waits given up: {nf}")
    check("forward", got_f, ref_f, nf)
    if nf > 0:
        assert not bool(torch.isfinite(got_f[0]).all())
    if D <= 64:
        got_b, nb = backward(ref_f[1])
        _say(f"[exact time-out path] backward waits given up: {nb}")
        check("backward", got_b, ref_b, nb)
        if nb > 0:
            assert not bool(torch.isfinite(got_b[0]).all())
    monkeypatch.delenv("SWR_CHAIN_SPIN_LIMIT")
    again_f, n1 = forward()
    assert n1 == 0
    for u, w in zip(again_f, ref_f):
        assert torch.equal(u, w)
