"""A seeded sweep of the jagged window (swr_forward / swr_backward) over
random valid problems: ragged T, every block length, head widths that are
any multiple of 16 up to 256, odd and even head counts, both I/O types and
decay modes, the fused sigmoids, the residual, the [B, H, T, d] layout, and
the backward with saved or recomputed block carriers; every output against
the oracle."""
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


def _bhtd(t):
    # stored as [B, H, T, ...], handed over as a strided [B, T, H, ...] view
    if t.dim() == 4:
        return t.permute(0, 2, 1, 3).contiguous().permute(0, 2, 1, 3)
    return t.permute(0, 2, 1).contiguous().permute(0, 2, 1)


def _cases(n=32, seed=4051):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        pc = bool(rng.random() < 0.3)
        widths = [16, 32, 48, 64, 80, 96, 112, 128, 144, 160, 192, 224, 240, 256]
        D = int(rng.choice(widths))
        out.append(dict(B=int(rng.integers(1, 4)), T=int(rng.integers(1, 3000)), H=int(rng.integers(1, 7)), D=D,
                        block=int(rng.choice([16, 32, 64, 128])), dtype=str(rng.choice(["bf16", "f32"])), pc=pc,
                        feat=bool(rng.random() < 0.3), residual=bool(rng.random() < 0.3),
                        bhtd=bool(rng.random() < 0.25), carriers=bool(rng.random() < 0.7),
                        seed=int(rng.integers(1 << 30))))
    return out


@pytest.mark.parametrize("case", _cases(), ids=lambda c: "B{B}T{T}H{H}D{D}l{block}{dtype}{pcs}".format(
    pcs="pc" if c["pc"] else "", **c))
def test_jagged_sweep(swr, case):
    c = case
    print(f"[sweep] {c}", flush=True)
    prob = W.random_problem(c["seed"], c["B"], c["T"], c["H"], c["D"], c["block"], c["dtype"], "sigmoid", 2.0,
                            per_channel=c["pc"], logits=c["feat"])
    feat = dict(sigmoid_decay=True, sigmoid_pregate=True) if c["feat"] else {}
    dt = c["dtype"]
    x, a, b, cc, dy = (to_device(getattr(prob, n), dt) for n in ("x", "a", "b", "c", "dy"))
    if c["bhtd"]:
        x, a, b, cc, dy = (_bhtd(t) for t in (x, a, b, cc, dy))
    y, v = swr.swr_forward(x, a, b, cc, c["block"], residual=c["residual"], save_carriers=True, **feat)
    grads = swr.swr_backward(x, a, b, cc, dy, v if c["carriers"] else None, c["block"], residual=c["residual"],
                             **feat)
    torch.cuda.synchronize()
    ref_y = oracle.forward(prob.x, prob.a, prob.b, prob.c, c["block"], c["residual"], **feat)
    assert_close(to_host(y), ref_y, dt, "sweep y")
    ref = oracle.backward(prob.x, prob.a, prob.b, prob.c, prob.dy, c["block"], c["residual"], **feat)
    for name, g, r in zip(("dx", "da", "db", "dc"), grads, ref):
        assert_close(to_host(g), r, dt, f"sweep {name}")


def _cases_other(n=16, seed=977):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        out.append(dict(B=int(rng.integers(1, 4)), T=int(rng.integers(1, 2500)), D=int(rng.choice([16, 32, 64, 128])),
                        block=int(rng.choice([16, 32, 64, 128])), dtype=str(rng.choice(["bf16", "f32"])),
                        feat=bool(rng.random() < 0.3), residual=bool(rng.random() < 0.3),
                        group=int(rng.choice([1, 2, 4])), G=int(rng.integers(1, 4)), seed=int(rng.integers(1 << 30))))
    return out


@pytest.mark.parametrize("case", _cases_other(), ids=lambda c: "B{B}T{T}D{D}k{block}{dtype}".format(**c))
def test_uniform_sweep(swr, case):
    # the uniform window (window = block tokens; one decay per head)
    c = case
    H = c["G"] * c["group"]
    print(f"[uniform sweep] {c}", flush=True)
    prob = W.random_problem(c["seed"], c["B"], c["T"], H, c["D"], c["block"], c["dtype"], "sigmoid", 2.0,
                            logits=c["feat"])
    feat = dict(sigmoid_decay=True, sigmoid_pregate=True) if c["feat"] else {}
    dt = c["dtype"]
    x, a, b, cc, dy = (to_device(getattr(prob, n), dt) for n in ("x", "a", "b", "c", "dy"))
    y = swr.swr_uniform_forward(x, a, b, cc, c["block"], residual=c["residual"], **feat)
    grads = swr.swr_uniform_backward(x, a, b, cc, dy, c["block"], residual=c["residual"], **feat)
    torch.cuda.synchronize()
    ref_y = oracle.uniform_forward(prob.x, prob.a, prob.b, prob.c, c["block"], c["residual"], **feat)
    assert_close(to_host(y), ref_y, dt, "uniform sweep y")
    ref = oracle.uniform_backward(prob.x, prob.a, prob.b, prob.c, prob.dy, c["block"], c["residual"], **feat)
    for name, g, r in zip(("dx", "da", "db", "dc"), grads, ref):
        assert_close(to_host(g), r, dt, f"uniform sweep {name}")


@pytest.mark.parametrize("case", _cases_other(seed=978), ids=lambda c: "B{B}T{T}G{G}x{group}D{D}l{block}{dtype}".format(**c))
def test_shared_gates_sweep(swr, case):
    # gates shared by groups of heads: b and c [B, T, H / group, D]
    c = case
    H = c["G"] * c["group"]
    print(f"[shared gates sweep] {c}", flush=True)
    prob = W.random_problem(c["seed"], c["B"], c["T"], H, c["D"], c["block"], c["dtype"], "sigmoid", 2.0,
                            logits=c["feat"])
    feat = dict(sigmoid_decay=True, sigmoid_pregate=True) if c["feat"] else {}
    dt = c["dtype"]
    bg = np.ascontiguousarray(prob.b[:, :, ::c["group"]])
    cg = np.ascontiguousarray(prob.c[:, :, ::c["group"]])
    x, a, dy = (to_device(getattr(prob, n), dt) for n in ("x", "a", "dy"))
    b, cc = to_device(bg, dt), to_device(cg, dt)
    y, v = swr.swr_forward_shared_gates(x, a, b, cc, c["block"], c["group"], residual=c["residual"],
                                        save_carriers=True, **feat)
    grads = swr.swr_backward_shared_gates(x, a, b, cc, dy, v, c["block"], c["group"], residual=c["residual"], **feat)
    torch.cuda.synchronize()
    ref_y = oracle.grouped_forward(prob.x, prob.a, bg, cg, c["block"], c["group"], c["residual"], **feat)
    assert_close(to_host(y), ref_y, dt, "gates sweep y")
    ref = oracle.grouped_backward(prob.x, prob.a, bg, cg, prob.dy, c["block"], c["group"], c["residual"], **feat)
    for name, g, r in zip(("dx", "da", "db", "dc"), grads, ref):
        assert_close(to_host(g), r, dt, f"gates sweep {name}")
