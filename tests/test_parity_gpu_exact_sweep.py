"""A seeded sweep of the exact recurrence over random valid problems: shapes
(ragged T, every block length and head width, odd and even head counts),
both I/O types, both decay modes, the fused sigmoids, the residual, h0
present or not, and the optional outputs; forward and backward against the
oracle.  It reaches every schedule the library picks for the exact calls --
the one-pass forwards (a decay per head, heads of 64 in pairs, a decay per
channel), the three stages, and the one-pass backward on long sequences."""
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


def _cases(n=32, seed=2024):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        D = int(rng.choice([16, 32, 64, 128]))
        block = int(rng.choice([16, 32, 64, 128]))
        long = i % 8 == 7   # a few sequences of 256 chunks or more
        T = int(rng.integers(32768, 34000)) if long else int(rng.integers(1, 5000))
        B = 1 if long else int(rng.integers(1, 4))
        H = 1 if long else int(rng.integers(1, 7))
        D = min(D, 64) if long else D
        dtype, pc = str(rng.choice(["bf16", "f32"])), bool(rng.random() < 0.3)
        if i % 8 == 3:   # bf16 heads of 64 with an even head count: the paired forward
            D, dtype, pc, H = 64, "bf16", False, 2 * int(rng.integers(1, 4))
        out.append(dict(B=B, T=T, H=H, D=D, block=block, dtype=dtype,
                        pc=pc, feat=bool(rng.random() < 0.3),
                        residual=bool(rng.random() < 0.3), h0=bool(rng.random() < 0.7),
                        dhl=bool(rng.random() < 0.5), seed=int(rng.integers(1 << 30))))
    return out


@pytest.mark.parametrize("case", _cases(), ids=lambda c: "B{B}T{T}H{H}D{D}l{block}{dtype}{pcs}".format(
    pcs="pc" if c["pc"] else "", **c))
def test_exact_sweep(swr, case):
    c = case
    print(f"[exact sweep] {c}", flush=True)
    prob = W.random_problem(c["seed"], c["B"], c["T"], c["H"], c["D"], c["block"], c["dtype"], "sigmoid", 3.0,
                            per_channel=c["pc"], logits=c["feat"])
    feat = dict(sigmoid_decay=True, sigmoid_pregate=True) if c["feat"] else {}
    rng = np.random.default_rng(c["seed"] + 1)
    shape = (c["B"], c["H"], c["D"])
    h0 = rng.standard_normal(shape).astype(np.float32) if c["h0"] else None
    dhl = rng.standard_normal(shape).astype(np.float32) if c["dhl"] else None
    dt = c["dtype"]
    x, a, b, cc, dy = (to_device(getattr(prob, n), dt) for n in ("x", "a", "b", "c", "dy"))
    h0_t = None if h0 is None else torch.from_numpy(h0).cuda()
    dhl_t = None if dhl is None else torch.from_numpy(dhl).cuda()
    y, v, hl = swr.swr_exact_forward(x, a, b, cc, c["block"], h0=h0_t, residual=c["residual"], save_carriers=True,
                                     want_h_last=True, **feat)
    grads = swr.swr_exact_backward(x, a, b, cc, dy, v, c["block"], h0=h0_t, dh_last=dhl_t, residual=c["residual"],
                                   want_dh0=True, **feat)
    torch.cuda.synchronize()
    ref_y, ref_hl = oracle.exact_forward(prob.x, prob.a, prob.b, prob.c, h0, c["residual"], **feat)
    assert_close(to_host(y), ref_y, dt, "sweep y")
    assert_close(to_host(hl), ref_hl, "bf16" if dt == "bf16" else "f32", "sweep h_last")
    ref = oracle.exact_backward(prob.x, prob.a, prob.b, prob.c, prob.dy, h0, dhl, c["residual"], **feat)
    for name, g, r in zip(("dx", "da", "db", "dc", "dh0"), grads, ref):
        assert_close(to_host(g), r, dt, f"sweep {name}")
