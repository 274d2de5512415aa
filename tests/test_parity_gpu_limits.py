"""GPU parity at the addressing limit: the kernels reach a lane's rows with
32-bit byte offsets from a per-step base, which the library guarantees by
rejecting row strides whose 16-row span exceeds 2^31 bytes.  These tests run
the largest accepted row stride (tensors of several GB, mostly untouched) and
compare the few addressed rows with the oracle."""
import sys

import numpy as np
import pytest

import oracle
import workloads as W
from parity import assert_close, to_host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def swr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2512_13921_amd as lib
    lib.load()
    return lib


@pytest.mark.parametrize("dtype,D", [("bf16", 64), ("f32", 128)])
def test_largest_row_stride(swr, dtype, D):
    es = 2 if dtype == "bf16" else 4
    T, block = 40, 16
    # the largest stride the library accepts, rounded down to whole 16-byte lane slices
    sx_t = ((1 << 31) - 1 - D * es) // (16 * es) // 4 * 4
    print(f"[limits] {dtype} D={D} T={T} row stride {sx_t} elements ({T * sx_t * es / 2**30:.1f} GiB per tensor)",
          flush=True)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    prob = W.random_problem(31, 1, T, 1, D, block, dtype)

    def big(values=None):
        buf = torch.empty(T * sx_t, dtype=tdt, device="cuda")
        view = buf.as_strided((1, T, 1, D), (T * sx_t, sx_t, D, 1))
        if values is not None:
            src = torch.from_numpy(np.ascontiguousarray(values, np.float32)).to(tdt).cuda()
            view.copy_(src)
        return view

    x, b, c, dy = (big(getattr(prob, n)) for n in ("x", "b", "c", "dy"))
    a = torch.from_numpy(np.ascontiguousarray(prob.a, np.float32)).to(tdt).cuda()
    y = big()
    yv, v = swr.swr_forward(x, a, b, c, block, y=y, save_carriers=True)
    outs = (big(), torch.empty(a.shape, dtype=torch.float32, device="cuda"), big(), big())
    grads = swr.swr_backward(x, a, b, c, dy, v, block, outputs=outs)
    torch.cuda.synchronize()
    assert_close(to_host(yv), oracle.forward(prob.x, prob.a, prob.b, prob.c, block), dtype, "limit y")
    ref = oracle.backward(prob.x, prob.a, prob.b, prob.c, prob.dy, block)
    for name, g, r in zip(("dx", "da", "db", "dc"), grads, ref):
        assert_close(to_host(g), r, dtype, f"limit {name}")
    # the uniform window through the same strides
    yu = swr.swr_uniform_forward(x, a, b, c, block, y=y)
    torch.cuda.synchronize()
    assert_close(to_host(yu), oracle.uniform_forward(prob.x, prob.a, prob.b, prob.c, block), dtype,
                 "limit uniform y")
    del x, b, c, dy, y, outs, yv, grads, yu
    torch.cuda.empty_cache()


def test_one_past_the_largest_row_stride_is_rejected(swr):
    D, es = 64, 2
    sx_t = ((1 << 31) - 1 - D * es) // (16 * es) + 1
    p = swr.make_problem(1, 40, 1, D, 16, swr.SWR_DTYPE_BF16, (40 * sx_t, sx_t, D), (40, 1, 1))
    info = swr.load().swr_launch_info
    import ctypes
    v = [ctypes.c_int64() for _ in range(4)]
    assert info(ctypes.byref(p), *(ctypes.byref(t) for t in v)) == -7
