"""Valid calls through every entry point of the C ABI, for the host-only
sanitizer build (launch_stub.cpp stands in for the kernels and reports that
there is no device).  Run by tests/test_sanitizers.py in a subprocess whose
library is that build; not collected by the main suite.  Each call must get
through validation and launch planning (the stub checks the plan) and come
back with SWR_ERR_HIP; AddressSanitizer and UndefinedBehaviorSanitizer watch
the 64-bit size, stride and overlap arithmetic on the way."""
import ctypes
import itertools

import pytest

import paper_2512_13921_amd as swr

E_HIP = -8
GB = 1 << 30
X, A, B_, C, Y, DY, DX, DA, DB, DC, V, H0, HL, WS, DH0, DHL, ST = (GB * 4 * (i + 1) for i in range(17))
vp = ctypes.c_void_p

SHAPES = [
    # B, T, H, D, block
    (1, 1, 1, 16, 16), (1, 17, 3, 32, 16), (2, 255, 4, 64, 64), (2, 1000, 5, 128, 128),
    (8, 16384, 16, 128, 128), (1, 131072, 32, 64, 128), (16, 8192, 32, 64, 64), (1, 4096, 128, 16, 16),
    (3, 129, 2, 64, 32),
]


def problem(B, T, H, D, block, dtype, layout, per_channel=False, residual=False):
    if layout == "bthd":
        xs, as_ = (T * H * D, H * D, D), (T * H, H, 1)
    else:   # [B, H, T, D] storage described by strides
        xs, as_ = (H * T * D, D, T * D), (H * T, 1, T)
    return swr.make_problem(B, T, H, D, block, dtype, xs, as_, residual, 0, per_channel)


CASES = list(itertools.product(SHAPES, (swr.SWR_DTYPE_BF16, swr.SWR_DTYPE_F32), ("bthd", "bhtd"),
                               (False, True)))


@pytest.mark.parametrize("shape,dtype,layout,pc", CASES)
def test_valid_calls_reach_the_launch(shape, dtype, layout, pc):
    lib = swr.load()
    p = problem(*shape, dtype, layout, per_channel=pc)
    P = ctypes.byref(p)
    assert lib.swr_forward(P, vp(X), vp(A), vp(B_), vp(C), vp(Y), vp(V), None) == E_HIP
    assert lib.swr_carriers(P, vp(X), vp(A), vp(B_), vp(V), None) == E_HIP
    assert lib.swr_backward(P, vp(X), vp(A), vp(B_), vp(C), vp(DY), vp(V), vp(DX), vp(DA), vp(DB),
                            vp(DC), None) == E_HIP
    assert lib.swr_exact_forward(P, vp(X), vp(A), vp(B_), vp(C), vp(H0), vp(Y), vp(V), vp(HL), vp(WS),
                                 None) == E_HIP
    assert lib.swr_exact_backward(P, vp(X), vp(A), vp(B_), vp(C), vp(DY), vp(H0), vp(V), vp(DHL), vp(DX),
                                  vp(DA), vp(DB), vp(DC), vp(DH0), vp(WS), None) == E_HIP
    assert lib.swr_carrier_elems(P) == shape[0] * shape[2] * -(-shape[1] // shape[4]) * shape[3]
    assert lib.swr_exact_workspace_bytes(P) >= 0
    info = swr.swr_launch_info(p)
    assert info["fwd_workgroups"] >= 1 and info["bwd_workgroups"] >= 1
    if not pc:
        assert lib.swr_uniform_forward(P, vp(X), vp(A), vp(B_), vp(C), vp(Y), None) == E_HIP
        assert lib.swr_uniform_backward(P, vp(X), vp(A), vp(B_), vp(C), vp(DY), vp(DX), vp(DA), vp(DB),
                                        vp(DC), None) == E_HIP
