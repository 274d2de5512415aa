"""The Python binding refuses tensors on another device than x (a, da, a
workspace): the kernels would dereference their addresses on the GPU."""
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def swr():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2512_13921_amd as lib
    lib.load()
    return lib


def _inputs(H=2, D=64, T=128):
    x = torch.randn(1, T, H, D, device="cuda").to(torch.bfloat16)
    a = torch.full((1, T, H), 0.9, device="cuda").to(torch.bfloat16)
    return x, a


def test_decay_on_the_host_is_refused(swr):
    x, a = _inputs()
    with pytest.raises(ValueError, match="a must be on x's device"):
        swr.swr_forward(x, a.cpu(), x, x, 64)
    with pytest.raises(ValueError, match="a must be on x's device"):
        swr.swr_uniform_forward(x, a.cpu(), x, x, 64)


def test_decay_gradient_on_the_host_is_refused(swr):
    x, a = _inputs()
    y, v = swr.swr_forward(x, a, x, x, 64, save_carriers=True)
    dx, db, dc = (torch.empty_like(x) for _ in range(3))
    da = torch.empty(a.shape, dtype=torch.float32)          # host
    for call in (lambda: swr.swr_backward(x, a, x, x, x, v, 64, outputs=(dx, da, db, dc)),
                 lambda: swr.swr_uniform_backward(x, a, x, x, x, 64, outputs=(dx, da, db, dc))):
        with pytest.raises(ValueError, match="device of a"):
            call()
    torch.cuda.synchronize()


def test_workspace_on_the_host_is_refused(swr):
    x, a = _inputs(H=32)
    y, v = swr.swr_exact_forward(x, a, x, x, 64, save_carriers=True)
    with pytest.raises(ValueError, match="on x's device"):
        swr.swr_exact_backward(x, a, x, x, x, v, 64, workspace=torch.empty(1 << 20))
    g = torch.randn(1, x.shape[1], 1, x.shape[3], device="cuda").to(torch.bfloat16)   # one group of 32
    y, v = swr.swr_forward_shared_gates(x, a, g, g, 64, 32, save_carriers=True)
    with pytest.raises(ValueError, match="on x's device"):
        swr.swr_backward_shared_gates(x, a, g, g, x, v, 64, 32, workspace=torch.empty(1 << 20))
    torch.cuda.synchronize()
