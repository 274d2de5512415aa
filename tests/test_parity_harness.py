"""The whole-tensor comparison used by the full-size GPU parity tests, checked
on the CPU: streamed over chunks it must give the same figures as the metric
evaluated on the whole tensor at once, and it must catch a single wrong
element anywhere."""
import numpy as np
import pytest

import oracle
import workloads as W
from parity import compare_whole, error_stats

torch = pytest.importorskip("torch")


def _bf16(a):
    return W.round_to(np.asarray(a, np.float32), "bf16")


def _setup(B=2, T=300, H=6, D=16, block=32):
    prob = W.random_problem(3, B, T, H, D, block, "bf16")
    y = oracle.forward(prob.x, prob.a, prob.b, prob.c, block)
    da = oracle.backward(prob.x, prob.a, prob.b, prob.c, prob.dy, block)[1]

    def ref_chunk(b, h0, h1):
        args = [np.asarray(getattr(prob, n))[b:b + 1, :, h0:h1] for n in ("x", "a", "b", "c")]
        return dict(y=oracle.forward(*args, block),
                    da=oracle.backward(*args, prob.dy[b:b + 1, :, h0:h1], block)[1])

    return prob, y, da, ref_chunk


@pytest.mark.parametrize("chunk_elems", [1, 300 * 16 * 2, 1 << 30])
def test_streamed_figures_equal_the_whole_tensor_metric(chunk_elems):
    prob, y, da, ref_chunk = _setup()
    got_y, got_da = _bf16(y), da.astype(np.float32)
    outs = [("y", torch.from_numpy(got_y), 2, 1), ("da", torch.from_numpy(got_da), 2, 1)]
    st = compare_whole("harness", "bf16", 2, 6, outs, ref_chunk, chunk_elems=chunk_elems)
    for name, got, ref in (("y", got_y, y), ("da", got_da, da)):
        whole = error_stats(got, ref)
        for key in ("max_e", "mean_e", "max_abs", "mean_abs", "rms"):
            assert st[name][key] == pytest.approx(whole[key], rel=1e-12, abs=1e-300), (name, key)
        assert st[name]["elements"] == ref.size
        assert st[name]["normwise"] == pytest.approx(whole["max_abs"] / np.abs(ref).max(), rel=1e-12)


@pytest.mark.parametrize("where", [(0, 0, 0, 0), (1, 299, 5, 15), (1, 150, 3, 7)])
def test_one_wrong_element_fails(where):
    prob, y, da, ref_chunk = _setup()
    got = _bf16(y)
    got[where] += np.float32(0.05) * max(1.0, abs(float(got[where])))
    outs = [("y", torch.from_numpy(got), 2, 1)]
    with pytest.raises(AssertionError):
        compare_whole("harness", "bf16", 2, 6, outs, ref_chunk, chunk_elems=300 * 16)


def test_non_finite_output_fails():
    prob, y, da, ref_chunk = _setup()
    got = _bf16(y)
    got[1, 7, 2, 3] = np.nan
    with pytest.raises(AssertionError):
        compare_whole("harness", "bf16", 2, 6, [("y", torch.from_numpy(got), 2, 1)], ref_chunk)


def test_grouped_and_state_outputs_are_sliced_per_group():
    # outputs with a head axis of H / group entries (shared gates) and state
    # tensors [B, H, D] (head axis 1), chunked on group boundaries
    group = 3
    prob, y, da, _ = _setup()
    G = 6 // group
    gsum = y.reshape(2, 300, G, group, 16).sum(axis=3)          # [B, T, G, D]
    state = y[:, -1]                                             # [B, H, D]

    def ref_chunk(b, h0, h1):
        assert h0 % group == 0 and h1 % group == 0
        return dict(g=gsum[b:b + 1, :, h0 // group:h1 // group], s=state[b:b + 1, h0:h1])

    outs = [("g", torch.from_numpy(gsum.astype(np.float32)), 2, group),
            ("s", torch.from_numpy(state.astype(np.float32)), 1, 1)]
    st = compare_whole("harness", "f32", 2, 6, outs, ref_chunk, quantum=group, chunk_elems=300 * 16)
    assert st["g"]["elements"] == gsum.size and st["s"]["elements"] == state.size
    assert st["g"]["max_e"] < 1e-6 and st["s"]["max_e"] < 1e-6
