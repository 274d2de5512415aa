"""The oracle's pins catch plausible mistakes: each test here builds a copy of
the oracle's C source with one planted mistake (a wrong window start, a
dropped gate, a decay index off by one, the wrong state in a gradient, ...),
loads it, and checks that the brute-force constructions the pins use
(explicit products, torch autograd) disagree with it.  CPU only; nothing
here touches the GPU library."""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import brute

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "swr_oracle.c")
DP = ctypes.POINTER(ctypes.c_double)


def _mutant(tmp_path, old, new, occurrence=0):
    src = open(SRC).read()
    parts = src.split(old)
    assert len(parts) > occurrence + 1, f"snippet not found: {old!r}"
    mutated = old.join(parts[:occurrence + 1]) + new + old.join(parts[occurrence + 1:])
    assert mutated != src
    c = tmp_path / "mutant.c"
    c.write_text(mutated)
    so = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                    "-I", os.path.join(ROOT, "oracle"), str(c), "-o", str(so)], check=True)
    return ctypes.CDLL(str(so))


def _p(a):
    return np.ascontiguousarray(a, np.float64).ctypes.data_as(DP)


def _inputs(T=23, D=2, seed=0):
    rng = np.random.default_rng(seed)
    x, b, c, dy = (rng.standard_normal((T, D)) for _ in range(4))
    a = rng.uniform(0.1, 1.0, T)
    return x, a, b, c, dy


def _fwd(lib, fn, x, a, b, c, k, flags=0):
    T, D = x.shape
    y = np.zeros((T, D))
    arrs = [np.ascontiguousarray(v, np.float64) for v in (x, a, b, c)]
    getattr(lib, fn)(ctypes.c_int64(T), ctypes.c_int64(D), ctypes.c_int64(k), 0, flags,
                     *(v.ctypes.data_as(DP) for v in arrs), y.ctypes.data_as(DP))
    return y


def _bwd(lib, fn, x, a, b, c, dy, k, flags=0):
    T, D = x.shape
    outs = [np.zeros((T, D)), np.zeros(T), np.zeros((T, D)), np.zeros((T, D))]
    arrs = [np.ascontiguousarray(v, np.float64) for v in (x, a, b, c, dy)]
    getattr(lib, fn)(ctypes.c_int64(T), ctypes.c_int64(D), ctypes.c_int64(k), 0, flags,
                     *(v.ctypes.data_as(DP) for v in arrs), *(o.ctypes.data_as(DP) for o in outs))
    return outs


def _jagged_fwd_caught(lib, residual=False):
    x, a, b, c, _ = _inputs()
    y = _fwd(lib, "swr_oracle_forward_slice", x, a, b, c, 4, 1 if residual else 0)
    return not np.allclose(y, brute.swr_slice(x, a, b, c, 4, residual), rtol=1e-10, atol=1e-10)


def _jagged_bwd_caught(lib):
    x, a, b, c, dy = _inputs()
    got = _bwd(lib, "swr_oracle_backward_slice", x, a, b, c, dy, 4)
    ref = brute.torch_grads(x, a, b, c, dy, 4)
    return any(not np.allclose(g, r, rtol=1e-9, atol=1e-9) for g, r in zip(got, ref))


def _uniform_fwd_caught(lib):
    x, a, b, c, _ = _inputs()
    y = _fwd(lib, "swr_oracle_uniform_forward_slice", x, a, b, c, 4)
    return not np.allclose(y, c * brute.uniform_window_sum(a, b * x, 4), rtol=1e-10, atol=1e-10)


def _uniform_bwd_caught(lib):
    import torch
    x, a, b, c, dy = _inputs()
    got = _bwd(lib, "swr_oracle_uniform_backward_slice", x, a, b, c, dy, 4)
    ts = [torch.tensor(v, requires_grad=True) for v in (x, a, b, c)]
    (brute.torch_uniform(*ts, 4) * torch.tensor(dy)).sum().backward()
    return any(not np.allclose(g, t.grad.numpy(), rtol=1e-9, atol=1e-9) for g, t in zip(got, ts))


def _exact_fwd_caught(lib):
    x, a, b, c, _ = _inputs()
    T, D = x.shape
    h0 = np.random.default_rng(1).standard_normal(D)
    y, hl = np.zeros((T, D)), np.zeros(D)
    arrs = [np.ascontiguousarray(v, np.float64) for v in (x, a, b, c, h0)]
    lib.swr_oracle_exact_forward_slice(ctypes.c_int64(T), ctypes.c_int64(D), 0, 0,
                                       *(v.ctypes.data_as(DP) for v in arrs), y.ctypes.data_as(DP),
                                       hl.ctypes.data_as(DP))
    return not np.allclose(y, c * brute.exact_states(a, b * x, h0), rtol=1e-10, atol=1e-10)


def _step_caught(lib):
    x, a, b, c, _ = _inputs()
    T, D = x.shape
    st, y = np.zeros(2 * D), np.zeros((T, D))
    arrs = [np.ascontiguousarray(v, np.float64) for v in (x, a, b, c)]
    lib.swr_oracle_step_slice(ctypes.c_int64(T), ctypes.c_int64(D), ctypes.c_int64(4), ctypes.c_int64(0), 0, 0,
                              *(v.ctypes.data_as(DP) for v in arrs), st.ctypes.data_as(DP), y.ctypes.data_as(DP))
    return not np.allclose(y, brute.swr_slice(x, a, b, c, 4), rtol=1e-10, atol=1e-10)


MUTANTS = [
    # (name, old, new, occurrence, check)
    ("jagged window without the previous block", "const int64_t start = (tau > 0 ? tau - 1 : 0) * block;",
     "const int64_t start = tau * block;", 0, _jagged_fwd_caught),
    ("forward decay index off by one", "s[mu] = decay(a, a_per_channel, D, m, mu) * s[mu] + b[e] * x[e];",
     "s[mu] = decay(a, a_per_channel, D, m > 0 ? m - 1 : m, mu) * s[mu] + b[e] * x[e];", 0, _jagged_fwd_caught),
    ("residual dropped", "if (flags & SWR_ORACLE_RESIDUAL) y[e] += x[e];", ";", 0,
     lambda lib: _jagged_fwd_caught(lib, residual=True)),
    ("decay gradient from the state after the step", "da[m] += lam[mu] * pre[w];", "da[m] += lam[mu] * post[w];",
     0, _jagged_bwd_caught),
    ("adjoint without the post-gate", "lam[mu] += c[e] * dy[e];", "lam[mu] += dy[e];", 0, _jagged_bwd_caught),
    ("post-gate gradient from the state before the step", "dc[e] = dy[e] * post[w];", "dc[e] = dy[e] * pre[w];",
     0, _jagged_bwd_caught),
    ("pre-gate gradient with the wrong factor", "db[e] = x[e] * du[e];", "db[e] = b[e] * du[e];", 0,
     _jagged_bwd_caught),
    ("exact recurrence ignoring its initial state", "s[mu] = h0 ? h0[mu] : 0.0;", "s[mu] = 0.0;", 0,
     _exact_fwd_caught),
    ("decoding state exchanged one token late", "if (t % block == 0)", "if (t % block == 1)", 0, _step_caught),
    ("uniform window one token too long", "const int64_t start = i - k + 1 > 0 ? i - k + 1 : 0;",
     "const int64_t start = i - k > 0 ? i - k : 0;", 0, _uniform_fwd_caught),
    ("uniform backward window one token too short", "const int64_t start = i - k + 1 > 0 ? i - k + 1 : 0;",
     "const int64_t start = i - k + 2 > 0 ? i - k + 2 : 0;", 1, _uniform_bwd_caught),
    ("uniform pre-gate gradient with the wrong factor", "db[e] = x[e] * du[e];", "db[e] = b[e] * du[e];", 1,
     _uniform_bwd_caught),
]


@pytest.mark.parametrize("name,old,new,occurrence,check", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(tmp_path, name, old, new, occurrence, check):
    lib = _mutant(tmp_path, old, new, occurrence)
    assert check(lib), f"the pins do not catch: {name}"


def test_unmutated_source_passes_the_same_checks(tmp_path):
    lib = _mutant(tmp_path, "/* Decay coefficient of token m, channel mu. */", "/* unchanged */")
    for check in (_jagged_fwd_caught, _jagged_bwd_caught, _uniform_fwd_caught, _uniform_bwd_caught,
                  _exact_fwd_caught, _step_caught):
        assert not check(lib), check.__name__
    assert not _jagged_fwd_caught(lib, residual=True)


def test_shared_gate_mistakes_are_caught(monkeypatch):
    # Gates repeated in the wrong order over the heads (tile instead of
    # repeat), or the group's gradient averaged instead of summed.
    import oracle
    rng = np.random.default_rng(3)
    B, T, H, D, group = 1, 9, 4, 2, 2
    x = rng.standard_normal((B, T, H, D))
    a = rng.uniform(0.1, 1.0, (B, T, H))
    b, c = (rng.standard_normal((B, T, H // group, D)) for _ in range(2))
    dy = rng.standard_normal((B, T, H, D))

    def reference():
        y = np.stack([brute.swr_slice(x[0, :, h], a[0, :, h], b[0, :, h // group], c[0, :, h // group], 4)
                      for h in range(H)], axis=1)[None]
        import torch
        tx, ta, tb, tc = (torch.tensor(v, requires_grad=True) for v in (x, a, b, c))
        ys = torch.stack([brute.torch_forward(tx[0, :, h], ta[0, :, h], tb[0, :, h // group], tc[0, :, h // group], 4)
                          for h in range(H)], 1)[None]
        (ys * torch.tensor(dy)).sum().backward()
        return y, tb.grad.numpy()

    y_ref, db_ref = reference()
    assert np.allclose(oracle.grouped_forward(x, a, b, c, 4, group), y_ref, rtol=1e-12, atol=1e-12)
    with monkeypatch.context() as m:
        m.setattr(oracle, "_expand_heads", lambda g, k: np.tile(np.asarray(g, np.float64), (1, 1, k, 1)))
        assert not np.allclose(oracle.grouped_forward(x, a, b, c, 4, group), y_ref, rtol=1e-10, atol=1e-10)
    real_backward = oracle.backward
    with monkeypatch.context() as m:
        def averaged(*args, **kw):
            dx, da, db, dc = real_backward(*args, **kw)
            return dx, da, db / group, dc / group
        m.setattr(oracle, "backward", averaged)
        _, _, db, _ = oracle.grouped_backward(x, a, b, c, dy, 4, group)
        assert not np.allclose(db, db_ref, rtol=1e-10, atol=1e-10)
