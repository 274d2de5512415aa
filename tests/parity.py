"""Helpers shared by the GPU parity tests: moving seeded inputs to the device,
calling the library through its binding, and the error metric.

Error metric (one number per output tensor Z, against the oracle's float64
result R on the same rounded inputs):  e_i = |Z_i - R_i| / max(|R_i|, rms(R)).
It is relative for elements of typical size and absolute (in units of the
tensor's RMS) for elements near zero, where a relative error means nothing.
"""
import functools

import numpy as np

import workloads as W

# fp32 I/O: relative 1e-5 (scaled as above).
TOL_F32_MAX = 1e-5
# bf16 I/O, fp32 accumulation: max 2e-2 and mean 5e-3 in the scaled metric.
# (Rounding a correct result to bf16 alone gives up to 2^-9 ~ 2e-3 here.)
TOL_BF16_MAX = 2e-2
TOL_BF16_MEAN = 5e-3


def torch_dtype(dtype):
    import torch
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def to_device(arr_f32, dtype, device="cuda"):
    """A device tensor holding exactly the (already rounded) float32 values."""
    import torch
    if dtype == "bf16":
        bits = W.f32_to_bf16_bits(arr_f32).view(np.int16)
        return torch.from_numpy(bits).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(arr_f32, np.float32)).to(device)


def to_host(t):
    """float64 numpy copy of a device tensor (exact for bf16 and fp32)."""
    return t.detach().float().cpu().numpy().astype(np.float64)


def error_stats(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return dict(max_e=0.0, mean_e=0.0, max_abs=0.0, mean_abs=0.0, rms=0.0)
    rms = float(np.sqrt(np.mean(ref * ref)))
    denom = np.maximum(np.abs(ref), rms if rms > 0 else 1.0)
    diff = np.abs(got - ref)
    e = diff / denom
    return dict(max_e=float(e.max()), mean_e=float(e.mean()), max_abs=float(diff.max()),
                mean_abs=float(diff.mean()), rms=rms, nonfinite=int((~np.isfinite(got)).sum()))


def assert_close(got, ref, dtype, what=""):
    st = error_stats(got, ref)
    assert st["nonfinite"] == 0, f"{what}: non-finite values {st}"
    if dtype == "f32":
        assert st["max_e"] <= TOL_F32_MAX, f"{what}: {st}"
    else:
        assert st["max_e"] <= TOL_BF16_MAX and st["mean_e"] <= TOL_BF16_MEAN, f"{what}: {st}"
    return st


def run_gpu(swr, prob, residual=False, run_len=0, backward=True, layout="bthd", carriers=True, **feat):
    """Forward (saving the block carriers) and backward through the library
    (carriers=False: the backward is called without them and recomputes them)."""
    import torch
    cfg = prob.cfg
    dt = cfg.dtype
    x, b, c = (to_device(getattr(prob, n), dt) for n in ("x", "b", "c"))
    a = to_device(prob.a, dt)            # [B, T, H], or [B, T, H, D] for a per-channel decay
    dy = to_device(prob.dy, dt) if backward else None
    if layout == "bhtd":   # store as [B, H, T, D] and hand the library a strided view
        def bhtd(t):
            if t.dim() == 4:
                return t.permute(0, 2, 1, 3).contiguous().permute(0, 2, 1, 3)
            return t.permute(0, 2, 1).contiguous().permute(0, 2, 1)
        x, b, c, a = (bhtd(t) for t in (x, b, c, a))
        if dy is not None:
            dy = bhtd(dy)
    y, v = swr.swr_forward(x, a, b, c, cfg.block, residual=residual, run_len=run_len,
                           save_carriers=True, **feat)
    grads = swr.swr_backward(x, a, b, c, dy, v if carriers else None, cfg.block, residual=residual,
                             run_len=run_len, **feat) if backward else None
    torch.cuda.synchronize()
    return y, grads


def check_full(prob, y, grads, residual=False, what="", **feat):
    """Every output against the oracle on the same inputs; returns the error stats."""
    import oracle
    cfg = prob.cfg
    ref_y = oracle.forward(prob.x, prob.a, prob.b, prob.c, cfg.block, residual, **feat)
    stats = {"y": assert_close(to_host(y), ref_y, cfg.dtype, what + " y")}
    if grads is not None:
        ref = oracle.backward(prob.x, prob.a, prob.b, prob.c, prob.dy, cfg.block, residual, **feat)
        for name, g, r in zip(("dx", "da", "db", "dc"), grads, ref):
            stats[name] = assert_close(to_host(g), r, cfg.dtype, f"{what} {name}")
    return stats


# ----------------------------------------------------------------------------- full-size workloads

@functools.lru_cache(maxsize=3)
def workload(cfg):
    """Seeded inputs of a full-size workload, kept for the next tests that use
    the same one (drawing the headline shape takes tens of seconds).  Callers
    must not modify the arrays."""
    return W.generate(cfg)


# One line per compared output of a whole-tensor check; conftest.py prints
# them in the session's terminal summary, whatever pytest's capture mode.
WHOLE_TENSOR_REPORT = []


def compare_whole(what, dtype, B, H, outputs, ref_chunk, quantum=1, chunk_elems=1 << 24):
    """Every element of every output against the oracle, streamed over chunks
    of (batch entry, run of heads) so that host memory stays bounded.

    outputs: list of (name, tensor, head_axis, div).  The tensor's batch axis
    is 0 and its head axis (2 for [B, T, H, ...], 1 for [B, H, ...] states)
    holds H // div entries (div > 1 for gates shared by groups of div heads).
    ref_chunk(b, h0, h1) returns a dict name -> float64 array shaped like
    tensor[b:b+1] restricted to head entries h0 // div ... h1 // div - 1.
    Chunks hold a multiple of `quantum` heads.

    The scaled metric floors each element's denominator at the reference
    tensor's RMS, so the oracle runs twice: a first pass for the RMS of every
    reference tensor, a second for the comparison.  Returns per-output stats
    (max and mean scaled error, literal max-abs and mean-abs error, and the
    norm-wise max|Z - R| / max|R|)."""
    import torch
    per_head = outputs[0][1].numel() // max(1, B * H)
    hc = max(1, chunk_elems // max(1, per_head)) // quantum * quantum
    hc = min(H, max(quantum, hc))
    chunks = [(b, h0, min(H, h0 + hc)) for b in range(B) for h0 in range(0, H, hc)]
    acc = {name: dict(ss=0.0, n=0, rmax=0.0, emax=0.0, esum=0.0, dmax=0.0, dsum=0.0, bad=0)
           for name, *_ in outputs}
    for b, h0, h1 in chunks:                       # pass 1: the reference's RMS
        ref = ref_chunk(b, h0, h1)
        for name, *_ in outputs:
            r = torch.from_numpy(np.ascontiguousarray(ref[name], np.float64))
            acc[name]["ss"] += float(torch.dot(r.reshape(-1), r.reshape(-1))) if r.numel() else 0.0
            acc[name]["n"] += r.numel()
            acc[name]["rmax"] = max(acc[name]["rmax"], float(r.abs().max()) if r.numel() else 0.0)
    for name, st in acc.items():
        st["rms"] = float(np.sqrt(st["ss"] / st["n"])) if st["n"] else 0.0
    for b, h0, h1 in chunks:                       # pass 2: the comparison
        ref = ref_chunk(b, h0, h1)
        for name, t, axis, div in outputs:
            st = acc[name]
            r = torch.from_numpy(np.ascontiguousarray(ref[name], np.float64))
            g = t.narrow(0, b, 1).narrow(axis, h0 // div, (h1 - h0) // div).cpu().double()
            assert g.shape == r.shape, (what, name, tuple(g.shape), tuple(r.shape))
            st["bad"] += int((~torch.isfinite(g)).sum())
            d = (g - r).abs()
            e = d / r.abs().clamp_min(st["rms"] if st["rms"] > 0 else 1.0)
            if d.numel():
                st["emax"] = max(st["emax"], float(e.max()))
                st["esum"] += float(e.sum())
                st["dmax"] = max(st["dmax"], float(d.max()))
                st["dsum"] += float(d.sum())
    stats = {}
    for name, st in acc.items():
        n = max(1, st["n"])
        s = dict(max_e=st["emax"], mean_e=st["esum"] / n, max_abs=st["dmax"], mean_abs=st["dsum"] / n,
                 normwise=st["dmax"] / st["rmax"] if st["rmax"] > 0 else st["dmax"], rms=st["rms"],
                 elements=st["n"], nonfinite=st["bad"])
        line = (f"{what} {name}: max_e={s['max_e']:.3e} mean_e={s['mean_e']:.3e} "
                f"max_abs={s['max_abs']:.3e} mean_abs={s['mean_abs']:.3e} normwise={s['normwise']:.3e} "
                f"rms={s['rms']:.3g} elements={s['elements']}")
        WHOLE_TENSOR_REPORT.append(line)
        print(line, flush=True)
        stats[name] = s
    for name, s in stats.items():
        assert s["nonfinite"] == 0, f"{what} {name}: non-finite values {s}"
        if dtype == "f32":
            assert s["max_e"] <= TOL_F32_MAX, f"{what} {name}: {s}"
        else:
            assert s["max_e"] <= TOL_BF16_MAX and s["mean_e"] <= TOL_BF16_MEAN, f"{what} {name}: {s}"
    return stats
