#!/usr/bin/env python3
"""Benchmark of the Sliding Window Recurrence hot path on one MI355X.

One step = one forward (swr_forward) and one backward (swr_backward) pass over
the whole workload, inputs already resident in HBM.  Prints ONE JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 3] [--decay head|channel]

--decay channel times the per-channel-decay path (a and da of shape
[B, T, H, D]) on the same workload shape instead of the shared decay.
--sigmoid feeds a and b as logits through the kernels' fused sigmoid (the
Phalanx featurisation); a's logits are then drawn N(3, 1).
--recurrence exact times the exact (untruncated) recurrence instead of the
jagged window: swr_exact_forward / swr_exact_backward, three launches each
(run aggregates, carrier scan, reconstruction), timed as a whole.
--recurrence uniform times the uniform window of the same length (every token
sees its `block` most recent tokens): swr_uniform_forward / swr_uniform_backward.
--gate-groups G shares b and c across groups of H/G heads (the Phalanx gate
sharing): swr_forward_shared_gates / swr_backward_shared_gates, the backward
timed with its group reduction.

Throughput is tokens/s = B*T / (time of one forward + one backward).  Kernel
durations come from HIP events recorded on the stream the kernels run on.
The roofline entry reports the dominant kernel's algorithmic HBM bytes per
launch (every input read once, every output written once) divided by its
average duration, against the MI355X's 8 TB/s.  The CPU baseline times the
double-precision oracle on a bounded sample of the same workload on this
machine's host cores.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402

METRIC = "SWR fwd+bwd tokens/sec and achieved HBM GB/s at B=8,H=16,d=128,T=16384"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E peak
BF16_MFMA_PEAK_TFLOPS = 2500.0 # dense bf16 MFMA peak
F32_MFMA_PEAK_TFLOPS = 157.3


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def algorithmic_bytes(cfg, backward, with_carriers=True, gate_groups=0):
    """HBM bytes one launch must move: inputs read once, outputs written once.
    The block carriers (4*D bytes per block per (batch, head), written by the
    forward and read by the backward: 4*D/block bytes per token-head) are part
    of the algorithm's state and are counted (the uniform window has none)."""
    e = 2 if cfg.dtype == "bf16" else 4
    th = cfg.B * cfg.T * cfg.H
    carriers = th * 4 * cfg.D // cfg.block if with_carriers else 0
    na = cfg.D if cfg.per_channel else 1     # decays per token-head
    if gate_groups:   # b, c (and db, dc) once per group of heads
        tg = cfg.B * cfg.T * gate_groups
        if backward:
            return th * (e * (3 * cfg.D + na) + 4 * na) + tg * e * 4 * cfg.D + carriers
        return th * e * (2 * cfg.D + na) + tg * e * 2 * cfg.D + carriers
    if backward:   # x, b, c, dy, a, carriers in; dx, db, dc out; da out in fp32
        return th * (e * (7 * cfg.D + na) + 4 * na) + carriers
    return th * e * (4 * cfg.D + na) + carriers   # x, b, c, a in; y, carriers out


def contraction_flops(cfg, backward, uniform=False):
    """Dense flops of the intra-block contractions (16x16 sub-block tiles):
    2 * 16 * D per token-head per contraction; the jagged backward runs two
    (the forward's local solve recomputed, and the reverse solve; the one
    reverse solve per run for the block after it is left out); the uniform
    window's forward two (local and strict-suffix solves) and its backward six
    (local, reverse, prefix and previous block's suffix solves, and the two
    solves of its decay gradient).  None for a per-channel decay, whose local
    solves are scans on the vector ALUs."""
    if cfg.per_channel:
        return None
    per = 2 * 16 * cfg.D * cfg.B * cfg.T * cfg.H
    if uniform:
        return per * (6 if backward else 2)
    return per * (2 if backward else 1)


# The sources that decide what a launch does (kernels, grid policy): the
# recorded traffic is stale once any of them changes.
KERNEL_SOURCES = ("swr_kernels.hip", "swr_uniform.hip", "swr_groups.hip", "swr_chain.hip", "swr_device.h", "swr_api.cpp",
                  "swr_launch.h")


def recorded(kernel, workload, what="traffic"):
    """A record measured with rocprofv3 counters for this kernel and workload
    and kept in profiles/ -- "traffic" (HBM bytes per launch) or "counters"
    (matrix-pipe utilisation, executed MFMA flops, VALU busy, occupancy) --
    or None when a kernel or launch-policy source has changed since the
    counters were taken."""
    import hashlib
    import re
    csrc = os.path.join(ROOT, "paper_2512_13921_amd", "csrc")
    prof = os.path.join(ROOT, "profiles", f"{kernel}_{workload}.md")
    if not os.path.exists(prof):
        return None
    m = re.search(r"<!-- " + what + r": (\{.*\}) -->", open(prof).read())
    if not m:
        return None
    rec = json.loads(m.group(1))
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        h.update(open(os.path.join(csrc, name), "rb").read())
    sha = h.hexdigest()
    return rec if rec.get("kernel_sha256") == sha else None


def to_device(arr, dtype):
    import torch
    if dtype == "bf16":
        bits = W.f32_to_bf16_bits(arr).view(np.int16)
        return torch.from_numpy(bits).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(arr, np.float32)).cuda()


def _cpu_model():
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(cfg, prob, budget_s=10.0, exact=False, uniform=False):
    """Oracle throughput on whole (batch, head) slices of the workload, in
    tokens/s of the full job (a token carries all H heads).  Slices are taken
    in a fixed shuffled order and revisited until about budget_s seconds of
    oracle time have been spent on all host cores (forward and backward timed
    separately); then one slice's forward and backward run on one core."""
    import oracle
    threads = oracle.max_threads()
    nslices = cfg.B * cfg.H
    batch = max(1, min(threads, nslices))
    order = np.random.default_rng(0).permutation(nslices)

    def take_slices(idx):
        bi, hi = idx // cfg.H, idx % cfg.H

        def take(t):
            return np.ascontiguousarray(np.asarray(t)[bi, :, hi], dtype=np.float64)

        return [take(getattr(prob, n)) for n in ("x", "a", "b", "c", "dy")]

    def run(xs, as_, bs, cs, dys):
        """(forward seconds, backward seconds) of the oracle on these slices."""
        t0 = time.perf_counter()
        if cfg.logits:     # the featurisation is part of the timed work
            as_, bs = oracle.sigmoid(as_), oracle.sigmoid(bs)
        if exact:
            oracle.exact_forward_slices(xs, as_, bs, cs)
        elif uniform:
            oracle.uniform_forward_slices(xs, as_, bs, cs, cfg.block)
        else:
            oracle.forward_slices(xs, as_, bs, cs, cfg.block)
        t1 = time.perf_counter()
        if exact:
            oracle.exact_backward_slices(xs, as_, bs, cs, dys)
        elif uniform:
            oracle.uniform_backward_slices(xs, as_, bs, cs, dys, cfg.block)
        else:
            oracle.backward_slices(xs, as_, bs, cs, dys, cfg.block)
        return t1 - t0, time.perf_counter() - t1

    done, t_fwd, t_bwd, passes, pos = 0, 0.0, 0.0, 0, 0
    while t_fwd + t_bwd < budget_s or done == 0:
        idx = order[pos:pos + batch]
        f, b = run(*take_slices(idx))
        t_fwd, t_bwd = t_fwd + f, t_bwd + b
        done += len(idx)
        pos += len(idx)
        if pos >= nslices:
            pos, passes = 0, passes + 1
    # one core, one slice
    oracle.set_threads(1)
    try:
        f1, b1 = run(*take_slices(order[:1]))
    finally:
        oracle.set_threads(threads)
    tokens = done * cfg.T / cfg.H          # full-job tokens the sample stands for
    tok1 = cfg.T / cfg.H
    return {
        "value": tokens / (t_fwd + t_bwd),
        "unit": "tokens/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"{done} (batch, head) slices of {nslices} (full T={cfg.T}; {passes} full passes), "
                  f"forward+backward in float64, OpenMP over slices; {t_fwd + t_bwd:.1f} s of oracle time",
        "forward_tokens_per_s": tokens / t_fwd,
        "backward_tokens_per_s": tokens / t_bwd,
        "single_core": {"value": tok1 / (f1 + b1), "forward_tokens_per_s": tok1 / f1,
                        "backward_tokens_per_s": tok1 / b1, "sample": "one (batch, head) slice"},
        "cpu_model": _cpu_model(),
    }


# The paper's forward times of its B2P kernel at this shape (Sec. 6, the
# mixer forward-time figure; H100, batch not stated), in ms.
PAPER_B2P_FWD_MS = {1024: 0.04324, 2048: 0.07401, 4096: 0.115, 8192: 0.201, 16384: 0.362,
                    32768: 0.682, 65536: 1.31, 131072: 2.568, 262144: 5.055, 524288: 10.033}


def paper_shape_bench(args, swr, torch):
    """Forward-only sweep at the shape the paper times its own kernel on
    (model width 2048 as 128 heads of 16 channels, block 16), B = 1, bf16,
    synthetic inputs drawn on the device.  The paper's numbers come from
    another GPU and are context, not a target."""
    H, D, l = 128, 16, 16
    rows = []
    g = torch.Generator(device="cuda").manual_seed(0)
    for T in sorted(PAPER_B2P_FWD_MS):
        x, b, c = (torch.randn(1, T, H, D, device="cuda", generator=g).to(torch.bfloat16) for _ in range(3))
        a = torch.sigmoid(torch.randn(1, T, H, device="cuda", generator=g) + 3.0).to(torch.bfloat16)
        y = torch.empty_like(x)
        for _ in range(args.warmup):
            swr.swr_forward(x, a, b, c, l, y=y)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            swr.swr_forward(x, a, b, c, l, y=y)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        nbytes = T * H * 2 * (4 * D + 1)
        rows.append({"T": T, "ms": ms, "GB/s": nbytes / (ms * 1e-3) / 1e9, "tokens_per_s": T / (ms * 1e-3),
                     "paper_ms": PAPER_B2P_FWD_MS[T]})
        log(f"[paper shape] T={T}: {ms * 1e3:.1f} us ({rows[-1]['GB/s']:.0f} GB/s), paper {PAPER_B2P_FWD_MS[T] * 1e3:.1f} us")
        del x, b, c, a, y
    out = {"metric": "SWR forward time at the paper's mixer shape (B=1, D=2048 = 128 heads x 16, block 16)",
           "value": rows[-1]["tokens_per_s"], "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": rows[-1]["ms"], "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded device draws)",
           "config": {"workload": "paper_shape_B1_H128_d16_l16_forward", "sweep": rows},
           "cpu_baseline": None}
    print(json.dumps(out), flush=True)
    return 0


def decode_bench(args, cfg, swr, torch):
    """Recurrent decoding: K=1 token for each of the B sequences per call, at
    sequence positions following a prompt of the workload's length T.  A
    step is one call; its time is launch-bound (B*H*D channels of a few flops
    each), so the line reports tokens/s and microseconds per step, and the
    bytes a step must move (inputs, outputs, the state read and written)."""
    exact = args.recurrence == "exact"
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    B, H, D = cfg.B, cfg.H, cfg.D
    g = torch.Generator(device="cuda").manual_seed(cfg.seed)
    n = args.steps
    x, b, c = (torch.randn(B, n, H, D, device="cuda", generator=g).to(dt) for _ in range(3))
    per_channel = args.decay == "channel"
    a = torch.sigmoid(torch.randn((B, n, H, D) if per_channel else (B, n, H), device="cuda",
                                  generator=g) + 3.0).to(dt)
    y = torch.empty_like(x)
    state = torch.zeros((B, H, D) if exact else (B, H, 2, D), dtype=torch.float32, device="cuda")
    t0 = cfg.T

    def step(i, out):
        s = slice(i, i + 1)
        if exact:
            swr.swr_exact_step(x[:, s], a[:, s], b[:, s], c[:, s], state, y=out[:, s])
        else:
            swr.swr_step(x[:, s], a[:, s], b[:, s], c[:, s], cfg.block, t0 + i, state, y=out[:, s])

    for i in range(min(args.warmup, n)):
        step(i, y)
    torch.cuda.synchronize()
    # Eager calls: what a Python caller sees (host launch overhead included).
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(n):
        step(i, y)
    e1.record()
    torch.cuda.synchronize()
    ms_eager = e0.elapsed_time(e1) / n
    # The same n steps captured once in a HIP graph and replayed: the device
    # time per step, as a decoder that captures its step would see it.
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for i in range(n):
                step(i, y)
    torch.cuda.current_stream().wait_stream(s)
    g.replay()
    torch.cuda.synchronize()
    e0.record()
    g.replay()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / n
    e = 2 if cfg.dtype == "bf16" else 4
    nbytes = B * H * (e * (3 * D + (D if per_channel else 1)) + e * D + 4 * D * (2 if exact else 4))
    out = {
        "metric": "SWR recurrent decoding step (one token per sequence)",
        "value": B / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": n, "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded device draws)",
        "config": {"workload": cfg.name + ("_perchannel" if per_channel else "") + ("_exact" if exact else "")
                   + "_decode", "B": B, "H": H, "d": D, "block": cfg.block, "prompt_len": cfg.T,
                   "decay": "per channel" if per_channel else "per head",
                   "recurrence": "exact (untruncated)" if exact else "jagged window"},
        "bytes_per_step": nbytes,
        "us_per_step": ms * 1e3,
        "us_per_step_eager": ms_eager * 1e3,
        "timing": "HIP graph of the timed steps, replayed once (us_per_step_eager: Python calls)",
        "GB/s": nbytes / (ms * 1e-3) / 1e9,
        "cpu_baseline": None,
    }
    print(json.dumps(out), flush=True)
    return 0


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=W.HEADLINE, choices=sorted(W.CONFIGS))
    ap.add_argument("--run-len", type=int, default=0, help="tokens per workgroup run (0 = library default)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--decay", choices=("head", "channel"), default="head",
                    help="one decay per token and head (default) or per token, head and channel")
    ap.add_argument("--sigmoid", action="store_true",
                    help="a and b are logits; the kernels apply the sigmoid (fused featurisation)")
    ap.add_argument("--recurrence", choices=("window", "exact", "uniform"), default="window",
                    help="the jagged-window recurrence (default), the exact, untruncated one, or "
                         "the uniform window of the same length")
    ap.add_argument("--gate-groups", type=int, default=0,
                    help="share b and c across this many groups of heads (0: no sharing)")
    ap.add_argument("--paper-shape", action="store_true",
                    help="forward-only sweep at the paper's own mixer-timing shape (B=1, D=2048 as "
                         "H=128 heads of d=16, block 16, bf16) over T = 1K .. 512K")
    ap.add_argument("--channels", type=int, default=0,
                    help="channels per head d (any multiple of 16 up to 256) in place of the workload's, "
                         "with B, T, H and the rest of the recipe unchanged")
    ap.add_argument("--no-carriers", action="store_true",
                    help="the jagged window without saved block carriers: the forward keeps none "
                         "and the backward recomputes them (the problem statement's call shape)")
    ap.add_argument("--decode", action="store_true",
                    help="time recurrent decoding instead: one token per sequence per call "
                         "(swr_step / swr_exact_step) after a prompt of the workload's length")
    args = ap.parse_args()

    if args.gpus != 1:
        print("bench.py measures one GPU only: the SWR hot path here runs on a single MI355X "
              "and has no multi-GPU path (use --gpus 1).", file=sys.stderr)
        return 2

    import torch
    import paper_2512_13921_amd as swr

    if not torch.cuda.is_available():
        print("no GPU visible: bench.py needs an MI355X", file=sys.stderr)
        return 1
    swr.load()

    cfg = W.CONFIGS[args.config]
    if args.recurrence == "uniform" and (args.decode or args.paper_shape):
        print("--recurrence uniform times the forward and backward passes only", file=sys.stderr)
        return 2
    if args.decode:
        return decode_bench(args, cfg, swr, torch)
    if args.paper_shape:
        return paper_shape_bench(args, swr, torch)
    if args.decay == "channel":
        cfg = W.PER_CHANNEL.get(args.config) or cfg.with_(name=cfg.name + "_perchannel", per_channel=True)
    if args.sigmoid:
        cfg = cfg.with_(name=cfg.name + "_sigmoid", logits=True, a_kind="sigmoid",
                        a_mu=cfg.a_mu if cfg.a_kind == "sigmoid" else 3.0)
    feat = dict(sigmoid_decay=args.sigmoid, sigmoid_pregate=args.sigmoid)
    exact = args.recurrence == "exact"
    uniform = args.recurrence == "uniform"
    if exact:
        cfg = cfg.with_(name=cfg.name + "_exact")
    if uniform:
        if cfg.per_channel:
            print("the uniform window supports one decay per head only", file=sys.stderr)
            return 2
        cfg = cfg.with_(name=cfg.name + "_uniform")
    groups = args.gate_groups
    if groups:
        if cfg.per_channel or exact or uniform or groups < 1 or cfg.H % groups:
            print("--gate-groups needs the jagged window, one decay per head and a divisor of H",
                  file=sys.stderr)
            return 2
        cfg = cfg.with_(name=cfg.name + f"_gates{groups}")
    if args.channels:
        if uniform or groups or (exact and args.channels not in (16, 32, 64, 128)):
            print("--channels applies to the jagged window's own entry points, and to the exact "
                  "recurrence with 16, 32, 64 or 128 channels", file=sys.stderr)
            return 2
        cfg = cfg.with_(D=args.channels, name=cfg.name.replace(f"_d{cfg.D}", f"_d{args.channels}"))
    nocar = args.no_carriers
    if nocar:
        if exact or uniform or groups:
            print("--no-carriers applies to the jagged window's own entry points only", file=sys.stderr)
            return 2
        cfg = cfg.with_(name=cfg.name + "_nocarriers")
    if not cfg.backward:
        cfg = cfg.with_(backward=True)
    log(f"[bench] workload {cfg.name}: generating inputs")
    prob = W.generate(cfg)
    x, a, b, c, dy = (to_device(getattr(prob, n), cfg.dtype) for n in ("x", "a", "b", "c", "dy"))
    y = torch.empty_like(x)
    dx, db, dc = (torch.empty_like(x) for _ in range(3))
    da = torch.empty(a.shape, dtype=torch.float32, device=a.device)   # a's shape, contiguous
    carriers = torch.empty(swr.carrier_shape(x, cfg.block), dtype=torch.float32, device=x.device)
    stream = torch.cuda.current_stream()
    if groups:   # each group's gates: those drawn for its first head
        gsz = cfg.H // groups
        b, c = b[:, :, ::gsz].contiguous(), c[:, :, ::gsz].contiguous()
        db, dc = torch.empty_like(b), torch.empty_like(c)
        gprob = swr.make_problem(cfg.B, cfg.T, cfg.H, cfg.D, cfg.block, 1 if cfg.dtype == "bf16" else 0,
                                 x.stride()[:3], a.stride()[:3])
        gbytes = swr.swr_shared_gates_workspace_bytes(gprob, gsz)
        gws = torch.empty(gbytes // 4, dtype=torch.float32, device=x.device) if gbytes else None
    if exact:
        wsp = swr.make_problem(cfg.B, cfg.T, cfg.H, cfg.D, cfg.block, 1 if cfg.dtype == "bf16" else 0,
                               x.stride()[:3], a.stride()[:3], False, args.run_len, cfg.per_channel)
        workspace = torch.empty(max(swr.swr_exact_workspace_bytes(wsp) // 4, 1), dtype=torch.float32,
                                device=x.device)
    torch.cuda.synchronize()

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        if exact:
            swr.swr_exact_forward(x, a, b, c, cfg.block, y=y, carriers=carriers, workspace=workspace,
                                  run_len=args.run_len, **feat)
        elif uniform:
            swr.swr_uniform_forward(x, a, b, c, cfg.block, y=y, run_len=args.run_len, **feat)
        elif groups:
            swr.swr_forward_shared_gates(x, a, b, c, cfg.block, gsz, y=y, carriers=carriers,
                                         run_len=args.run_len, **feat)
        else:
            swr.swr_forward(x, a, b, c, cfg.block, y=y, carriers=None if nocar else carriers,
                            run_len=args.run_len, **feat)
        if ev is not None:
            ev[1].record(stream)
        if exact:
            swr.swr_exact_backward(x, a, b, c, dy, carriers, cfg.block, outputs=(dx, da, db, dc),
                                   workspace=workspace, run_len=args.run_len, **feat)
        elif uniform:
            swr.swr_uniform_backward(x, a, b, c, dy, cfg.block, outputs=(dx, da, db, dc),
                                     run_len=args.run_len, **feat)
        elif groups:
            swr.swr_backward_shared_gates(x, a, b, c, dy, carriers, cfg.block, gsz, outputs=(dx, da, db, dc),
                                          workspace=gws, run_len=args.run_len, **feat)
        else:
            swr.swr_backward(x, a, b, c, dy, None if nocar else carriers, cfg.block, outputs=(dx, da, db, dc),
                             run_len=args.run_len, **feat)
        if ev is not None:
            ev[2].record(stream)

    log(f"[bench] warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    log(f"[bench] timing {args.steps} steps")
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    for i in range(args.steps):
        step(events[i])
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall

    fwd_ms = np.array([e[0].elapsed_time(e[1]) for e in events])
    bwd_ms = np.array([e[1].elapsed_time(e[2]) for e in events])
    total_ms = float(events[0][0].elapsed_time(events[-1][2]))
    ms_per_step = total_ms / args.steps
    tokens = cfg.B * cfg.T
    value = tokens / (ms_per_step * 1e-3)

    fb = algorithmic_bytes(cfg, False, not (uniform or nocar), groups)
    bb = algorithmic_bytes(cfg, True, not (uniform or nocar), groups)
    f_gbs, b_gbs = fb / (fwd_ms.mean() * 1e-3) / 1e9, bb / (bwd_ms.mean() * 1e-3) / 1e9
    dominant_bwd = bwd_ms.mean() >= fwd_ms.mean()
    dom_gbs = b_gbs if dominant_bwd else f_gbs
    pc = "_pc" if cfg.per_channel else ""
    dom_kernel = f"swr_bwd{pc}_kernel" if dominant_bwd else f"swr_fwd{pc}_kernel"
    if uniform:
        dom_kernel = "swr_uni_bwd_kernel" if dominant_bwd else "swr_uni_fwd_kernel"
    if groups and dominant_bwd:   # two launches, timed together
        dom_kernel = ("swr_bwd_grouped_kernel" if not gbytes else
                      "swr_backward_shared_gates (swr_bwd_kernel + swr_gate_reduce_kernel)")
    # The exact recurrence's passes are three launches each; their time is
    # taken as a whole and no single kernel's counters stand for it.
    traffic = None if exact or groups else recorded(dom_kernel, cfg.name, "traffic")
    counters = None if exact or groups else recorded(dom_kernel, cfg.name, "counters")
    if exact:
        dom_kernel = ("swr_exact_backward (swr_bwd_agg_kernel + swr_scan_kernel + swr_bwd_kernel)"
                      if dominant_bwd else
                      "swr_exact_forward (swr_fwd_kernel aggregate + swr_scan_kernel + swr_fwd_kernel)")
    mfma_peak = BF16_MFMA_PEAK_TFLOPS if cfg.dtype == "bf16" else F32_MFMA_PEAK_TFLOPS

    def mfma_rate(backward, ms):
        f = contraction_flops(cfg, backward, uniform)
        return None if f is None else f / (ms * 1e-3) / 1e12

    launch = (swr.swr_uniform_launch_info if uniform else swr.swr_launch_info)(swr.make_problem(
        cfg.B, cfg.T, cfg.H, cfg.D, cfg.block, 1 if cfg.dtype == "bf16" else 0,
        x.stride()[:3], a.stride()[:3], False, args.run_len, cfg.per_channel))

    # Reference: a plain device-to-device copy of one [B,T,H,D] tensor (read + write).
    cbuf = torch.empty_like(x)
    ce = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for _ in range(3):
        cbuf.copy_(x)
    ce[0].record(stream)
    for _ in range(10):
        cbuf.copy_(x)
    ce[1].record(stream)
    torch.cuda.synchronize()
    copy_gbs = 2 * x.numel() * x.element_size() * 10 / (ce[0].elapsed_time(ce[1]) * 1e-3) / 1e9
    del cbuf

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded host draws, rounded to the I/O dtype)",
        "config": {"workload": cfg.name, "B": cfg.B, "T": cfg.T, "H": cfg.H, "d": cfg.D,
                   "block": cfg.block, "decay": "per channel" if cfg.per_channel else "per head",
                   "featurisation": "fused sigmoid of a and b" if args.sigmoid else "none",
                   "recurrence": ("exact (untruncated)" if exact else
                                  "uniform window" if uniform else "jagged window"),
                   "gate_groups": groups or None,
                   "block_carriers": None if (exact or uniform or groups) else
                                     ("recomputed by the backward" if nocar else "saved by the forward"),
                   "global_batch": cfg.B, "seq_len": cfg.T,
                   "parallelism": "single GPU", "launch": launch},
        "roofline": {
            "bound": "hbm",
            "kernel": dom_kernel,
            "achieved": dom_gbs,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": dom_gbs / HBM_PEAK_GBS,
            "traffic": None if traffic is None else traffic["traffic_bytes"] / 1e9,
            "traffic_unit": "GB per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-scaled)",
            "traffic_vs_algorithmic": None if traffic is None else
                traffic["traffic_bytes"] / (bb if dominant_bwd else fb),
            # the same kernel's compute counters (rocprofv3 --pmc, recorded in
            # profiles/ for these sources): matrix-pipe busy fraction
            # (MfmaUtil), executed MFMA flops (SQ_INSTS_VALU_MFMA_MOPS_* x 512)
            # at the profiled average duration against the dense peak of their
            # dtype, VALU busy fraction and mean resident waves per CU
            "mfma_util": None if counters is None else counters.get("mfma_util"),
            "mfma_tflops_counted": None if counters is None else counters.get("mfma_tflops"),
            "mfma_frac_counted": None if counters is None else counters.get("mfma_frac"),
            "valu_busy": None if counters is None else counters.get("valu_busy"),
            "occupancy_waves_per_cu": None if counters is None else counters.get("occupancy_waves_per_cu"),
        },
        "kernels": {
            "forward": {"ms": float(fwd_ms.mean()), "ms_min": float(fwd_ms.min()),
                        "ms_median": float(np.median(fwd_ms)),
                        "algorithmic_bytes": fb, "GB/s": f_gbs, "frac_hbm": f_gbs / HBM_PEAK_GBS,
                        "mfma_tflops": mfma_rate(False, fwd_ms.mean()),
                        "tokens_per_s": tokens / (fwd_ms.mean() * 1e-3)},
            "backward": {"ms": float(bwd_ms.mean()), "ms_min": float(bwd_ms.min()),
                         "ms_median": float(np.median(bwd_ms)),
                         "algorithmic_bytes": bb, "GB/s": b_gbs, "frac_hbm": b_gbs / HBM_PEAK_GBS,
                         "mfma_tflops": mfma_rate(True, bwd_ms.mean()),
                         "tokens_per_s": tokens / (bwd_ms.mean() * 1e-3)},
            "mfma_peak_tflops": mfma_peak,
            "copy_GB/s": copy_gbs,
            "wall_s_timed": t_wall,
        },
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (oracle)")
        out["cpu_baseline"] = cpu_baseline(cfg, prob, exact=exact, uniform=uniform)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
