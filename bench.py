"""Benchmark: fwd+bwd of the segmented gated linear recurrence layer on one MI355X.

One step = chain_fwd + chain_bwd over the whole sequence of the workload
(every kernel of the hot path: prep, state scan, output walk, and the
backward's replay, scans, dq walk and dk/dv/dg walk), inputs resident in HBM.
Default workload: B=1, H=40, d=128, L=262144 in 8 nonuniform segments
(the 256K-context layer of a hidden-5120 model), bf16 I/O, fp32 state.
--workload selects the other shapes (tiny_fp32, mid_bf16, vector_gate,
scan_stress); --conv and --gdn the short convolution and the gated delta rule.

Prints one JSON line: the metric, the dominant kernel's roofline (algorithmic
bytes or flops per launch over its HIP-event time) and the oracle's CPU baseline.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16 = 2.5e15    # dense bf16 MFMA, FLOP/s
PEAK_F32_MFMA = 157.3e12  # dense fp32 matrix, FLOP/s
PEAK_HBM = 8.0e12     # HBM3E, B/s
METRIC = "fwd+bwd tokens/s per layer (H=40,d=128, 256K ctx); % bf16 MFMA peak"
MALL_FLUSH_MIB = 512  # written between timed steps of workloads whose inputs are small enough to stay cached

# interface bytes per token-head that each kernel must move (io = element bytes, D = head dim):
#   fwd_prep: k, v, g            fwd_out: q, k, v, g in; o out
#   bwd_prep: q, k, v, dO, g     bwd_dq: dO, v, k, q, g in; dq, dg out
#   bwd_dkv:  q, k, v, dO, g, dg in; dk, dv, dg out
# gb = bytes of one token-head's gate (4 scalar, 4*D per-key-channel); the
# per-key-channel backward runs dv and dk as two walks, each reading its inputs
KERNEL_BYTES = {
    "fwd_prep": lambda D, io, gb: 2 * D * io + gb,
    "fwd_out": lambda D, io, gb: 4 * D * io + gb,
    "bwd_prep": lambda D, io, gb: 4 * D * io + gb * (1 if gb == 4 else 2),
    "bwd_dq": lambda D, io, gb: 5 * D * io + 2 * gb,
    "bwd_dkv": lambda D, io, gb: 6 * D * io + 3 * gb if gb == 4 else 9 * D * io + 4 * gb,
}
RECURRENCE_KERNELS = ["fwd_prep", "scan", "fwd_out", "bwd_prep", "bwd_dq", "bwd_dkv"]


def alg_flops_per_token_head(D, C=64):
    """Causal-tile algorithmic flops of one fwd+bwd per token and head (2 per
    multiply-add, causal score tiles at their triangular size): fwd
    (C+1)(2D) + 4 D^2; bwd incl. the state replay (C+1)(5D) + 10 D^2."""
    return (C + 1) * 2 * D + 4 * D * D + (C + 1) * 5 * D + 10 * D * D


def alg_bytes_per_token_head(D, io, gb=4):
    """Every interface tensor touched once: fwd q,k,v in, o out, g in;
    bwd q,k,v,dO,g in, dq,dk,dv,dg out."""
    return (4 * D * io + gb) + (7 * D * io + 2 * gb)


def _src_hash(files):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2608_06838_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def kernel_src_hash():
    return _src_hash(("sf_kernels.hip", "sf_chunk.hpp", "sf_device.hpp"))


def vg_src_hash():
    return _src_hash(("sf_kernels_vg.hip", "sf_chunk.hpp", "sf_device.hpp"))


def conv_src_hash():
    return _src_hash(("sf_conv.hip", "sf_device.hpp"))


def gdn_src_hash():
    return _src_hash(("sf_gdn.hip", "sf_device.hpp"))


def read_traffic(kernel, workload, src_hash):
    """HBM bytes per launch for `kernel` from the committed rocprofv3 counter
    summary, or None when absent or taken on a different kernel source."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for ln in f:
            if "=" in ln and not ln.startswith("#"):
                a, b = ln.split("=", 1)
                kv[a.strip()] = b.strip()
    if kv.get("src_sha") != src_hash:
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(w, inp, budget_s=15.0):
    """Time the fp64 oracle (fwd + bwd) on the host cores on a bounded sample of
    the same workload: the first n_h heads of batch 0 over the first L_s tokens."""
    import oracle

    cores = len(os.sched_getaffinity(0))
    nh = min(w["H"], cores)
    L = sum(w["seg_lens"])

    def sample(L_s):
        sl = {k: inp[k][:1, :L_s, :nh] for k in ("q", "k", "v", "g", "dO")}
        return {k: v.detach().cpu().double().numpy() for k, v in sl.items()}

    def run(s):
        t0 = time.perf_counter()
        oracle.forward(s["q"], s["k"], s["v"], s["g"], None, threads=nh)
        oracle.backward(s["q"], s["k"], s["v"], s["g"], None, s["dO"], None, threads=nh)
        return time.perf_counter() - t0

    L0 = min(L, 1024)
    t_cal = run(sample(L0))
    L_s = int(min(L, max(L0, (budget_s / max(t_cal, 1e-6)) * L0)) // 64 * 64)
    s = sample(L_s)
    t = run(s)
    value = nh * L_s / w["H"] / t  # layer tokens/s: a layer token is H token-heads
    return {"value": value, "unit": "tokens/s", "cores": nh, "kind": "oracle",
            "sample": f"batch 0, heads 0..{nh - 1}, first {L_s} tokens, fwd+bwd fp64, "
                      f"{t:.1f} s wall; value scaled to a {w['H']}-head layer"}


class Flusher:
    """Writes a buffer larger than the 256 MB Infinity Cache (MALL) between
    timed steps, so that a small workload's inputs are read from HBM."""

    def __init__(self, torch, dev, mib):
        self.buf = torch.empty(mib * (1 << 20) // 4, dtype=torch.float32, device=dev) if mib > 0 else None

    def __call__(self):
        if self.buf is not None:
            self.buf.fill_(1.0)


def timed_steps(torch, step, steps, flush):
    """ms per step over `steps` calls of step().  Without a flush: host clock
    across all steps, bracketed by device synchronisations.  With one: each
    step is bracketed by synchronisations and the flush runs outside them."""
    if flush.buf is None:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            step()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3 / steps
    tot = 0.0
    for _ in range(steps):
        flush()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        step()
        torch.cuda.synchronize()
        tot += time.perf_counter() - t0
    return tot * 1e3 / steps


def copy_calibration(torch, dev, mib):
    """One plain device copy of known size (FETCH_SIZE / WRITE_SIZE
    calibration under rocprofv3 --pmc)."""
    if mib <= 0:
        return
    src = torch.ones(mib * (1 << 20) // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


CONV_METRIC = "short-conv fwd+bwd tokens/s (C=15360=3x40x128, W=4, SiLU, 256K ctx, 8 segments, carried tails)"
# interface bytes per token and channel: forward x in, y out; backward x, dy in, dx out
CONV_BYTES = {"conv_fwd": lambda io: 2 * io, "conv_bwd": lambda io: 3 * io}


def conv_cpu_baseline(inp, w, act, budget_s=15.0):
    """The fp64 oracle of the short convolution (numpy, one process) over the
    whole sequence of batch 0 on its first nc channels, nc chosen for about
    budget_s of CPU work, scaled to the workload's channel count."""
    import oracle

    L = sum(w["seg_lens"])

    def sample(nc):
        return {k: (v[:1, :, :nc] if v.dim() == 3 else v[:nc]).detach().cpu().double().numpy()
                for k, v in inp.items() if v is not None}

    def run(s):
        t0 = time.perf_counter()
        oracle.conv_forward(s["x"], s["w"], s["tail_in"], act=act)
        oracle.conv_backward(s["x"], s["w"], s["tail_in"], s["dy"], s["dtail_out"], act=act)
        return time.perf_counter() - t0

    nc0 = 64
    t_cal = run(sample(nc0))
    nc = int(min(w["C"], max(nc0, budget_s / max(t_cal, 1e-6) * nc0)) // 8 * 8)
    t = run(sample(nc))
    value = L * nc / w["C"] / t
    return {"value": value, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": f"batch 0, all {L} tokens, channels 0..{nc - 1}, fwd+bwd fp64 numpy, {t:.1f} s wall; "
                      f"value scaled to {w['C']} channels"}


def bench_conv(args):
    """One step = the short convolution forward over the 8 segments (tails
    carried), then its backward over the segments in reverse order (tail
    gradients carried), inputs resident in HBM, outputs preallocated."""
    import torch
    import paper_2608_06838_amd as sf
    from paper_2608_06838_amd import synth

    w = synth.conv_workload("conv_ctx256k")
    B, C, W, seg, act = w["B"], w["C"], w["W"], w["seg_lens"], w["act"]
    L = sum(seg)
    dev = torch.device("cuda:0")
    inp = synth.make_conv_inputs(B, L, C, W, io=w["io"], device=dev, seed=2002)
    x, wt, dy = inp["x"], inp["w"], inp["dy"]
    io = x.element_size()
    y, dx = torch.empty_like(x), torch.empty_like(x)
    tails = torch.empty((len(seg) + 1, B, W - 1, C), dtype=torch.float32, device=dev)
    tails[0].copy_(inp["tail_in"])
    dtails = torch.empty_like(tails)
    dtails[-1].copy_(inp["dtail_out"])
    dws = torch.empty((len(seg), C, W), dtype=torch.float32, device=dev)
    nws = max(sf.conv_bwd_workspace_bytes(x[:, :n], wt, act) for n in seg)
    ws = torch.empty(nws, dtype=torch.uint8, device=dev)
    starts = [sum(seg[:i]) for i in range(len(seg))]
    kernels = ["conv_fwd", "conv_bwd"]
    timer = sf.KernelTimer(capacity=64 * max(1, args.steps))

    def step(tm=None):
        for i, (t, n) in enumerate(zip(starts, seg)):
            sf.conv_fwd(x[:, t:t + n], wt, tails[i], act, out=(y[:, t:t + n], tails[i + 1]), timing=tm)
        for i in reversed(range(len(seg))):
            t, n = starts[i], seg[i]
            sf.conv_bwd(x[:, t:t + n], wt, tails[i], dy[:, t:t + n], dtails[i + 1], act,
                        out=(dx[:, t:t + n], dws[i], dtails[i], ws), timing=tm)

    for i in range(args.warmup):
        if i == args.warmup - 1:
            torch.cuda.synchronize()
            timer.select(kernels)
            step(timer)
        else:
            step()
    torch.cuda.synchronize()
    wtime = timer.read()
    dom = max(kernels, key=lambda k: wtime.get(k, (0.0, 0))[0]) if wtime else "conv_bwd"
    timer.select([dom])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(timer)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    tot_ms, nl = timer.read()[dom]
    ms = (t1 - t0) * 1e3 / args.steps
    copy_calibration(torch, dev, args.copy_mib)
    avg_s = tot_ms / 1e3 / max(nl, 1)
    bytes_per_launch = CONV_BYTES[dom](io) * B * L * C * args.steps / max(nl, 1)
    achieved = bytes_per_launch / avg_s / 1e9
    if args.kernel_times:
        for k in kernels:
            t, n = wtime.get(k, (0.0, 0))
            print(f"# {k:9s} {t:8.3f} ms/step  {n:4d} launches/step", file=sys.stderr)
    out = {
        "metric": CONV_METRIC, "value": B * L / (ms / 1e3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16" if io == 2 else "f32", "data": "synthetic",
        "config": {"workload": w["name"], "B": B, "C": C, "W": W, "L": L, "segments": seg, "act": act,
                   "io": w["io"]},
        "hbm_frac_alg": sum(f(io) for f in CONV_BYTES.values()) * B * L * C / (ms / 1e3) / PEAK_HBM,
        "roofline": {"kernel": dom, "bound": "hbm", "achieved": achieved, "peak": PEAK_HBM / 1e9, "unit": "GB/s",
                     "frac": achieved * 1e9 / PEAK_HBM, "traffic": read_traffic(dom, "conv_ctx256k", conv_src_hash()),
                     "launches": nl, "avg_launch_us": avg_s * 1e6},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = conv_cpu_baseline(inp, w, act)
    print(json.dumps(out), flush=True)
    timer.close()


def make_chain_step(sf, torch, inp, seg, ts, overlap, keep=False):
    """fwd+bwd chain over segments `seg` with preallocated outputs and
    workspaces (the step allocates nothing).  step(timer) times the launches
    of the kernels the timer selects.  keep: the forward keeps its superchunk
    states and the backward reads them (else the backward replays them)."""
    dev = inp["q"].device
    B, L, H, D = inp["q"].shape
    o = torch.empty_like(inp["q"])
    S_bnd = torch.empty((len(seg) + 1, B, H, D, D), dtype=torch.float32, device=dev)
    nws = sf.chain_workspace_bytes(inp["q"], inp["g"], seg, ts=ts)
    ws_f = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
    ws_b = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
    dq, dk, dv = (torch.empty_like(inp["q"]) for _ in range(3))
    dg = torch.empty_like(inp["g"])
    dS0 = torch.empty((B, H, D, D), dtype=torch.float32, device=dev)
    nck = sf.chain_ckpt_bytes(inp["q"], inp["g"], seg, ts=ts, overlap=overlap)
    ck = torch.empty(max(nck, 1), dtype=torch.uint8, device=dev)

    def step(tm=None, overlap=overlap, keep=keep):
        sf.chain_fwd(inp["q"], inp["k"], inp["v"], inp["g"], seg, inp["S_in"], ts=ts, overlap=overlap,
                     out=(o, S_bnd, ws_f, ck), timing=tm, keep_states=keep)
        sf.chain_bwd(inp["q"], inp["k"], inp["v"], inp["g"], seg, S_bnd, inp["dO"], inp["dS_out"],
                     ts=ts, overlap=overlap, out=(dq, dk, dv, dg, dS0, ws_b), timing=tm, ckpt=ck if keep else None)
    step.ckpt_bytes = nck
    return step


def time_steps(torch, step, warmup, steps):
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / steps


# Hybrid cost model of the partition study (the paper gives the form of the
# per-segment cost, not its coefficients).  A 15B-class period-4 hybrid stack,
# hidden d = 5120: per 4 layers, 3 linear-recurrence layers and 1 softmax layer,
# each with q/k/v/o projections (8 d^2 FLOPs per token) and an MLP of width 4d
# (16 d^2); softmax attention costs 4 d FLOPs per query-key pair (QK^T and AV).
HYBRID_D = 5120
HYBRID_W_TOK = 3 * 8 * HYBRID_D ** 2 + 4 * 16 * HYBRID_D ** 2 + 8 * HYBRID_D ** 2
HYBRID_W_SOFT = 4 * HYBRID_D


def study_main(args):
    """--tune-ts / --partition-study: time the recurrence layer's fwd+bwd chain
    per candidate and print one JSON line with the table (Sec. 3.2 / 3.4
    selection by profiling)."""
    import torch
    import paper_2608_06838_amd as sf
    from paper_2608_06838_amd import synth, tune

    w = synth.workload(args.workload)
    dev = torch.device("cuda:0")
    inp = synth.make_inputs(w, device=dev, seed=1002)
    T = inp["q"].shape[1]
    if args.tune_ts:
        cands = [(ts, ov) for ts in tune.ts_candidates(w["seg_lens"]) for ov in (1, 0, 2)]

        def time_fn(c):
            return time_steps(torch, make_chain_step(sf, torch, inp, w["seg_lens"], c[0], c[1]), 1, args.steps)

        best, table = tune.search(cands, time_fn)
        sp = tune.speedups(table, (0, 1))
        rows = [dict(ts=r["candidate"][0] or "auto", overlap=r["candidate"][1], ms=r["ms"], status=r["status"],
                     speedup_vs_auto_overlap=x) for r, x in zip(table, sp)]
        out = dict(study="superchunk stride and scan overlap", workload=w["name"], steps=args.steps, table=rows,
                   best=dict(ts=best[0] or "auto", overlap=best[1]) if best else None)
    else:
        cands = tune.partition_candidates(T, HYBRID_W_TOK, HYBRID_W_SOFT)

        def time_fn(c):
            return time_steps(torch, make_chain_step(sf, torch, inp, c[2], 0, True), 1, args.steps)

        best, table = tune.search(cands, time_fn)
        sp = tune.speedups(table, next((c for c in cands if c[0] == 8 and c[1] == 0.0), None))
        rows = []
        for r, x in zip(table, sp):
            N, a, lens = r["candidate"]
            bnd = [0]
            for n in lens:
                bnd.append(bnd[-1] + n)
            costs = [HYBRID_W_TOK * (b1 - b0) + HYBRID_W_SOFT * (b0 * (b1 - b0) + 0.5 * (b1 - b0) ** 2)
                     for b0, b1 in zip(bnd[:-1], bnd[1:])]
            rows.append(dict(N=N, alpha=a, seg_lens=lens, recurrence_ms=r["ms"], status=r["status"],
                             speedup_vs_equal8=x, hybrid_cost_max_over_mean=max(costs) / (sum(costs) / len(costs))))
        out = dict(study="hybrid-aware partition (recurrence layer timed; hybrid cost modelled)",
                   workload=w["name"], steps=args.steps,
                   cost_model=dict(w_tok=HYBRID_W_TOK, w_soft=HYBRID_W_SOFT, note="period-4 hybrid, hidden 5120"),
                   table=rows, best_for_the_recurrence=dict(N=best[0], alpha=best[1]) if best else None)
    print(json.dumps(out), flush=True)


GDN_METRIC = "gated-delta-rule training-step (fwd+bwd) tokens/s per layer (H=40, d=128, 256K ctx, 8 segments chained through S)"
GDN_KERNELS = ["gdn_prep", "gdn_scan", "gdn_out", "gdn_store", "gdn_dprep", "gdn_dscan", "gdn_dwalk", "gdn_dchunk"]


def gdn_dchunk_flops(D, C=64):
    """Algorithmic flops per 64-token chunk and head of the delta rule's
    per-chunk parameter gradients, given the state S entering the chunk and
    the gradient dS' of the state leaving it (2 m n k per product, triangular
    factors at their triangular size):
      five C x D x D products (K S, K dS', G_U S^T, dO S^T, U dS'^T): 10 C D^2;
      lower-triangular-with-diagonal C x C products (Q K^T, T R, P^T dO, T^T dU,
      dO U^T, (dP o Gamma) K, (dP o Gamma)^T Q): 7 C (C + 1) D;
      strictly lower ones (K K^T, G_U U^T, Ah K, Ah^T K): 4 C (C - 1) D;
      the triangular inverse: C^3 / 3."""
    return 10 * C * D * D + 7 * C * (C + 1) * D + 4 * C * (C - 1) * D + C ** 3 // 3


def bench_gdn(args):
    """One step = the gated-delta-rule forward over the 8 segments of the
    256K-context layer, the state carried from segment to segment, then the
    backward over the segments in reverse, the state gradient carried back
    (random bf16 dO, no loss term on the final state), through the chain entry
    points (state scans overlapped on a second stream unless --gdn-serial)."""
    import torch
    import paper_2608_06838_amd as sf
    from paper_2608_06838_amd import synth

    w = synth.workload("ctx256k_h40")
    seg = w["seg_lens"]
    B, H, D, L = w["B"], w["H"], w["D"], sum(seg)
    dev = torch.device("cuda:0")
    inp = synth.make_gdn_inputs(B, L, H, D, device=dev, seed=4002)
    gen = torch.Generator(device=dev).manual_seed(4003)
    dO = torch.randn((B, L, H, D), device=dev, generator=gen).to(torch.bfloat16)
    x = (inp["q"], inp["k"], inp["v"], inp["g"], inp["beta"], seg)
    ov = not args.gdn_serial
    timer = sf.KernelTimer(capacity=256 * max(1, args.steps))

    keep = args.keep_states

    def step(tm=None, keep=keep):
        out = sf.gdn_chain_fwd(*x, inp["S_in"], ts=args.gdn_ts, overlap=ov, timing=tm, keep_states=keep)
        sf.gdn_chain_bwd(*x, out[1], dO, None, ts=args.gdn_ts, overlap=ov, timing=tm,
                         ckpt=out[2] if keep else None)

    for i in range(args.warmup):
        if i == args.warmup - 1:
            torch.cuda.synchronize()
            timer.select(GDN_KERNELS)
            step(timer)
        else:
            step()
    torch.cuda.synchronize()
    wtime = timer.read()
    dom = max(GDN_KERNELS, key=lambda k: wtime.get(k, (0.0, 0))[0]) if wtime else "gdn_dchunk"
    timer.select([dom])
    torch.cuda.reset_peak_memory_stats()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(timer)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    peak = torch.cuda.max_memory_allocated()
    tot_ms, nl = timer.read()[dom]
    ms = (t1 - t0) * 1e3 / args.steps
    # the same step with the backward reading the superchunk states and maps the
    # forward kept (or replaying them, under --keep-states)
    kept = {"kept": keep, "bytes": sf.gdn_chain_ckpt_bytes(inp["q"], inp["g"], seg, ts=args.gdn_ts, overlap=ov)}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(keep=not keep)
    torch.cuda.synchronize()
    kept["t_recompute_ms" if keep else "t_kept_ms"] = (time.perf_counter() - t0) * 1e3 / args.steps
    copy_calibration(torch, dev, args.copy_mib)
    avg_s = tot_ms / 1e3 / max(nl, 1)
    if dom == "gdn_dchunk":
        flops = gdn_dchunk_flops(D) * B * H * (L // 64) * args.steps / max(nl, 1)
        roof = {"kernel": dom, "bound": "mfma", "achieved": flops / avg_s / 1e12, "peak": PEAK_BF16 / 1e12,
                "unit": "TFLOP/s", "frac": flops / avg_s / PEAK_BF16}
    else:
        roof = {"kernel": dom, "bound": "mfma", "achieved": None, "peak": PEAK_BF16 / 1e12, "unit": "TFLOP/s",
                "frac": None}
    roof.update(traffic=read_traffic(dom, "gdn_ctx256k_h40", gdn_src_hash()), launches=nl,
                avg_launch_us=avg_s * 1e6)
    if args.kernel_times:
        for k in GDN_KERNELS:
            t, n = wtime.get(k, (0.0, 0))
            print(f"# {k:10s} {t:8.3f} ms/step  {n:4d} launches/step", file=sys.stderr)
    out = {
        "metric": GDN_METRIC, "value": B * L / (ms / 1e3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "gdn_ctx256k_h40", "B": B, "H": H, "Dk": D, "Dv": D, "L": L, "segments": seg,
                   "ts": args.gdn_ts or "auto", "overlap": ov,
                   "parallelism": "superchunks: [M|N] prep walk, fp32 state scan, output walk; backward: "
                                  "state-gradient walk over superchunks, per-chunk gradients over all chunks"},
        "kernels_ms_per_step": {k: wtime.get(k, (0.0, 0))[0] for k in GDN_KERNELS},
        "peak_mem_bytes": peak,
        "roofline": roof,
        "superchunk_states": kept,
    }
    if not args.no_cpu_baseline:
        from oracle import gdn as ogdn
        nh = min(H, len(os.sched_getaffinity(0)))
        L_s = 1024
        cs = {k: inp[k][:1, :L_s, :nh].detach().cpu().double().numpy() for k in ("q", "k", "v", "g", "beta")}
        do = dO[:1, :L_s, :nh].detach().cpu().double().numpy()
        tc = time.perf_counter()
        ogdn.forward(cs["q"], cs["k"], cs["v"], cs["g"], cs["beta"], None, threads=nh)
        ogdn.backward(cs["q"], cs["k"], cs["v"], cs["g"], cs["beta"], None, do, None, threads=nh)
        tc = time.perf_counter() - tc
        out["cpu_baseline"] = {"value": nh * L_s / H / tc, "unit": "tokens/s", "cores": nh, "kind": "oracle",
                               "sample": f"batch 0, heads 0..{nh - 1}, first {L_s} tokens, fwd + bwd fp64, "
                                         f"{tc:.1f} s wall; value scaled to a {H}-head layer"}
    print(json.dumps(out), flush=True)
    timer.close()


TABLE4_HEADS = (20, 10, 8)           # heads per GPU of the paper's 3B / 15B / 32B GDN models
TABLE4_LENS = (8192, 16384, 32768, 65536)
TABLE4_SPLITS = (None, 0.3, 0.5, 0.7, 0.9)  # split fraction f of the call (None: one segment)


def _split(L, f):
    if f is None:
        return [L]
    a = int(round(f * L / 64)) * 64
    return [a, L - a] if 0 < a < L else [L]


def table4_main(args):
    """Table-4(a)-style study (Sec. 3.4 "State Transition Grid Optimization"
    and "Split and Overlap", Table 4(a)): for each operator call of L tokens
    at the per-GPU head counts of the paper's models, time the forward and the
    backward separately for every superchunk length and split fraction f (the
    call run as two chained segments f L and (1 - f) L with the state scans
    overlapped, the paper's split schedule), and report the default and the
    fastest setting per pass."""
    import torch
    import paper_2608_06838_amd as sf
    from paper_2608_06838_amd import synth, tune

    dev = torch.device("cuda:0")
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    ops = [args.table4] if args.table4 in ("gla", "gdn") else ["gla", "gdn"]
    rows = []
    for op in ops:
        for H in TABLE4_HEADS:
            for L in TABLE4_LENS:
                if op == "gla":
                    w = synth.workload("ctx256k_h40", H=H, seg_lens=[L])
                    inp = synth.make_inputs(w, device=dev, seed=1100 + H)
                    tss = [0, 256, 512, 1024, 2048, 4096]
                else:
                    inp = synth.make_gdn_inputs(1, L, H, 128, device=dev, seed=4100 + H)
                    gen = torch.Generator(device=dev).manual_seed(4200 + H)
                    inp["dO"] = torch.randn((1, L, H, 128), device=dev, generator=gen).to(torch.bfloat16)
                    tss = [0, 1024, 2048, 4096, 8192]
                res = []
                for f in TABLE4_SPLITS:
                    seg = _split(L, f)
                    if f is not None and len(seg) == 1:
                        continue
                    for ts in tss:
                        if ts and ts > max(seg):
                            continue
                        ov = f is not None

                        def call():
                            if op == "gla":
                                o, S_bnd = sf.chain_fwd(inp["q"], inp["k"], inp["v"], inp["g"], seg, inp["S_in"],
                                                        ts=ts, overlap=ov)
                                ev[1].record()
                                sf.chain_bwd(inp["q"], inp["k"], inp["v"], inp["g"], seg, S_bnd, inp["dO"], None,
                                             ts=ts, overlap=ov)
                            else:
                                x = (inp["q"], inp["k"], inp["v"], inp["g"], inp["beta"], seg)
                                o, S_bnd = sf.gdn_chain_fwd(*x, inp["S_in"], ts=ts, overlap=ov)
                                ev[1].record()
                                sf.gdn_chain_bwd(*x, S_bnd, inp["dO"], None, ts=ts, overlap=ov)

                        try:
                            call()
                            torch.cuda.synchronize()
                            tf = tb = 0.0
                            for _ in range(args.steps):
                                ev[0].record()
                                call()
                                ev[2].record()
                                torch.cuda.synchronize()
                                tf += ev[0].elapsed_time(ev[1])
                                tb += ev[1].elapsed_time(ev[2])
                            res.append(dict(ts=ts or "auto", f=f, fwd_ms=tf / args.steps, bwd_ms=tb / args.steps))
                        except Exception as e:  # a candidate that does not run is reported
                            res.append(dict(ts=ts or "auto", f=f, error=str(e)[:200]))
                ok = [r for r in res if "error" not in r]
                base = next(r for r in ok if r["ts"] == "auto" and r["f"] is None)
                bf = min(ok, key=lambda r: r["fwd_ms"])
                bb = min(ok, key=lambda r: r["bwd_ms"])
                rows.append(dict(op=op, heads=H, L=L, default=dict(fwd_ms=base["fwd_ms"], bwd_ms=base["bwd_ms"]),
                                 best_fwd=dict(ts=bf["ts"], f=bf["f"], ms=bf["fwd_ms"],
                                               speedup=base["fwd_ms"] / bf["fwd_ms"]),
                                 best_bwd=dict(ts=bb["ts"], f=bb["f"], ms=bb["bwd_ms"],
                                               speedup=base["bwd_ms"] / bb["bwd_ms"]),
                                 total_speedup=(base["fwd_ms"] + base["bwd_ms"]) / (bf["fwd_ms"] + bb["bwd_ms"]),
                                 candidates=res))
                print(json.dumps({k: v for k, v in rows[-1].items() if k != "candidates"}), file=sys.stderr, flush=True)
                del inp
                torch.cuda.empty_cache()
    print(json.dumps(dict(study="Table 4(a)-style: superchunk length x split fraction, fwd and bwd per call",
                          steps=args.steps, rows=rows)), flush=True)


def bench_recurrence(args):
    import torch
    import paper_2608_06838_amd as sf
    from paper_2608_06838_amd import synth, tuned

    w = synth.workload(args.workload)
    w["L"] = sum(w["seg_lens"])
    dev = torch.device("cuda:0")
    inp = synth.make_inputs(w, device=dev, seed=1002)
    B, L, H, D = inp["q"].shape
    io = inp["q"].element_size()
    gb = 4 * (D if inp["g"].dim() == 4 else 1)
    seg = w["seg_lens"]
    pick = tuned.choice(w["name"])  # the profiled per-shape setting (ts, overlap)
    ts = args.ts if args.ts is not None else pick["ts"]
    if args.no_overlap or args.overlap or args.overlap_prep:
        overlap = 0 if args.no_overlap else (2 if args.overlap_prep else 1)
    else:
        overlap = pick["overlap"]
    # inputs below ~2 GiB could sit partly in the 256 MB MALL between steps
    in_bytes = sum(inp[k].numel() * inp[k].element_size() for k in ("q", "k", "v", "g", "dO"))
    flush = Flusher(torch, dev, MALL_FLUSH_MIB if in_bytes < (2 << 30) else 0)
    keep = args.keep_states
    step = make_chain_step(sf, torch, inp, seg, ts, overlap, keep=keep)
    timer = sf.KernelTimer(capacity=max(512, 8 * len(seg) * (args.steps + 1)))

    # The last warmup step carries HIP events on every kernel launch: per-kernel
    # times for the report and the choice of the dominant kernel.  The timed
    # steps then carry events on the dominant kernel's launches only.
    for i in range(args.warmup):
        flush()
        if i == args.warmup - 1:
            torch.cuda.synchronize()
            timer.select(RECURRENCE_KERNELS)
            step(timer)
        else:
            step()
    torch.cuda.synchronize()
    kstep = timer.read()
    dom = max(KERNEL_BYTES, key=lambda k: kstep.get(k, (0.0, 0))[0]) if kstep else "bwd_dkv"
    timer.select([dom])
    torch.cuda.reset_peak_memory_stats()
    ms = timed_steps(torch, lambda: step(timer), args.steps, flush)
    peak = torch.cuda.max_memory_allocated()
    tot_ms, nlaunch = timer.read()[dom]
    if not kstep:  # no warmup: per-kernel times from one more step
        timer.select(RECURRENCE_KERNELS)
        step(timer)
        kstep = timer.read()

    # Split-and-overlap figures (Sec. 3.4): the same step with the scans
    # serialised on the main stream, the scans' own time there, and with them
    # overlapped on the aux stream (the scans alone, then each segment's
    # preparation kernel with its scan).
    ov = {"default_overlap": overlap}
    if not args.no_overlap_study:
        timer.select(["scan"])
        t_serial = timed_steps(torch, lambda: step(timer, overlap=False), args.steps, flush)
        t_scan = timer.read().get("scan", (0.0, 0))[0] / args.steps
        t_over = timed_steps(torch, lambda: step(None, overlap=1), args.steps, flush)
        t_over2 = timed_steps(torch, lambda: step(None, overlap=2), args.steps, flush)
        t_intra = t_serial - t_scan
        ov.update(t_e2e_ms=ms, t_overlapped_ms=t_over, t_overlapped_prep_ms=t_over2, t_serial_ms=t_serial,
                  t_scan_serial_ms=t_scan,
                  t_intra_only_ms=t_intra, e2e_over_intra_only=ms / t_intra if t_intra > 0 else None,
                  hidden_frac_of_scan=(t_serial - t_over) / t_scan if t_scan > 0 else None)
    # The superchunk states: replayed by the backward (the default: the paper's
    # full recomputation, every row of the path in the timed step), or kept by
    # the forward for the backward (the same step without the replay).
    kept = {"kept": keep, "bytes": step.ckpt_bytes}
    if not args.no_overlap_study:
        kept["t_recompute_ms" if keep else "t_kept_ms"] = timed_steps(torch, lambda: step(None, keep=not keep),
                                                                      args.steps, flush)
    copy_calibration(torch, dev, args.copy_mib)

    value = B * L / (ms / 1e3)
    avg_s = tot_ms / 1e3 / max(nlaunch, 1)
    bytes_per_launch = KERNEL_BYTES[dom](D, io, gb) * B * H * L * args.steps / max(nlaunch, 1)
    achieved = bytes_per_launch / avg_s / 1e9
    vec = gb > 4
    traffic = read_traffic(dom, w["name"], vg_src_hash() if vec else kernel_src_hash())
    flops = alg_flops_per_token_head(D) * B * H * L
    peak_mfma = PEAK_BF16 if io == 2 else PEAK_F32_MFMA
    if args.kernel_times:
        for k in RECURRENCE_KERNELS:
            msk, n = kstep.get(k, (0.0, 0))
            print(f"# {k:9s} {msk:8.3f} ms/step  {n:4d} launches/step", file=sys.stderr)
    out = {
        "metric": METRIC, "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16" if io == 2 else "f32", "data": "synthetic",
        "config": {"workload": w["name"], "B": B, "H": H, "Dk": D, "Dv": D, "L": L, "segments": seg,
                   "gate": "per-key-channel" if vec else "scalar",
                   "chunk": 64, "io": "bf16" if io == 2 else "f32", "state": "f32",
                   "overlap": overlap, "ts": ts or "auto", "mall_flush_mib": MALL_FLUSH_MIB if flush.buf is not None
                   else 0},
        "mfma_frac_of_peak": flops / (ms / 1e3) / peak_mfma,
        "mfma_peak": "bf16 2.5 PFLOP/s" if io == 2 else "fp32 matrix 157.3 TFLOP/s",
        "hbm_frac_alg": alg_bytes_per_token_head(D, io, gb) * B * H * L / (ms / 1e3) / PEAK_HBM,
        "kernels_ms_per_step": {k: kstep.get(k, (0.0, 0))[0] for k in RECURRENCE_KERNELS},
        "peak_mem_bytes": peak,
        "roofline": {"kernel": dom, "bound": "hbm", "achieved": achieved, "peak": PEAK_HBM / 1e9,
                     "unit": "GB/s", "frac": achieved * 1e9 / PEAK_HBM, "traffic": traffic,
                     "launches": nlaunch, "avg_launch_us": avg_s * 1e6},
        "overlap": ov,
        "superchunk_states": kept,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, inp)
    print(json.dumps(out), flush=True)
    timer.close()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="ctx256k_h40",
                    help="ctx256k_h40 (default), mid_bf16, tiny_fp32, vector_gate or scan_stress")
    ap.add_argument("--ts", type=int, default=None, help="superchunk length (0: automatic; default: the tuned one)")
    ap.add_argument("--no-overlap", action="store_true", help="scans serialised on the main stream")
    ap.add_argument("--overlap", action="store_true", help="scans overlapped on the aux stream")
    ap.add_argument("--overlap-prep", action="store_true",
                    help="each segment's preparation kernel and scan on the aux stream")
    ap.add_argument("--no-overlap-study", action="store_true",
                    help="skip the serial / overlapped comparison after the timed steps")
    ap.add_argument("--keep-states", action="store_true",
                    help="time the step whose backward reads the superchunk states the forward kept, instead of "
                         "replaying them (the paper's full recomputation, the default)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--kernel-times", action="store_true", help="print per-kernel times to stderr")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after timing, run one plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--conv", action="store_true",
                    help="measure the short convolution with carried tails instead of the recurrence")
    ap.add_argument("--gdn", action="store_true", help="measure the gated-delta-rule training step instead")
    ap.add_argument("--gdn-ts", type=int, default=0, help="gated delta rule superchunk length (0: automatic)")
    ap.add_argument("--gdn-serial", action="store_true", help="gated delta rule: state scans on the main stream")
    ap.add_argument("--tune-ts", action="store_true",
                    help="time the chain for each superchunk stride and overlap setting (one JSON table)")
    ap.add_argument("--partition-study", action="store_true",
                    help="time the chain for the hybrid-aware partition candidates (one JSON table)")
    ap.add_argument("--table4", default=None, choices=("gla", "gdn", "both"),
                    help="per-call study over heads 20/10/8 and 8K-64K tokens: superchunk length x split fraction")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); across GPUs the recurrence would "
              "shard over heads (no exchange) or over sequence segments (boundary states passed on)",
              file=sys.stderr)
        sys.exit(2)
    if args.conv:
        bench_conv(args)
    elif args.gdn:
        bench_gdn(args)
    elif args.tune_ts or args.partition_study:
        study_main(args)
    elif args.table4:
        table4_main(args)
    else:
        bench_recurrence(args)


if __name__ == "__main__":
    main()
