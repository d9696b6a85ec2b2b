"""Benchmark: one V-MoE layer forward + backward on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
                    [--flush-mall] [--no-diagnostics] [--copy-probe]

A step is one pass of the whole layer: routing (router product, noisy top-k,
batch-prioritized capacity), dispatch, expert MLP forward, combine, and the
backward of all of them, on synthetic ViT-shaped tokens already resident in
HBM. The default workload is the largest: ViT-L/16 at 384 px, 64 images x 577
tokens, d_model 1024, d_ff 4096, 32 experts (four hot), top-2, capacity
factor 1.05. W untimed warm-up steps, then K timed steps between device
synchronisations. Prints ONE JSON line.

Inside the timed steps only the dominant call, the expert-MLP backward, is
bracketed by HIP events on the stream it runs on, so its roofline is
measured live over the timed steps while the step time carries no other
instrumentation. A second pass of K steps after the timed region brackets
every C-ABI call with events for the per-call breakdown.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "V-MoE layer fwd+bwd tokens/s on 1 MI355X; % bf16 MFMA peak; route GB/s"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 matrix peak
PEAK_F32_TFLOPS = 157.3        # MI355X f32 matrix peak
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E

# The step's C-ABI calls in order; the dispatch and router backward run as
# one call (vmoe_dispatch_route_bwd, bit-identical to the two separate calls).
CALLS = ["route", "dispatch", "ffn_fwd", "combine_fwd", "combine_bwd", "ffn_bwd",
         "dispatch_route_bwd"]


def algorithmic_cost(cfg, A: int, n_noise: bool, n_bias: bool, NK: int = -1):
    """Per-call algorithmic (flops, bytes): only what the definition must touch.

    A = kept assignments, NK = tokens that keep at least one (their rows of
    x and dy are the only ones dispatch and combine backward need; default
    every token). Bytes count each tensor once at its storage width;
    workspace, sort passes and re-reads are overhead, not algorithmic.
    """
    N, d, f, E, k, G = cfg.n_tokens, cfg.d_model, cfg.d_ff, cfg.n_experts, cfg.k, cfg.n_groups
    B = 2 if cfg.dtype == "bf16" else 4
    NK = N if NK < 0 else NK
    meta = N * k * 4 * 2 + G * E * 4  # idx + slot, row_base
    c = {}
    c["route"] = (2 * N * d * E, N * d * B + G * E * d * B + N * E * 4 * (2 + (1 if n_noise else 0))
                  + N * k * 12 + N * 4 + G * E * 8)
    c["dispatch"] = (0, NK * d * B + A * d * B + meta)
    c["ffn_fwd"] = (4 * A * d * f, 2 * E * d * f * B + E * (d + f) * B + A * d * B + 2 * A * f * B
                    + A * d * B)
    c["combine_fwd"] = (2 * A * d, A * d * B + N * d * B + meta + N * k * 4)
    c["combine_bwd"] = (2 * A * d, NK * d * B + 2 * A * d * B + meta + N * k * 8)
    c["ffn_bwd"] = (8 * A * d * f, 2 * E * d * f * B + A * d * B + 2 * A * f * B + A * d * B
                    + A * f * B + A * d * B + E * (2 * d * f + d + f) * 4)
    c["dispatch_bwd"] = (0, A * d * B + N * d * 4 + meta)
    c["route_bwd"] = (4 * N * d * E, N * d * B + 2 * N * d * 4 + N * E * 4 + N * k * 12
                      + G * E * d * (B + 4))
    # dxe rows in, dx out once, x, probs, routing data, router and its gradient
    c["dispatch_route_bwd"] = (4 * N * d * E, A * d * B + N * d * B + N * d * 4 + N * E * 4
                               + N * k * 12 + G * E * 4 + G * E * d * (B + 4))
    return c


TRAFFIC_PROFILE = {"vitb16_bf16": "profiles/vitb16_bf16_hbm_traffic.txt",
                   "vitl16_384_bf16": "profiles/vitl16_384_bf16_hbm_traffic.txt"}


def source_digest(path: str) -> str:
    """sha256 of a C/HIP source with its // comments and blank lines removed,
    so that edits to comments alone keep measured counters valid."""
    import hashlib
    lines = []
    for line in open(path, encoding="utf-8"):
        code = line.split("//", 1)[0].rstrip()
        if code:
            lines.append(code)
    return hashlib.sha256("\n".join(lines).encode()).hexdigest()


def measured_traffic(workload: str, call: str):
    """HBM bytes per call from the committed rocprofv3 PMC summary.

    The summary holds calibrated FETCH_SIZE / WRITE_SIZE bytes per C-ABI call
    and the code digest (source_digest) of the sources the counters were
    taken with; a call whose code has changed since then has no measured
    traffic (None).
    """
    rel = TRAFFIC_PROFILE.get(workload)
    if rel is None or not os.path.exists(os.path.join(ROOT, rel)):
        return None
    calls, sources = {}, {}
    for line in open(os.path.join(ROOT, rel)):
        w = line.split()
        if len(w) == 6 and w[0] == "call":
            calls[w[1]] = int(w[3]) + int(w[5])
        elif len(w) == 4 and w[0] == "source":
            sources[w[1]] = w[3]
    used = {"ffn_fwd": ["ffn.hip"], "ffn_bwd": ["ffn.hip"], "route": ["route.hip"],
            "route_bwd": ["route_bwd.hip"],
            "dispatch_route_bwd": ["route_bwd.hip"]}.get(call, ["moves.hip"]) + ["common.h"]
    csrc = os.path.join(ROOT, "paper_2608_16188_amd", "csrc")
    for f in used:
        if sources.get(f) != source_digest(os.path.join(csrc, f)):
            return None
    return calls.get(call)


def _cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, inputs, C_full):
    """The oracle as it stands (the one the full-size parity tests use) on the
    whole workload, the same inputs and routing as the GPU step: routing,
    moves and router backward in the plain-loop C oracle (OpenMP over
    tokens), the expert MLP in float64 matrix products (multi-threaded BLAS).
    Input widening to float64 is not timed."""
    import oracle
    from oracle.layer_full import layer_packed
    from paper_2608_16188_amd import workloads as W
    oracle.load()
    f = {key: W.to_f64(inputs[key], cfg.dtype) for key in ("x", "w_router", "w1", "b1", "w2",
                                                            "b2", "dy")}
    threads = int(os.environ.get("OMP_NUM_THREADS") or os.cpu_count() or 1)
    t0 = time.perf_counter()
    layer_packed(f["x"], f["w_router"], f["w1"], f["b1"], f["w2"], f["b2"], f["dy"], k=cfg.k,
                 C=C_full, n_groups=cfg.n_groups, bias=inputs["logit_bias"],
                 noise=inputs["noise"], want_dwr=not cfg.routers_frozen)
    dt = time.perf_counter() - t0
    return {"value": cfg.n_tokens / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"the whole workload ({cfg.n_tokens} tokens, its own routing), one "
                      f"forward + backward in float64: C oracle (OpenMP) for routing, moves "
                      f"and router backward, float64 BLAS products for the expert MLP; "
                      f"{dt:.1f} s on {threads} threads",
            "nproc": os.cpu_count(), "cpu_model": _cpu_model()}


def balance_losses(L, V, stream, K):
    """The auxiliary balance losses (importance and load CV^2 per group, with
    their logit gradient) and the router backward that takes that gradient,
    timed after the layer step on the same buffers (not part of the step)."""
    import torch
    s, cfg = L.shape, L.cfg
    N, G, E = cfg.n_tokens, cfg.n_groups, cfg.n_experts
    # the load term's width is the standard deviation the gating noise was
    # drawn with; a noise-free workload takes 1/E as its smoothing width
    noisy = L.noise is not None
    sigma = float(np.sqrt(cfg.noise_var)) if noisy else 1.0 / E
    f32 = torch.float32
    losses = torch.empty(G, 2, dtype=f32, device="cuda")
    dl = torch.empty(max(N, 1), E, dtype=f32, device="cuda")
    ws = torch.empty(max(V.vmoe_balance_loss_workspace_bytes(s), 16), dtype=torch.uint8,
                     device="cuda")

    def loss():
        V.vmoe_balance_loss(s, L.logits, L.logit_bias, L.noise, L.probs, sigma, 0.01, 0.01,
                            losses, None, None, dl, ws, stream)

    def bwd(with_dl):
        if with_dl:
            V.vmoe_dispatch_route_bwd_dlogits(s, L.dxe, L.row_base, L.x, L.w_router, L.probs,
                                              L.expert_idx, L.slot, L.dgate, dl, L.dx,
                                              L.dw_router, L.route_bwd_ws, stream)
        else:
            V.vmoe_dispatch_route_bwd(s, L.dxe, L.row_base, L.x, L.w_router, L.probs,
                                      L.expert_idx, L.slot, L.dgate, L.dx, L.dw_router,
                                      L.route_bwd_ws, stream)

    def timed(fn):
        for _ in range(3):
            fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(K):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / K

    ms = timed(loss)
    ms_bwd = timed(lambda: bwd(False))
    ms_bwd_dl = timed(lambda: bwd(True))
    # two passes read logits and probs (and noise), the second writes dlogits
    rows = 2 + (L.noise is not None)
    nbytes = (2 * rows + 1) * N * E * 4
    return {"ms": round(ms, 4), "gbs": round(nbytes / (ms * 1e-3) / 1e9, 1),
            "algorithmic_bytes": nbytes,
            ("noise_std" if noisy else "smoothing_width_no_noise"): sigma,
            "dispatch_route_bwd_ms": round(ms_bwd, 4),
            "dispatch_route_bwd_dlogits_ms": round(ms_bwd_dl, 4),
            "note": "vmoe_balance_loss, then the fused router backward without and with its "
                    "logit gradient; timed after the step, not part of it"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="vitl16_384_bf16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--flush-mall", action="store_true",
                    help="after the timed region, time every call again with a 512 MiB "
                         "buffer written before each step (the 256 MB MALL holds no inputs)")
    ap.add_argument("--no-diagnostics", action="store_true",
                    help="skip the passes after the timed region that run other calls (the "
                         "quota-scheduled and dispatch-fused steps, the balance losses), so a "
                         "profiler run sees the step's kernels only")
    ap.add_argument("--copy-probe", action="store_true",
                    help="before warm-up, copy one 256 MiB buffer (a plain copy kernel of known "
                         "size, to calibrate the HBM byte counters of a profiler run)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (--gpus {args.gpus} requested); the layer's "
              "multi-GPU sharding is a design note, not part of this build.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_16188_amd import vmoe as V
    from paper_2608_16188_amd import workloads as W
    from paper_2608_16188_amd.layer import LayerBuffers

    cfg = W.CONFIGS[args.workload]
    inputs = W.make_inputs(cfg)
    torch.cuda.set_device(0)
    L = LayerBuffers(cfg, inputs)
    # A stream of its own (default priority): the same chain of kernels on the
    # null stream measured about 3 % slower (longer gaps between kernels).
    torch.cuda.synchronize()  # the buffers above were filled on the null stream
    stream = torch.cuda.Stream()
    torch.cuda.set_stream(stream)
    s = L.shape

    calls = {
        "route": lambda: L.route(stream=stream),
        "dispatch": lambda: V.vmoe_dispatch(s, L.x, L.expert_idx, L.slot, L.row_base, L.xe,
                                            stream),
        "ffn_fwd": lambda: V.vmoe_expert_ffn_fwd(s, L.xe, L.counts, L.w1, L.b1, L.w2, L.b2, L.a,
                                                 L.a_grad, L.ye, stream),
        "combine_fwd": lambda: V.vmoe_combine_fwd(s, L.ye, L.expert_idx, L.slot, L.row_base,
                                                  L.gate, L.y, stream),
        "combine_bwd": lambda: V.vmoe_combine_bwd(s, L.dy, L.ye, L.expert_idx, L.slot,
                                                  L.row_base, L.gate, L.dye, L.dgate, stream),
        "ffn_bwd": lambda: V.vmoe_expert_ffn_bwd(s, L.xe, L.counts, L.w1, L.w2, L.a, L.a_grad,
                                                 L.dye, L.dh, L.dxe, L.dw1, L.db1, L.dw2, L.db2,
                                                 stream),
        "dispatch_bwd": lambda: V.vmoe_dispatch_bwd(s, L.dxe, L.expert_idx, L.slot, L.row_base,
                                                    L.dx, stream),
        "route_bwd": lambda: V.vmoe_route_bwd(s, L.x, L.w_router, L.probs, L.expert_idx, L.slot,
                                              L.dgate, L.dx, L.dw_router, L.route_bwd_ws, stream),
        "dispatch_route_bwd": lambda: V.vmoe_dispatch_route_bwd(
            s, L.dxe, L.row_base, L.x, L.w_router, L.probs, L.expert_idx, L.slot, L.dgate, L.dx,
            L.dw_router, L.route_bwd_ws, stream),
        # the expert MLP through the fill-clamp-refill tile scheduler (same results)
        "ffn_fwd_quota": lambda: V.vmoe_expert_ffn_fwd_quota(
            s, L.xe, L.counts, L.w1, L.b1, L.w2, L.b2, L.a, L.a_grad, L.ye, stream),
        "ffn_bwd_quota": lambda: V.vmoe_expert_ffn_bwd_quota(
            s, L.xe, L.counts, L.w1, L.w2, L.a, L.a_grad, L.dye, L.dh, L.dxe, L.dw1, L.db1, L.dw2,
            L.db2, stream),
        # the dispatch fused into the expert MLP's loads (no xe; same results)
        "dispatch_ffn_fwd": lambda: V.vmoe_dispatch_ffn_fwd(
            s, L.x, L.expert_idx, L.slot, L.row_base, L.counts, L.w1, L.b1, L.w2, L.b2,
            L.row_token, L.a, L.a_grad, L.ye, stream),
        "ffn_bwd_gather": lambda: V.vmoe_expert_ffn_bwd_gather(
            s, L.x, L.row_token, L.counts, L.w1, L.w2, L.a, L.a_grad, L.dye, L.dh, L.dxe, L.dw1,
            L.db1, L.dw2, L.db2, stream),
    }

    if args.copy_probe:
        src = torch.ones(256 << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    for _ in range(args.warmup):
        for name in CALLS:
            calls[name]()
    torch.cuda.synchronize()

    K = args.steps
    # Timed region: K whole steps; the only events inside bracket the
    # roofline's kernel call, the expert-MLP backward (two thirds of the
    # step's flops), so the step carries no other instrumentation (events
    # around both expert-MLP calls measured ~11 us per step slower).
    dom = "ffn_bwd"
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        for name in CALLS:
            if name == dom:
                ev[i][0].record(stream)
                calls[name]()
                ev[i][1].record(stream)
            else:
                calls[name]()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / K
    dom_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))

    # Per-call breakdown (diagnostic, after the timed region): every call
    # bracketed by events on the call stream.
    evc = [[torch.cuda.Event(enable_timing=True) for _ in range(len(CALLS) + 1)] for _ in range(K)]
    torch.cuda.synchronize()
    for i in range(K):
        evc[i][0].record(stream)
        for c, name in enumerate(CALLS):
            calls[name]()
            evc[i][c + 1].record(stream)
    torch.cuda.synchronize()
    per_call = {name: float(np.mean([evc[i][c].elapsed_time(evc[i][c + 1]) for i in range(K)]))
                for c, name in enumerate(CALLS)}
    step_ms_events = float(np.mean([evc[i][0].elapsed_time(evc[i][-1]) for i in range(K)]))

    # the same step with the expert MLP calls through the fill-clamp-refill
    # tile scheduler, each call bracketed by events (diagnostic)
    quota = None
    if cfg.dtype == "bf16" and not args.no_diagnostics:
        qcalls = [("ffn_fwd_quota" if n == "ffn_fwd" else "ffn_bwd_quota" if n == "ffn_bwd"
                   else n) for n in CALLS]
        evq = [[torch.cuda.Event(enable_timing=True) for _ in range(len(CALLS) + 1)]
               for _ in range(K)]
        for i in range(K):
            evq[i][0].record(stream)
            for c, name in enumerate(qcalls):
                calls[name]()
                evq[i][c + 1].record(stream)
        torch.cuda.synchronize()
        qt = [float(np.mean([evq[i][c].elapsed_time(evq[i][c + 1]) for i in range(K)]))
              for c in range(len(CALLS))]
        quota = {"ffn_fwd_ms": round(qt[CALLS.index("ffn_fwd")], 4),
                 "ffn_bwd_ms": round(qt[CALLS.index("ffn_bwd")], 4),
                 "step_ms_events": float(np.mean([evq[i][0].elapsed_time(evq[i][-1])
                                                  for i in range(K)])),
                 "note": "vmoe_expert_ffn_fwd_quota / _bwd_quota (persistent workgroups, "
                         "per-expert quotas by fill-clamp-refill) in place of the default "
                         "calls; compare per_call ffn_fwd / ffn_bwd"}

    # the step with the dispatch fused into the expert MLP's loads: the
    # dispatch call is gone, the forward and backward read x through row_token
    gathered = None
    if cfg.dtype == "bf16" and L.C * cfg.n_groups <= 6144 and not args.no_diagnostics:
        gcalls = ["route", "dispatch_ffn_fwd", "combine_fwd", "combine_bwd", "ffn_bwd_gather",
                  "dispatch_route_bwd"]
        evg = [[torch.cuda.Event(enable_timing=True) for _ in range(len(gcalls) + 1)]
               for _ in range(K)]
        for i in range(K):
            evg[i][0].record(stream)
            for c, name in enumerate(gcalls):
                calls[name]()
                evg[i][c + 1].record(stream)
        torch.cuda.synchronize()
        gt = {name: float(np.mean([evg[i][c].elapsed_time(evg[i][c + 1]) for i in range(K)]))
              for c, name in enumerate(gcalls)}
        gathered = {"per_call_ms": {n: round(v, 4) for n, v in gt.items()},
                    "step_ms_events": float(np.mean([evg[i][0].elapsed_time(evg[i][-1])
                                                     for i in range(K)])),
                    "note": "vmoe_dispatch_ffn_fwd in place of vmoe_dispatch + "
                            "vmoe_expert_ffn_fwd, vmoe_expert_ffn_bwd_gather in place of "
                            "vmoe_expert_ffn_bwd (xe never written)"}

    # the same step captured once in a HIP graph and replayed K times
    # (diagnostic: the kernels are the step's, only the launch path differs)
    graph = None
    if not args.no_diagnostics:
        g = torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=stream):
            for name in CALLS:
                calls[name]()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(K):
            g.replay()
        b.record(stream)
        torch.cuda.synchronize()
        graph = {"ms_per_step": a.elapsed_time(b) / K,
                 "note": "the step's seven calls captured in one HIP graph, K replays"}
        del g

    flushed = None
    if args.flush_mall:
        # per-call times with the MALL flushed before every step: a 512 MiB
        # buffer is written between steps, outside the events
        scratch = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
        evf = [[torch.cuda.Event(enable_timing=True) for _ in range(len(CALLS) + 1)]
               for _ in range(K)]
        for i in range(K):
            scratch.fill_(i & 0xFF)
            evf[i][0].record(stream)
            for c, name in enumerate(CALLS):
                calls[name]()
                evf[i][c + 1].record(stream)
        torch.cuda.synchronize()
        del scratch
        flushed = {name: float(np.mean([evf[i][c].elapsed_time(evf[i][c + 1])
                                        for i in range(K)])) for c, name in enumerate(CALLS)}

    balance = None if args.no_diagnostics else balance_losses(L, V, stream, K)

    counts = L.counts.cpu().numpy()
    A = int(counts.sum())
    NK = int((L.slot.view(cfg.n_tokens, cfg.k) >= 0).any(dim=1).sum().item())
    cost = algorithmic_cost(cfg, A, L.noise is not None, L.logit_bias is not None, NK)
    peak_mfma = PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_F32_TFLOPS
    fl, by = cost[dom]
    ach = fl / (dom_ms * 1e-3) / 1e12
    ach_gbs = by / (dom_ms * 1e-3) / 1e9
    # the call's binding roof: the larger of its matrix-core time at peak and
    # its algorithmic HBM bytes at peak bandwidth
    hbm_bound = by / (PEAK_HBM_GBS * 1e9) > fl / (peak_mfma * 1e12)
    if hbm_bound:
        roof = {"bound": "hbm", "kernel": f"vmoe_expert_{dom}", "achieved": ach_gbs,
                "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": ach_gbs / PEAK_HBM_GBS}
    else:
        roof = {"bound": "mfma", "kernel": f"vmoe_expert_{dom}", "achieved": ach,
                "peak": peak_mfma, "unit": "TFLOP/s", "frac": ach / peak_mfma}
    roof.update({"traffic": measured_traffic(args.workload, dom), "algorithmic_bytes": by,
                 "algorithmic_flops": fl, "mfma_frac": ach / peak_mfma,
                 "hbm_frac": ach_gbs / PEAK_HBM_GBS, "ms": dom_ms})
    # the expert-MLP summary: the backward from the timed region, the forward
    # from the per-call pass
    ffn_total_ms = per_call["ffn_fwd"] + dom_ms
    ffn_tflops = (cost["ffn_fwd"][0] + cost["ffn_bwd"][0]) / (ffn_total_ms * 1e-3) / 1e12
    moves = [n for n in CALLS if not n.startswith("ffn")]
    moves_bytes = sum(cost[n][1] for n in moves)
    moves_ms = sum(per_call[n] for n in moves)
    breakdown = {n: {"ms": round(per_call[n], 4),
                     "tflops": round(cost[n][0] / (per_call[n] * 1e-3) / 1e12, 2),
                     "gbs": round(cost[n][1] / (per_call[n] * 1e-3) / 1e9, 1)} for n in CALLS}

    out = {
        "metric": METRIC,
        "value": cfg.n_tokens / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.images} images x {cfg.tokens_per_image} tokens "
                               f"= {cfg.n_tokens} tokens, d_model {cfg.d_model}, d_ff {cfg.d_ff}, "
                               f"E {cfg.n_experts}, top-{cfg.k}, capacity factor "
                               f"{cfg.capacity_factor}, groups {cfg.n_groups}",
                   "global_batch": cfg.images, "seq_len": cfg.tokens_per_image,
                   "capacity": L.C, "kept_assignments": A, "parallelism": "single GPU"},
        "roofline": roof,
        "expert_gemms": {"tflops": ffn_tflops, "frac_of_peak": ffn_tflops / peak_mfma,
                         "ms": ffn_total_ms},
        "route_dispatch_combine": {"gbs": moves_bytes / (moves_ms * 1e-3) / 1e9,
                                   "frac_of_hbm": moves_bytes / (moves_ms * 1e-3) / 1e9
                                   / PEAK_HBM_GBS, "ms": moves_ms},
        "per_call": breakdown,
        "per_call_note": "diagnostic pass after the timed region, every call bracketed by events",
        "step_ms_events": step_ms_events,
        "balance_losses": balance,
        "ffn_quota_scheduler": quota,
        "dispatch_fused_step": gathered,
        "graph_step": graph,
    }
    if flushed is not None:
        fb = sum(cost[n][1] for n in moves)
        fm = sum(flushed[n] for n in moves)
        out["mall_flushed"] = {
            "per_call_ms": {n: round(v, 4) for n, v in flushed.items()},
            "route_dispatch_combine_gbs": fb / (fm * 1e-3) / 1e9,
            "route_dispatch_combine_frac_of_hbm": fb / (fm * 1e-3) / 1e9 / PEAK_HBM_GBS,
            "ffn_bwd_gbs": by / (flushed[dom] * 1e-3) / 1e9,
            "note": "a 512 MiB buffer written before each step, outside the events"}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, inputs, L.C)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
