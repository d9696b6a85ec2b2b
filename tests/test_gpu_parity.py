"""GPU parity: the HIP path through the C ABI vs the CPU oracle.

Router logits: bit for bit for f32 activations; for bf16 activations (an
f32 sum on the matrix cores) within the f32 summation error bound of each
logit. Routing is a decision taken on the f32 logits, so the oracle routes
the GPU's logits and integers (routing indices, slots, drop masks, order,
counts, row bases), probabilities and gates must then match bit for bit;
float outputs and gradients within max|gpu - oracle| / max|oracle| <= 2e-2
(bf16) or 1e-4 (f32). Small cases compare every element; the full-size workloads,
run exactly as the benchmark runs them, compare routing in full and sampled
outputs that the oracle computes one by one.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_16188_amd import vmoe as V
from paper_2608_16188_amd import workloads as W
from paper_2608_16188_amd.layer import LayerBuffers, to_numpy

from .gpu_common import (TOL, as_f64, assert_close, assert_router_logits, bits_equal,
                         oracle_capacity, say, workload_inputs)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _f64_out(t, dtype):
    """A whole output buffer as float64; rows past an expert's count are never
    written and may hold any bits (signalling NaNs included)."""
    a = to_numpy(t)
    with np.errstate(invalid="ignore"):
        return W.to_f64(a, dtype) if a.dtype == np.uint16 else a.astype(np.float64)


# ------------------------------------------------------------------ routing

def _gpu_route_logits_in(logits, k, G, bias=None, noise=None, capacity_override=0, cf=1.0):
    N, E = logits.shape
    s = V.make_shape(N, G, 8, 8, E, k, cf, V.VMOE_BF16, 0, capacity_override)
    C = V.vmoe_capacity(s)
    dev = "cuda"
    Nb = max(N, 1)
    lg = torch.zeros(Nb, E, dtype=torch.float32, device=dev)
    if N:
        lg[:N] = torch.from_numpy(logits).to(dev)
    out = dict(
        probs=torch.empty(Nb, E, dtype=torch.float32, device=dev),
        idx=torch.empty(Nb, k, dtype=torch.int32, device=dev),
        slot=torch.empty(Nb, k, dtype=torch.int32, device=dev),
        gate=torch.empty(Nb, k, dtype=torch.float32, device=dev),
        order=torch.empty(Nb, dtype=torch.int32, device=dev),
        counts=torch.empty(G, E, dtype=torch.int32, device=dev),
        row_base=torch.empty(G, E, dtype=torch.int32, device=dev),
    )
    ws = torch.empty(max(V.vmoe_route_workspace_bytes(s), 16), dtype=torch.uint8, device=dev)
    b = None if bias is None else torch.from_numpy(bias).to(dev)
    nz = None if noise is None else torch.from_numpy(noise).to(dev)
    V.vmoe_route(s, None, None, b, nz, V.VMOE_ROUTE_LOGITS_IN, lg, out["probs"], out["idx"],
                 out["slot"], out["gate"], out["order"], out["counts"], out["row_base"], ws)
    torch.cuda.synchronize()
    res = {key: to_numpy(v) for key, v in out.items()}
    for key in ("probs", "idx", "slot", "gate", "order"):
        res[key] = res[key][:N]
    return res, C


def _compare_routing(got, ref, what=""):
    for key in ("idx", "slot", "order", "counts", "row_base"):
        assert np.array_equal(got[key], ref[key]), f"{what} {key} differs"
    for key in ("probs", "gate"):
        assert bits_equal(got[key], ref[key]), f"{what} {key} not bit-exact"


ROUTE_CASES = [
    # name, N, E, k, G, kwargs
    ("random", 500, 8, 2, 1, dict(seed=1, scale=2.0)),
    ("ties", 640, 6, 3, 2, dict(seed=2, tie_every=2)),
    ("all_equal", 333, 5, 2, 1, dict(zero=True)),
    ("capacity1", 200, 8, 2, 4, dict(seed=3, capacity_override=1)),
    ("e_equals_k", 128, 4, 4, 1, dict(seed=4)),
    ("single_expert", 90, 1, 1, 3, dict(seed=5)),
    ("groups17", 17 * 96, 16, 2, 17, dict(seed=6, scale=3.0)),
    ("e64", 1000, 64, 8, 1, dict(seed=7, scale=1.5)),
    ("hot_expert_drops", 3000, 8, 2, 1, dict(seed=8, hot=True)),
    ("many_equal_priorities", 20000, 4, 2, 1, dict(seed=9, tie_every=1)),
    ("noise_and_bias", 777, 12, 3, 1, dict(seed=10, noise=True)),
    ("ragged_chunks", 3 * 257, 8, 2, 3, dict(seed=11)),
    ("empty", 0, 8, 2, 1, dict(seed=12)),
    # one block per group up to 8192 tokens and 16384 assignments, else the
    # multi-kernel path: both sides of that limit, and a one-bin worst case
    ("single_block_limit", 8192, 8, 2, 1, dict(seed=13, scale=2.0)),
    ("single_block_limit_plus_one", 8193, 8, 2, 1, dict(seed=14, scale=2.0)),
    ("single_block_equal_priorities", 8000, 4, 2, 1, dict(seed=15, tie_every=1)),
    ("single_block_k4_groups", 4 * 4096, 16, 4, 4, dict(seed=16, scale=2.0)),
    ("many_small_groups_e64", 300 * 8, 64, 2, 300, dict(seed=17, scale=2.0)),
    # the multi-block path with several groups: groups past 8192 tokens (hist
    # blocks of 4096 with a ragged last one, row bases across groups), and
    # groups of fewer tokens whose assignments pass 16384 (k = 4)
    ("multi_block_two_groups", 2 * 9000, 8, 2, 2, dict(seed=18, scale=2.0)),
    ("multi_block_k4_three_groups", 3 * 5000, 16, 4, 3, dict(seed=19, scale=2.0)),
    ("multi_block_groups_equal_priorities", 2 * 8500, 4, 2, 2, dict(seed=20, tie_every=1)),
]


@pytest.mark.parametrize("case", ROUTE_CASES, ids=[c[0] for c in ROUTE_CASES])
def test_route_logits_in_bit_exact(case):
    name, N, E, k, G, kw = case
    say("route logits-in", name, N, E, k, G)
    if kw.get("zero"):
        logits = np.zeros((N, E), np.float32)
    else:
        logits = W.random_logits(N, E, seed=kw["seed"], scale=kw.get("scale", 1.0),
                                 tie_every=kw.get("tie_every", 0))
    bias = noise = None
    if kw.get("hot"):
        bias = np.zeros(E, np.float32)
        bias[0] = 3.0
    if kw.get("noise"):
        bias = np.linspace(-0.5, 0.5, E).astype(np.float32)
        noise = W.random_logits(N, E, seed=99, scale=0.3)
    got, C = _gpu_route_logits_in(logits, k, G, bias, noise, kw.get("capacity_override", 0))
    ref = oracle.route(logits, k, C, G, bias, noise)
    _compare_routing(got, ref, name)
    if name == "hot_expert_drops":
        assert (ref["slot"] < 0).sum() > 1000


@pytest.mark.parametrize("name", list(W.CONFIGS))
def test_route_full_size_bit_exact(name):
    """Router product + routing at the benchmark sizes (routing of the GPU logits)."""
    cfg, inp = workload_inputs(name, with_experts=False)
    say("route full", name)
    L = LayerBuffers(cfg, inp)
    L.route()
    torch.cuda.synchronize()
    x64 = as_f64(inp["x"], cfg.dtype)
    wr64 = as_f64(inp["w_router"], cfg.dtype)
    logits = to_numpy(L.logits)
    assert_router_logits(logits, x64, wr64, cfg.n_groups, cfg.dtype)
    C = oracle_capacity(cfg)
    assert L.C == C
    ref = oracle.route(logits, cfg.k, C, cfg.n_groups, inp["logit_bias"], inp["noise"])
    got = dict(idx=to_numpy(L.expert_idx), slot=to_numpy(L.slot), order=to_numpy(L.order),
               counts=to_numpy(L.counts), row_base=to_numpy(L.row_base),
               probs=to_numpy(L.probs), gate=to_numpy(L.gate))
    _compare_routing(got, ref, name)


# ------------------------------------------------------------------ whole layer, small

SMALL = [
    W.CONFIGS["tiny_fp32"],
    W.custom_config("bf16_ragged", n_tokens=300, d_model=72, d_ff=200, n_experts=5, k=2,
                    capacity_factor=0.8, n_groups=3, router_std=0.2, noise_var=0.1),
    W.custom_config("bf16_tiles", n_tokens=520, d_model=256, d_ff=512, n_experts=4, k=1,
                    capacity_factor=1.5, router_std=0.1),
    W.custom_config("f32_ragged", n_tokens=210, d_model=40, d_ff=136, n_experts=3, k=2,
                    capacity_factor=1.0, dtype=W.F32, n_groups=2, router_std=0.2),
    W.custom_config("bf16_hot_empty", n_tokens=256, d_model=128, d_ff=384, n_experts=8, k=2,
                    capacity_factor=1.0, hot_experts=2, hot_offset=6.0),
    # k > 2 (row moves in passes of four assignments), 17..32 and 33..64 experts
    # (router backward with 32 / 64 expert columns), ragged widths
    W.custom_config("bf16_k4_e20", n_tokens=400, d_model=96, d_ff=160, n_experts=20, k=4,
                    capacity_factor=1.0, n_groups=2, router_std=0.3),
    W.custom_config("bf16_k6_e64", n_tokens=300, d_model=64, d_ff=128, n_experts=64, k=6,
                    capacity_factor=2.0, router_std=0.3, noise_var=0.05),
    W.custom_config("f32_k3", n_tokens=150, d_model=48, d_ff=96, n_experts=6, k=3,
                    capacity_factor=0.9, dtype=W.F32, router_std=0.2),
    # degenerate layers: one expert (a plain MLP on every token), every token
    # on every expert, and a capacity of 2 that drops almost every assignment
    W.custom_config("bf16_single_expert", n_tokens=128, d_model=64, d_ff=128, n_experts=1, k=1,
                    capacity_factor=1.0, router_std=0.2),
    W.custom_config("bf16_k_equals_e", n_tokens=96, d_model=64, d_ff=96, n_experts=4, k=4,
                    capacity_factor=1.0, router_std=0.3),
    W.custom_config("f32_capacity_two", n_tokens=200, d_model=32, d_ff=64, n_experts=4, k=2,
                    capacity_factor=0.02, dtype=W.F32, router_std=0.2),
    # several 256-row m-tiles per expert, every element: ten (the forward
    # GEMMs' patches of four m-tiles and a partial last patch) and eight (one
    # whole m-column per XCD chunk), with ragged n-tiles and k tails
    W.custom_config("bf16_ten_mtiles", n_tokens=2400, d_model=72, d_ff=264, n_experts=2, k=2,
                    capacity_factor=1.0, router_std=0.05),
    W.custom_config("bf16_eight_mtiles", n_tokens=3000, d_model=136, d_ff=520, n_experts=3,
                    k=2, capacity_factor=0.9, router_std=0.1),
    # heavy and light experts in one launch: two experts full (500 rows, two
    # m-tiles each), six with 53-85 rows, so the d-wide row GEMMs spread the
    # heavy experts' tile chunks among the light ones (a partial chunk in
    # each class)
    W.custom_config("bf16_two_classes", n_tokens=2000, d_model=72, d_ff=264, n_experts=8, k=2,
                    capacity_factor=1.0, hot_experts=2, hot_offset=2.0, router_std=0.1),
    # light experts: two experts full at 280 rows (a 24-row last m-tile), the
    # other 14 with 15-47 rows (most within one 32-row block), so the light
    # tiles' register-streamed path runs, with its column parts in the d-wide
    # GEMMs, beside the stage ring; k and n ragged (d 200, f 520)
    W.custom_config("bf16_light_tails", n_tokens=2240, d_model=200, d_ff=520, n_experts=16, k=2,
                    capacity_factor=1.0, hot_experts=2, hot_offset=0.8),
]


def _oracle_layer(cfg, inp, C, logits):
    f = {key: (None if v is None else as_f64(v, cfg.dtype))
         for key, v in inp.items() if key not in ("logit_bias", "noise")}
    return oracle.layer(f["x"], f["w_router"], f["w1"], f["b1"], f["w2"], f["b2"], f["dy"],
                        k=cfg.k, C=C, n_groups=cfg.n_groups, bias=inp["logit_bias"],
                        noise=inp["noise"], logits=logits, want_dwr=not cfg.routers_frozen)


@pytest.mark.parametrize("cfg", SMALL, ids=[c.name for c in SMALL])
def test_layer_small_every_element(cfg):
    inp = W.make_inputs(cfg)
    say("layer small", cfg.name)
    L = LayerBuffers(cfg, inp)
    L.step()
    torch.cuda.synchronize()
    C = oracle_capacity(cfg)
    logits = to_numpy(L.logits)
    assert_router_logits(logits, as_f64(inp["x"], cfg.dtype), as_f64(inp["w_router"], cfg.dtype),
                         cfg.n_groups, cfg.dtype)
    ref = _oracle_layer(cfg, inp, C, logits)
    tol = TOL[cfg.dtype]
    got_r = dict(idx=to_numpy(L.expert_idx), slot=to_numpy(L.slot), order=to_numpy(L.order),
                 counts=to_numpy(L.counts), row_base=to_numpy(L.row_base),
                 probs=to_numpy(L.probs), gate=to_numpy(L.gate))
    _compare_routing(got_r, ref, cfg.name)
    n_e = ref["n_e"]
    dt = cfg.dtype
    xe, a, ag, ye = (_f64_out(t, dt) for t in (L.xe, L.a, L.a_grad, L.ye))
    dye, dh, dxe = (_f64_out(t, dt) for t in (L.dye, L.dh, L.dxe))
    for e in range(cfg.n_experts):
        r = slice(0, n_e[e])
        assert np.array_equal(xe[e, r], ref["xe"][e, r]), "dispatch not exact"
        assert_close(f"A[{e}]", a[e, r], ref["A"][e, r], tol)
        assert_close(f"A'[{e}]", ag[e, r], ref["Gd"][e, r], tol)
        assert_close(f"ye[{e}]", ye[e, r], ref["ye"][e, r], tol)
        assert_close(f"dye[{e}]", dye[e, r], ref["dye"][e, r], tol)
        assert_close(f"dH[{e}]", dh[e, r], ref["dH"][e, r], tol)
        assert_close(f"dxe[{e}]", dxe[e, r], ref["dxe"][e, r], tol)
    assert_close("y", _f64_out(L.y, dt), ref["y"], tol)
    assert_close("dgate", to_numpy(L.dgate), ref["dgate"], tol)
    assert_close("dW1", to_numpy(L.dw1), ref["dw1"], tol)
    assert_close("db1", to_numpy(L.db1), ref["db1"], tol)
    assert_close("dW2", to_numpy(L.dw2), ref["dw2"], tol)
    assert_close("db2", to_numpy(L.db2), ref["db2"], tol)
    assert_close("dx", to_numpy(L.dx), ref["dx"], tol)
    if not cfg.routers_frozen:
        assert_close("dW_router", to_numpy(L.dw_router), ref["dw_router"], tol)
    for e in np.nonzero(n_e == 0)[0]:
        assert np.all(to_numpy(L.dw1)[e] == 0) and np.all(to_numpy(L.dw2)[e] == 0)
        assert np.all(to_numpy(L.db1)[e] == 0) and np.all(to_numpy(L.db2)[e] == 0)


@pytest.mark.parametrize("dtype", [W.BF16, W.F32])
def test_layer_empty_batch(dtype):
    """No tokens: every call runs, the weight, bias and router gradients are
    exactly zero (the closed form of an empty sum)."""
    cfg = W.custom_config(f"empty_{dtype}", n_tokens=0, d_model=64, d_ff=128, n_experts=4, k=2,
                          capacity_factor=1.0, dtype=dtype)
    say("layer empty", dtype)
    L = LayerBuffers(cfg, W.make_inputs(cfg))
    for t in (L.dw1, L.db1, L.dw2, L.db2, L.dw_router):
        t.fill_(float("nan"))
    L.step()
    torch.cuda.synchronize()
    for name in ("dw1", "db1", "dw2", "db2", "dw_router"):
        assert torch.all(getattr(L, name) == 0), name
    assert int(L.counts.sum()) == 0


FUSED_CASES = [c.name for c in SMALL] + ["vitb16_bf16", "vitl16_384_bf16"]


@pytest.mark.parametrize("name", FUSED_CASES)
def test_dispatch_route_bwd_matches_two_calls(name):
    """The fused dispatch + router backward is bit-identical to the two calls
    (k <= 4 gathers in the router kernel; larger k runs the two passes)."""
    cfg = next((c for c in SMALL if c.name == name), None) or W.CONFIGS[name]
    say("dispatch+route bwd", name)
    inp = W.make_inputs(cfg)
    L = LayerBuffers(cfg, inp)
    L.forward()
    L.backward(fused=False)
    torch.cuda.synchronize()
    dx2 = L.dx.clone()
    dw2 = None if L.dw_router is None else L.dw_router.clone()
    L.dx.fill_(float("nan"))
    if dw2 is not None:
        L.dw_router.fill_(float("nan"))
    L.backward(fused=True)
    torch.cuda.synchronize()
    assert torch.equal(L.dx.view(torch.int32), dx2.view(torch.int32)), "dx differs"
    if dw2 is not None:
        assert torch.equal(L.dw_router.view(torch.int32), dw2.view(torch.int32)), "dW_r differs"


def test_route_bwd_full_size_per_call():
    """Router backward alone at the ViT-L/16 size, fed the oracle's routing."""
    cfg, inp = workload_inputs("vitl16_384_bf16", with_experts=False)
    say("route_bwd full")
    f = {key: as_f64(inp[key], cfg.dtype) for key in ("x", "w_router")}
    C = oracle_capacity(cfg)
    ref = oracle.route(oracle.router_logits(f["x"], f["w_router"], 1), cfg.k, C, 1,
                       inp["logit_bias"], inp["noise"])
    dgate = W.random_logits(cfg.n_tokens, cfg.k, seed=31)
    dx0 = W.random_logits(cfg.n_tokens, cfg.d_model, seed=32)
    s = V.make_shape(cfg.n_tokens, 1, cfg.d_model, cfg.d_ff, cfg.n_experts, cfg.k,
                     cfg.capacity_factor, V.VMOE_BF16)
    dev = "cuda"
    tx = torch.from_numpy(inp["x"].view(np.int16)).view(torch.bfloat16).to(dev)
    twr = torch.from_numpy(inp["w_router"].view(np.int16)).view(torch.bfloat16).to(dev)
    tp = torch.from_numpy(ref["probs"]).to(dev)
    ti = torch.from_numpy(ref["idx"]).to(dev)
    ts = torch.from_numpy(ref["slot"]).to(dev)
    tg = torch.from_numpy(dgate).to(dev)
    tdx = torch.from_numpy(dx0).to(dev)
    tdw = torch.empty(1, cfg.n_experts, cfg.d_model, dtype=torch.float32, device=dev)
    ws = torch.empty(V.vmoe_route_bwd_workspace_bytes(s), dtype=torch.uint8, device=dev)
    V.vmoe_route_bwd(s, tx, twr, tp, ti, ts, tg, tdx, tdw, ws)
    torch.cuda.synchronize()
    dx_ref, dwr_ref, _ = oracle.route_bwd(f["x"], f["w_router"], ref["probs"], ref["idx"],
                                          ref["slot"], dgate.astype(np.float64), 1,
                                          dx_in=dx0.astype(np.float64))
    assert_close("dx", to_numpy(tdx), dx_ref, 1e-5)
    assert_close("dW_router", to_numpy(tdw), dwr_ref, 1e-4)


def test_step_is_deterministic():
    cfg, inp = workload_inputs("vitb16_bf16")
    say("determinism")
    L = LayerBuffers(cfg, inp)
    names = ["logits", "probs", "expert_idx", "slot", "gate", "order", "counts", "y", "dgate",
             "dw1", "db1", "dw2", "db2", "dx", "dw_router"]
    L.step()
    torch.cuda.synchronize()
    first = {n: to_numpy(getattr(L, n)).copy() for n in names}
    L.step()
    torch.cuda.synchronize()
    for n in names:
        assert np.array_equal(first[n], to_numpy(getattr(L, n))), f"{n} not deterministic"
