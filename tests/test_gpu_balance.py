"""Balance losses on the GPU against the oracle: the per-group importance,
load and CV^2 losses with their logit gradient, and the router backward that
takes that gradient in. The gate probabilities fed to both sides come from the
oracle's gate."""
import numpy as np
import pytest
import torch

import oracle
from oracle import balance as OB
from paper_2608_16188_amd import vmoe as V
from paper_2608_16188_amd import workloads as W
from paper_2608_16188_amd.layer import LayerBuffers, to_numpy

from .gpu_common import TOL, as_f64, assert_close, bits_equal, oracle_capacity, say
from .test_gpu_parity import _oracle_layer

pytestmark = pytest.mark.gpu

# name, N, G, E, k, noise std, bias, noise, hot experts
CASES = [
    ("e8_k2", 600, 1, 8, 2, 1 / 8, False, True, 0),
    ("groups3_e5_bias", 3 * 257, 3, 5, 2, 0.2, True, True, 0),
    ("e16_k4_no_noise", 1000, 2, 16, 4, 1 / 16, False, False, 0),
    ("e33_k3", 513, 1, 33, 3, 0.05, True, True, 0),
    ("e64_k8", 700, 1, 64, 8, 1 / 64, False, True, 0),
    ("k_equals_e", 300, 1, 4, 4, 0.25, False, True, 0),
    ("e8_bias_no_noise", 512, 2, 8, 2, 0.125, True, False, 0),
    ("e24_bias_no_noise_hot", 480, 1, 24, 2, 0.1, True, False, 2),
    ("single_expert", 128, 2, 1, 1, 1.0, False, True, 0),
    ("empty", 0, 1, 8, 2, 0.125, False, True, 0),
    ("vitb16_6304_e8", 6304, 1, 8, 2, 1 / 8, False, True, 0),
    ("vitl16_36928_e32_hot", 36928, 1, 32, 2, 1 / 32, True, True, 4),
]


def _inputs(N, E, k, sigma, with_bias, with_noise, hot, seed):
    rng = np.random.default_rng(seed)
    logits = rng.normal(0.0, 1.0, (N, E)).astype(np.float32)
    bias = None
    if with_bias:
        bias = rng.normal(0.0, 0.3, E).astype(np.float32)
        bias[:hot] += 2.0
    noise = (sigma * rng.normal(0.0, 1.0, (N, E))).astype(np.float32) if with_noise else None
    probs = oracle.gate(logits, k, bias, noise)["probs"]
    return logits, bias, noise, probs


def _dev(a, rows=None):
    if a is None:
        return None
    t = torch.from_numpy(np.ascontiguousarray(a))
    if rows is not None and a.shape[0] == 0:  # an empty batch still passes allocated rows
        t = torch.zeros((1,) + a.shape[1:], dtype=t.dtype)
    return t.cuda()


def _run_balance(N, G, E, k, sigma, logits, bias, noise, probs, w_imp, w_load):
    s = V.make_shape(N, G, 64, 64, E, k, 1.0, V.VMOE_F32)
    f32 = torch.float32
    losses = torch.full((G, 2), float("nan"), dtype=f32, device="cuda")
    imp = torch.full((G, E), float("nan"), dtype=f32, device="cuda")
    load = torch.full((G, E), float("nan"), dtype=f32, device="cuda")
    dl = torch.full((max(N, 1), E), float("nan"), dtype=f32, device="cuda")
    ws = torch.empty(max(V.vmoe_balance_loss_workspace_bytes(s), 16), dtype=torch.uint8,
                     device="cuda")
    V.vmoe_balance_loss(s, _dev(logits, 1), _dev(bias), _dev(noise, 1), _dev(probs, 1), sigma,
                        w_imp, w_load, losses, imp, load, dl, ws)
    torch.cuda.synchronize()
    return to_numpy(losses), to_numpy(imp), to_numpy(load), to_numpy(dl)[:N]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_balance_loss_matches_oracle(case):
    name, N, G, E, k, sigma, wb, wn, hot = case
    say("balance loss", name, N, G, E, k)
    logits, bias, noise, probs = _inputs(N, E, k, sigma, wb, wn, hot, seed=N + E + k)
    w_imp, w_load = 0.01, 0.02
    losses, imp, load, dl = _run_balance(N, G, E, k, sigma, logits, bias, noise, probs, w_imp,
                                         w_load)
    ref = OB.balance_loss(logits, k, G, sigma, w_imp, w_load, bias=bias, noise=noise,
                          probs=probs)
    if N == 0:
        assert np.all(losses == 0) and np.all(imp == 0) and np.all(load == 0)
        return
    assert_close("importance", imp, ref["imp"], 1e-5)
    assert_close("load", load, ref["load"], 1e-5)
    np.testing.assert_allclose(losses, ref["losses"], rtol=1e-4, atol=1e-7)
    if np.abs(ref["dlogits"]).max() == 0:
        assert np.all(dl == 0)
    else:
        assert_close("dlogits", dl, ref["dlogits"], TOL[W.F32])


def test_balance_loss_rejects_bad_noise_std():
    s = V.make_shape(64, 1, 64, 64, 8, 2, 1.0, V.VMOE_F32)
    t = torch.zeros(64, 8, device="cuda")
    g = torch.zeros(1, 2, device="cuda")
    ws = torch.empty(max(V.vmoe_balance_loss_workspace_bytes(s), 16), dtype=torch.uint8,
                     device="cuda")
    for bad in (0.0, -1.0, float("inf"), float("nan")):
        with pytest.raises(V.VmoeError):
            V.vmoe_balance_loss(s, t, None, None, t, bad, 1.0, 1.0, g, None, None, t, ws)


BWD_CASES = [
    # fused gather (E <= 16, k <= 4); f32 with E > 16 and k > 4 take the two
    # passes; bf16 with E >= 32 the matrix-core kernel
    W.custom_config("aux_bf16_e8_k2", n_tokens=300, d_model=72, d_ff=64, n_experts=8, k=2,
                    capacity_factor=1.0, n_groups=3, router_std=0.3),
    W.custom_config("aux_f32_e20_k2", n_tokens=256, d_model=48, d_ff=64, n_experts=20, k=2,
                    capacity_factor=1.0, dtype=W.F32, router_std=0.3),
    W.custom_config("aux_bf16_e16_k6", n_tokens=200, d_model=64, d_ff=64, n_experts=16, k=6,
                    capacity_factor=1.0, router_std=0.3),
    W.custom_config("aux_bf16_e32_k2", n_tokens=640, d_model=256, d_ff=64, n_experts=32, k=2,
                    capacity_factor=1.0, n_groups=2, router_std=0.3),
]


@pytest.mark.parametrize("cfg", BWD_CASES, ids=[c.name for c in BWD_CASES])
def test_dispatch_route_bwd_dlogits(cfg):
    say("route bwd + dlogits", cfg.name)
    inp = W.make_inputs(cfg)
    L = LayerBuffers(cfg, inp)
    L.step()  # forward + backward; dx and dw_router without the extra term
    s = L.shape
    dx0, dwr0 = L.dx.clone(), L.dw_router.clone()
    zero = torch.zeros(cfg.n_tokens, cfg.n_experts, dtype=torch.float32, device="cuda")
    V.vmoe_dispatch_route_bwd_dlogits(s, L.dxe, L.row_base, L.x, L.w_router, L.probs,
                                      L.expert_idx, L.slot, L.dgate, zero, L.dx, L.dw_router,
                                      L.route_bwd_ws)
    torch.cuda.synchronize()
    assert bits_equal(to_numpy(L.dx), to_numpy(dx0)), "zero extra gradient changed dx"
    assert bits_equal(to_numpy(L.dw_router), to_numpy(dwr0)), "zero extra gradient changed dW_r"

    rng = np.random.default_rng(7)
    dl = (0.05 * rng.normal(0.0, 1.0, (cfg.n_tokens, cfg.n_experts))).astype(np.float32)
    V.vmoe_dispatch_route_bwd_dlogits(s, L.dxe, L.row_base, L.x, L.w_router, L.probs,
                                      L.expert_idx, L.slot, L.dgate, _dev(dl), L.dx,
                                      L.dw_router, L.route_bwd_ws)
    torch.cuda.synchronize()
    ref = _oracle_layer(cfg, inp, oracle_capacity(cfg), to_numpy(L.logits))
    ex_dx, ex_dwr = OB.router_grad_extra(as_f64(inp["x"], cfg.dtype),
                                         as_f64(inp["w_router"], cfg.dtype), dl, cfg.n_groups)
    tol = TOL[cfg.dtype]
    assert_close("dx", to_numpy(L.dx), ref["dx"] + ex_dx, tol)
    assert_close("dW_router", to_numpy(L.dw_router), ref["dw_router"] + ex_dwr, tol)


def test_balance_loss_and_router_backward_full_size():
    """ViT-B/16 (6304 tokens, E = 8) as the bench runs it: the losses and
    dlogits from the layer's own routing, and the change that dlogits makes to
    dx and dW_router, against the oracle (its gate re-run on the layer's f32
    logits gives the probabilities)."""
    cfg = W.CONFIGS["vitb16_bf16"]
    say("balance loss full size", cfg.name)
    inp = W.make_inputs(cfg)
    L = LayerBuffers(cfg, inp)
    L.step()
    torch.cuda.synchronize()
    s, N, G, E, k = L.shape, cfg.n_tokens, cfg.n_groups, cfg.n_experts, cfg.k
    # weights of the order of the token count, so that the logit gradient
    # moves dx well above its f32 rounding
    sigma, w_imp, w_load = 1.0 / E, float(N), float(N)
    logits = to_numpy(L.logits)
    bias = inp.get("logit_bias")
    noise = inp.get("noise")
    probs = oracle.gate(logits, k, bias, noise)["probs"]
    assert bits_equal(to_numpy(L.probs), probs), "router probabilities differ from the oracle's"
    ref = OB.balance_loss(logits, k, G, sigma, w_imp, w_load, bias=bias, noise=noise,
                          probs=probs)
    f32 = torch.float32
    losses = torch.empty(G, 2, dtype=f32, device="cuda")
    dl = torch.empty(N, E, dtype=f32, device="cuda")
    ws = torch.empty(max(V.vmoe_balance_loss_workspace_bytes(s), 16), dtype=torch.uint8,
                     device="cuda")
    V.vmoe_balance_loss(s, L.logits, L.logit_bias, L.noise, L.probs, sigma, w_imp, w_load,
                        losses, None, None, dl, ws)
    dx0, dwr0 = L.dx.clone(), L.dw_router.clone()
    V.vmoe_dispatch_route_bwd_dlogits(s, L.dxe, L.row_base, L.x, L.w_router, L.probs,
                                      L.expert_idx, L.slot, L.dgate, dl, L.dx, L.dw_router,
                                      L.route_bwd_ws)
    torch.cuda.synchronize()
    np.testing.assert_allclose(to_numpy(losses), ref["losses"], rtol=1e-4, atol=1e-7)
    assert_close("dlogits", to_numpy(dl), ref["dlogits"], TOL[W.F32])
    ex_dx, ex_dwr = OB.router_grad_extra(as_f64(inp["x"], cfg.dtype),
                                         as_f64(inp["w_router"], cfg.dtype), ref["dlogits"], G)
    tol = TOL[cfg.dtype]
    assert_close("dx change", to_numpy(L.dx).astype(np.float64) - to_numpy(dx0), ex_dx, tol)
    assert_close("dW_router change", to_numpy(L.dw_router).astype(np.float64) - to_numpy(dwr0),
                 ex_dwr, tol)
