"""Pins of the CPU oracle against facts fixed outside it (CPU only).

Each test checks the oracle against something it does not share code with:
closed forms, invariants, a second formulation, brute force on tiny inputs,
a hand-worked example (tests/golden/), numpy / torch library routines on the
CPU in float64, and central finite differences.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2608_16188_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ------------------------------------------------------------------ exp_spec

def test_exp_spec_within_two_ulp_of_exp():
    u = np.concatenate([np.linspace(-87.0, 0.0, 200001), np.linspace(0.0, 88.0, 20001),
                        -np.logspace(-30, 1.9, 5001)]).astype(np.float32)
    got = oracle.exp_spec(u).astype(np.float64)
    ref = np.exp(u.astype(np.float64))
    ulp = np.spacing(ref.astype(np.float32)).astype(np.float64)
    assert np.max(np.abs(got - ref) / ulp) <= 2.0


def test_exp_spec_special_values():
    assert oracle.exp_spec(np.array([0.0]))[0] == 1.0
    assert oracle.exp_spec(np.array([-0.0]))[0] == 1.0
    # flush: results below the smallest normal are zero, never denormal
    low = oracle.exp_spec(np.array([-87.0001, -100.0, -1e30], np.float32))
    assert np.all(low == 0.0)
    v = oracle.exp_spec(np.linspace(-87.0, -80.0, 1001).astype(np.float32))
    assert np.all(v >= np.finfo(np.float32).tiny)
    # monotone non-decreasing over a dense sweep
    s = oracle.exp_spec(np.linspace(-20.0, 0.0, 100001).astype(np.float32))
    assert np.all(np.diff(s) >= 0)


# ------------------------------------------------------------------ capacity

@pytest.mark.parametrize("N,G,E,k,c,expect_round,expect_ceil", [
    (788, 1, 8, 2, 1.25, 246, 247),       # 2*788*1.25/8  = 246.25
    (6304, 1, 8, 2, 1.05, 1655, 1655),    # 2*6304*1.05/8 = 1654.8
    (25216, 1, 32, 2, 1.0, 1576, 1576),   # 2*25216/32    = 1576
    (26792, 17, 16, 2, 1.25, 246, 247),   # 2*1576*1.25/16 = 246.25
    (36928, 1, 32, 2, 1.05, 2423, 2424),  # 2*36928*1.05/32 = 2423.4
    (10, 1, 8, 1, 0.1, 1, 1),             # 0.125 -> at least one slot
    (4, 1, 8, 1, 1.0, 1, 1),              # 0.5 rounds half away from zero
])
def test_capacity_hand_values(N, G, E, k, c, expect_round, expect_ceil):
    assert oracle.capacity(N, G, E, k, c, 0) == expect_round
    assert oracle.capacity(N, G, E, k, c, 1) == expect_ceil


# ------------------------------------------------------------------ router

def test_router_logits_match_float64_matmul():
    cfg = W.custom_config(n_tokens=96, d_model=64, d_ff=64, n_experts=8, k=2,
                          capacity_factor=1.0, n_groups=3, router_std=0.1)
    inp = W.make_inputs(cfg, with_grad=False)
    x, wr = W.to_f64(inp["x"], cfg.dtype), W.to_f64(inp["w_router"], cfg.dtype)
    got = oracle.router_logits(x, wr, cfg.n_groups)
    ref = np.concatenate([x[g * 32:(g + 1) * 32] @ wr[g].T for g in range(3)])
    # Sum of exact products in double: rounding to f32 agrees to within half an f32 ulp.
    assert np.all(np.abs(got - ref) <= 0.5 * np.spacing(np.abs(got)) + 1e-30)


# ------------------------------------------------------------------ gate

def test_gate_softmax_priority_and_sum():
    z = W.random_logits(500, 16, seed=3, scale=3.0)
    noise = W.random_logits(500, 16, seed=4, scale=0.25)
    bias = np.linspace(-1, 1, 16).astype(np.float32)
    g = oracle.gate(z, 3, bias=bias, noise=noise)
    zz = (z + bias) + noise  # float32 arithmetic, same order
    assert np.array_equal(g["z"], zz)
    ref = np.exp(zz.astype(np.float64) - zz.max(1, keepdims=True))
    ref /= ref.sum(1, keepdims=True)
    assert np.max(np.abs(g["probs"] - ref) / ref) < 2e-6
    assert np.all(np.abs(g["probs"].astype(np.float64).sum(1) - 1.0) <= 16 * 2**-24)
    assert np.array_equal(g["prio"], g["probs"].max(1))
    assert np.array_equal(g["prio"], g["probs"][np.arange(500), g["idx"][:, 0]])


@pytest.mark.parametrize("E", [1, 2, 3, 5, 6])
def test_topk_brute_force(E):
    for k in range(1, E + 1):
        z = W.random_logits(32, E, seed=10 + E * 7 + k, tie_every=3)
        g = oracle.gate(z, k)
        for t in range(32):
            # best ordered k-tuple of distinct experts: larger z first, ties to lower e
            best = max(itertools.permutations(range(E), k),
                       key=lambda tup: tuple(v for e in tup for v in (z[t, e], -e)))
            assert tuple(g["idx"][t]) == best


# ------------------------------------------------------------------ BPR

def _bpr_second_formulation(idx, prio, G, E, C):
    """slot of (t, r) = number of same-expert assignments processed before it,
    if that number is below C (then all of them were kept), else dropped."""
    N, k = idx.shape
    ng = N // G
    slot = np.full((N, k), -1, np.int64)
    for g in range(G):
        toks = list(range(g * ng, (g + 1) * ng))
        pos = {t: i for i, t in enumerate(sorted(toks, key=lambda t: (-prio[t], t)))}
        for t in toks:
            for r in range(k):
                e = idx[t, r]
                before = sum(1 for t2 in toks for r2 in range(k)
                             if idx[t2, r2] == e and (r2 < r or (r2 == r and pos[t2] < pos[t])))
                slot[t, r] = before if before < C else -1
    return slot


@pytest.mark.parametrize("seed,N,G,E,k,C,ties", [
    (0, 40, 1, 4, 2, 6, 0), (1, 60, 3, 5, 2, 3, 2), (2, 48, 2, 3, 3, 5, 3),
    (3, 30, 1, 6, 1, 2, 0), (4, 24, 4, 4, 4, 1, 2), (5, 36, 1, 8, 2, 100, 0),
])
def test_bpr_matches_second_formulation(seed, N, G, E, k, C, ties):
    z = W.random_logits(N, E, seed=seed, tie_every=ties)
    r = oracle.route(z, k, C, n_groups=G)
    assert np.array_equal(r["slot"], _bpr_second_formulation(r["idx"], r["prio"], G, E, C))
    ng = N // G
    for g in range(G):
        lex = np.lexsort((np.arange(ng), -r["prio"][g * ng:(g + 1) * ng].astype(np.float64)))
        assert np.array_equal(r["order"][g * ng:(g + 1) * ng], lex + g * ng)


def _check_bpr_invariants(r, G, E, k, C):
    idx, slot, prio, gate, probs = r["idx"], r["slot"], r["prio"], r["gate"], r["probs"]
    N = idx.shape[0]
    ng = N // G
    for g in range(G):
        sl = slice(g * ng, (g + 1) * ng)
        demand = np.array([(idx[sl] == e).sum() for e in range(E)])
        assert np.array_equal(r["counts"][g], np.minimum(C, demand))
        for e in range(E):
            kept_slots = np.sort(slot[sl][(idx[sl] == e) & (slot[sl] >= 0)])
            assert np.array_equal(kept_slots, np.arange(len(kept_slots)))  # slots 0..n-1, no gaps
            for rr in range(k):
                m = idx[sl][:, rr] == e
                kept = m & (slot[sl][:, rr] >= 0)
                dropped = m & (slot[sl][:, rr] < 0)
                if kept.any() and dropped.any():
                    assert prio[sl][dropped].max() <= prio[sl][kept].min()
                if dropped.any() and rr + 1 < k:
                    assert np.all(slot[sl][:, rr + 1][idx[sl][:, rr + 1] == e] < 0)
    assert np.all(r["counts"] <= C)
    kept = slot >= 0
    pk = np.take_along_axis(probs, idx, 1)
    assert np.array_equal(gate, np.where(kept, pk, 0.0).astype(np.float32))
    assert np.array_equal(r["row_base"], np.cumsum(r["counts"], 0) - r["counts"])


@pytest.mark.parametrize("name", ["tiny_fp32", "vitb16_bf16", "multitask17_bf16"])
def test_bpr_invariants_on_workloads(name):
    cfg = W.CONFIGS[name]
    inp = W.make_inputs(cfg, with_grad=False)
    # logits drawn directly (the full router product is tested elsewhere)
    z = W.random_logits(cfg.n_tokens, cfg.n_experts, seed=cfg.cid, scale=2.0)
    C = oracle.capacity(cfg.n_tokens, cfg.n_groups, cfg.n_experts, cfg.k, cfg.capacity_factor)
    r = oracle.route(z, cfg.k, C, cfg.n_groups, inp["logit_bias"], inp["noise"])
    _check_bpr_invariants(r, cfg.n_groups, cfg.n_experts, cfg.k, C)


def test_bpr_invariants_heavy_drops_and_ties():
    z = W.random_logits(400, 6, seed=77, tie_every=2)
    z[:, 0] += 3.0  # most first choices hit expert 0
    r = oracle.route(z, 3, 10, n_groups=2)
    _check_bpr_invariants(r, 2, 6, 3, 10)
    assert (r["slot"] < 0).sum() > 200


def test_bpr_hand_worked_example():
    ex = json.load(open(os.path.join(GOLDEN, "bpr_hand_example.json")))
    r = oracle.bpr(np.array(ex["probs"], np.float32), np.array(ex["idx"]),
                   np.array(ex["prio"], np.float32), 1, ex["C"])
    assert r["order"].tolist() == ex["expected_order"]
    assert r["slot"].tolist() == ex["expected_slot"]
    assert r["counts"].tolist() == ex["expected_counts"]
    assert np.array_equal(r["gate"], np.array(ex["expected_gate"], np.float32))


def test_all_equal_logits_closed_form():
    N, E, k, C = 50, 5, 2, 7
    r = oracle.route(np.zeros((N, E), np.float32), k, C)
    assert np.all(r["probs"] == np.float32(1.0) / np.float32(E))
    assert np.all(r["idx"] == np.arange(k))
    assert np.array_equal(r["order"], np.arange(N))
    exp_slot = np.full((N, k), -1)
    exp_slot[:C, 0] = np.arange(C)  # expert 0 keeps the first C tokens' first choices
    exp_slot[:C, 1] = np.arange(C)  # expert 1 only sees second choices
    assert np.array_equal(r["slot"], exp_slot)
    assert r["counts"].tolist() == [[C, C, 0, 0, 0]]


# ------------------------------------------------------------------ dispatch / combine

def test_identity_experts_combine_closed_form():
    N, d, E, k, G = 60, 24, 5, 2, 2
    z = W.random_logits(N, E, seed=5)
    C = 7
    r = oracle.route(z, k, C, n_groups=G)
    x = np.random.default_rng(0).standard_normal((N, d))
    xe = oracle.dispatch(x, r["idx"], r["slot"], r["row_base"], E, C, G)
    n_e = r["counts"].sum(0)
    for e in range(E):  # packed rows: exactly n_e filled, rest untouched
        assert not np.isnan(xe[e, :n_e[e]]).any()
        assert np.isnan(xe[e, n_e[e]:]).all()
    y = oracle.combine_fwd(np.nan_to_num(xe), r["idx"], r["slot"], r["row_base"], r["gate"], N, C,
                           G)
    wsum = r["gate"].astype(np.float64).sum(1)
    assert np.allclose(y, wsum[:, None] * x, rtol=1e-14, atol=1e-14)
    dx = oracle.dispatch_bwd(np.nan_to_num(xe), r["idx"], r["slot"], r["row_base"], N, C, G)
    nk = (r["slot"] >= 0).sum(1)
    assert np.allclose(dx, nk[:, None] * x, rtol=1e-14, atol=1e-14)


# ------------------------------------------------------------------ whole layer vs torch

def _torch_layer(x, wr, w1, b1, w2, b2, idx, kept, G, bias=None, noise=None):
    """Dense masked formulation with routing decisions frozen (float64, CPU)."""
    N = x.shape[0]
    ng = N // G
    logits = torch.cat([x[g * ng:(g + 1) * ng] @ wr[g].T for g in range(G)])
    zz = logits
    if bias is not None:
        zz = zz + bias
    if noise is not None:
        zz = zz + noise
    p = torch.softmax(zz, dim=-1)
    y = torch.zeros_like(x)
    for j in range(idx.shape[1]):
        e = idx[:, j]
        h = torch.bmm(w1[e], x.unsqueeze(2)).squeeze(2) + b1[e]
        a = torch.nn.functional.gelu(h)
        o = torch.bmm(w2[e], a.unsqueeze(2)).squeeze(2) + b2[e]
        gj = p.gather(1, e[:, None]).squeeze(1) * kept[:, j]
        y = y + gj[:, None] * o
    return y


@pytest.mark.parametrize("G,c,noise", [(1, 0.6, False), (2, 1.0, True), (1, 4.0, True)])
def test_layer_forward_backward_vs_torch_autograd(G, c, noise):
    cfg = W.custom_config(n_tokens=48, d_model=16, d_ff=24, n_experts=4, k=2, capacity_factor=c,
                          n_groups=G, router_std=0.3, weight_std=0.3, dtype=W.F32,
                          noise_var=0.25 if noise else 0.0)
    inp = W.make_inputs(cfg)
    f64 = {k_: (None if v is None else v.astype(np.float64)) for k_, v in inp.items()}
    C = oracle.capacity(cfg.n_tokens, G, cfg.n_experts, cfg.k, c)
    o = oracle.layer(f64["x"], f64["w_router"], f64["w1"], f64["b1"], f64["w2"], f64["b2"],
                     f64["dy"], k=cfg.k, C=C, n_groups=G, noise=inp["noise"])
    if c < 1.0:
        assert (o["slot"] < 0).any()
    if c >= 4.0:
        assert (o["slot"] >= 0).all()
    T = {k_: (None if v is None else torch.tensor(v, requires_grad=True)) for k_, v in f64.items()}
    kept = torch.tensor((o["slot"] >= 0).astype(np.float64))
    y = _torch_layer(T["x"], T["w_router"], T["w1"], T["b1"], T["w2"], T["b2"],
                     torch.tensor(o["idx"].astype(np.int64)), kept, G, noise=T["noise"])
    (y * T["dy"]).sum().backward()

    def close(a, b, tol):
        b = b.detach().numpy() if torch.is_tensor(b) else b
        assert np.max(np.abs(a - b)) <= tol * max(np.max(np.abs(b)), 1e-30)

    close(o["y"], y, 1e-6)
    close(o["dx"], T["x"].grad, 1e-6)
    close(o["dw_router"], T["w_router"].grad, 1e-5)
    close(o["dw1"], T["w1"].grad, 1e-6)
    close(o["db1"], T["b1"].grad, 1e-6)
    close(o["dw2"], T["w2"].grad, 1e-6)
    close(o["db2"], T["b2"].grad, 1e-6)


def test_single_expert_layer_is_plain_mlp():
    cfg = W.custom_config(n_tokens=20, d_model=12, d_ff=20, n_experts=1, k=1, capacity_factor=1.0,
                          dtype=W.F32, weight_std=0.4)
    inp = W.make_inputs(cfg)
    f = {k_: (None if v is None else v.astype(np.float64)) for k_, v in inp.items()}
    o = oracle.layer(f["x"], f["w_router"], f["w1"], f["b1"], f["w2"], f["b2"], f["dy"], k=1,
                     C=oracle.capacity(20, 1, 1, 1, 1.0))
    F = torch.nn.functional
    x = torch.tensor(f["x"], requires_grad=True)
    w1 = torch.tensor(f["w1"][0], requires_grad=True)
    w2 = torch.tensor(f["w2"][0], requires_grad=True)
    y = F.linear(F.gelu(F.linear(x, w1, torch.tensor(f["b1"][0]))), w2, torch.tensor(f["b2"][0]))
    (y * torch.tensor(f["dy"])).sum().backward()
    assert np.allclose(o["y"], y.detach().numpy(), rtol=1e-12, atol=1e-12)
    assert np.allclose(o["dx"], x.grad.numpy(), rtol=1e-10, atol=1e-12)
    assert np.allclose(o["dw1"][0], w1.grad.numpy(), rtol=1e-10, atol=1e-12)
    assert np.allclose(o["dw2"][0], w2.grad.numpy(), rtol=1e-10, atol=1e-12)
    assert np.all(o["dz"] == 0.0)


def test_expert_mlp_gradients_central_differences():
    rng = np.random.default_rng(9)
    rows, d, f = 5, 6, 7
    xe = rng.standard_normal((rows, d))
    w1, b1 = rng.standard_normal((f, d)) * 0.5, rng.standard_normal(f) * 0.5
    w2, b2 = rng.standard_normal((d, f)) * 0.5, rng.standard_normal(d) * 0.5
    dye = rng.standard_normal((rows, d))

    def loss(xe_, w1_, b1_, w2_, b2_):
        return float((oracle.ffn_fwd(xe_, w1_, b1_, w2_, b2_)[2] * dye).sum())

    dw1, db1, dw2, db2 = oracle.ffn_bwd_weights(xe, w1, b1, w2, dye)
    dxe, _ = oracle.ffn_bwd_rows(xe, w1, b1, w2, dye)
    h = 1e-6
    for name, arr, grad in [("xe", xe, dxe), ("w1", w1, dw1), ("b1", b1, db1), ("w2", w2, dw2),
                            ("b2", b2, db2)]:
        for flat in range(0, arr.size, 3):
            args = dict(xe_=xe, w1_=w1, b1_=b1, w2_=w2, b2_=b2)
            plus, minus = arr.copy(), arr.copy()
            plus.flat[flat] += h
            minus.flat[flat] -= h
            args[name + "_"] = plus
            lp = loss(**args)
            args[name + "_"] = minus
            lm = loss(**args)
            assert abs((lp - lm) / (2 * h) - grad.flat[flat]) < 1e-6, (name, flat)


def test_weight_entries_equal_full_gradients():
    rng = np.random.default_rng(2)
    rows, d, f = 9, 8, 12
    xe, w1, b1 = rng.standard_normal((rows, d)), rng.standard_normal((f, d)), rng.standard_normal(f)
    w2, dye = rng.standard_normal((d, f)), rng.standard_normal((rows, d))
    dw1, db1, dw2, db2 = oracle.ffn_bwd_weights(xe, w1, b1, w2, dye)
    which = [1, 1, 2, 2, 3, 4]
    row = [3, 11, 0, 7, 5, 6]
    col = [2, 7, 11, 3, 0, 0]
    got = oracle.ffn_bwd_weight_entries(xe, w1, b1, w2, dye, which, row, col)
    ref = [dw1[3, 2], dw1[11, 7], dw2[0, 11], dw2[7, 3], db1[5], db2[6]]
    assert np.allclose(got, ref, rtol=1e-13, atol=1e-13)
    z = oracle.ffn_bwd_weights(xe[:0], w1, b1, w2, dye[:0])
    assert all(np.all(a == 0.0) for a in z)


def test_multitask_pool_load_follows_zipf():
    """The 17-task workload's pooled top-1 load fits Zipf with s close to 1.2."""
    import importlib.util
    spec = importlib.util.spec_from_file_location(
        "fit_gamma", os.path.join(GOLDEN, "fit_multitask_gamma.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    s = mod.zipf_exponent(W.CONFIGS["multitask17_bf16"])
    assert abs(s - 1.2) < 0.01


def test_ffn_forward_saved_gelu_derivative_matches_autograd():
    rng = np.random.default_rng(4)
    rows, d, f = 7, 10, 13
    xe, w1, b1 = rng.standard_normal((rows, d)), rng.standard_normal((f, d)), rng.standard_normal(f)
    w2, b2 = rng.standard_normal((d, f)), rng.standard_normal(d)
    H, A, G, ye = oracle.ffn_fwd(xe, w1, b1, w2, b2, with_grad=True)
    h = torch.tensor(H, requires_grad=True)
    torch.nn.functional.gelu(h).sum().backward()
    assert np.allclose(G, h.grad.numpy(), rtol=1e-12, atol=1e-14)
    assert np.allclose(A, torch.nn.functional.gelu(torch.tensor(H)).numpy(), rtol=1e-12, atol=1e-14)
