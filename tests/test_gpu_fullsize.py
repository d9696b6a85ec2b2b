"""GPU parity at full size, every element, in the benchmark's launch
configuration: the four bf16 workloads (ViT-B/16, the wide 32-expert layer,
the 17-task pool, ViT-L/16 at 384 px) run one whole layer step through the
C ABI, and every output and intermediate is compared with the oracle
(oracle/layer_full.py, float64) fed the GPU's own f32 router logits:

- routing (indices, slots, drops, order, counts, row bases, probabilities,
  gates): bit for bit;
- each expert's packed rows of xe (bit for bit), gelu(H), gelu'(H), ye,
  dye, dH and dxe; the token tensors y and dx; every expert's dW1, dW2 rows
  and db1, db2: each row within 2e-2 of that row's own largest reference
  magnitude (so a wrong row of a light expert or a single token cannot hide
  under another's scale), and the whole tensor within 2e-2;
- dgate, a dot product over d per kept assignment, element by element:
  |a - b| <= 2e-2 max(|b|, ||dy_t * ye_row||_2), the second term the size of
  its summands (a wrong element is off by about that much);
- the router gradient's rows; empty experts' gradients exactly zero.
The ViT-L/16 layer runs twice more: with the expert MLP through the
fill-clamp-refill tile scheduler (vmoe_expert_ffn_fwd_quota / _bwd_quota) and
with the dispatch fused into the expert MLP's loads (vmoe_dispatch_ffn_fwd,
vmoe_expert_ffn_bwd_gather; xe is then never written and not compared).

With VMOE_PARITY_REPORT_DIR set, each case writes its metrics (per tensor,
worst row, element-wise) there as JSON.
"""
import numpy as np
import pytest
import torch

from oracle.layer_full import layer_packed
from paper_2608_16188_amd import workloads as W
from paper_2608_16188_amd.layer import LayerBuffers, to_numpy

from .gpu_common import (TOL, Report, as_f64, assert_rows_close, assert_router_logits,
                         elementwise_rel, oracle_capacity, rel_err, say, workload_inputs)
from .test_gpu_parity import _compare_routing

pytestmark = pytest.mark.gpu

# (workload, variant of the expert MLP calls: "" the default ones, "quota" the
# fill-clamp-refill tile scheduler, "gather" the dispatch fused into the loads)
FULL = [("vitb16_bf16", ""), ("vitl16_384_bf16", ""), ("vitl16_384_bf16", "quota"),
        ("vitl16_384_bf16", "gather"), ("wide_e32_bf16", ""), ("multitask17_bf16", "")]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _rows(t, e, n, dtype):
    """Expert e's first n rows of a [E, G*C, width] device buffer as float64."""
    return W.to_f64(to_numpy(t[e, :n]), dtype) if n else np.zeros((0, t.shape[2]))


@pytest.mark.parametrize("name,variant", FULL,
                         ids=[n + ("-" + v if v else "") for n, v in FULL])
def test_layer_full_size_every_element(name, variant):
    cfg, inp = workload_inputs(name)
    say("full size, every element:", name, variant, "GPU step")
    L = LayerBuffers(cfg, inp)
    L.step(quota=variant == "quota", gather=variant == "gather")
    torch.cuda.synchronize()
    dt, tol = cfg.dtype, TOL[cfg.dtype]
    f = {key: as_f64(inp[key], dt) for key in ("x", "w_router", "w1", "b1", "w2", "b2", "dy")}
    logits = to_numpy(L.logits)
    assert_router_logits(logits, f["x"], f["w_router"], cfg.n_groups, dt)
    C = oracle_capacity(cfg)
    say(name, "oracle")
    ref = layer_packed(f["x"], f["w_router"], f["w1"], f["b1"], f["w2"], f["b2"], f["dy"],
                       k=cfg.k, C=C, n_groups=cfg.n_groups, bias=inp["logit_bias"],
                       noise=inp["noise"], logits=logits, want_dwr=not cfg.routers_frozen,
                       progress=lambda m: say(name, m))
    got_r = dict(idx=to_numpy(L.expert_idx), slot=to_numpy(L.slot), order=to_numpy(L.order),
                 counts=to_numpy(L.counts), row_base=to_numpy(L.row_base),
                 probs=to_numpy(L.probs), gate=to_numpy(L.gate))
    _compare_routing(got_r, ref, name)
    say(name, "routing bit-exact; comparing expert rows")
    rep = Report(name + ("-" + variant if variant else ""))
    n_e = ref["n_e"]
    dw1, db1, dw2, db2 = (to_numpy(t) for t in (L.dw1, L.db1, L.dw2, L.db2))
    for e in range(cfg.n_experts):
        n = int(n_e[e])
        if variant != "gather":  # the fused forward never writes xe
            assert np.array_equal(_rows(L.xe, e, n, dt), ref["xe"][e]), f"xe[{e}] not exact"
        for key, buf in (("A", L.a), ("Gd", L.a_grad), ("ye", L.ye), ("dye", L.dye),
                         ("dH", L.dh), ("dxe", L.dxe)):
            assert_rows_close(f"{key}", _rows(buf, e, n, dt), ref[key][e], tol, rep)
        if n == 0:
            for g_ in (dw1[e], db1[e], dw2[e], db2[e]):
                assert np.all(g_ == 0.0), f"expert {e} has no rows: gradients must be 0"
            continue
        assert_rows_close("dW1", dw1[e], ref["dw1"][e], tol, rep, block=32)
        assert_rows_close("dW2", dw2[e], ref["dw2"][e], tol, rep, block=32)
        assert_rows_close("db1", db1[e][None], ref["db1"][e][None], tol, rep)
        assert_rows_close("db2", db2[e][None], ref["db2"][e][None], tol, rep)
    say(name, "comparing token tensors")
    assert_rows_close("y", W.to_f64(to_numpy(L.y), dt), ref["y"], tol, rep)
    assert_rows_close("dx", to_numpy(L.dx), ref["dx"], tol, rep)
    if not cfg.routers_frozen:
        got_wr = to_numpy(L.dw_router)
        assert_rows_close("dW_router", got_wr.reshape(-1, got_wr.shape[-1]),
                          ref["dw_router"].reshape(-1, got_wr.shape[-1]), tol, rep)
    # dgate: each kept assignment's dot product against the size of its terms
    dg, dg_ref = to_numpy(L.dgate).astype(np.float64), ref["dgate"]
    kept = ref["slot"] >= 0
    assert np.all(dg[~kept] == 0.0), "dropped assignments must have dgate 0"
    ng = cfg.n_tokens // cfg.n_groups
    mag = np.zeros_like(dg_ref)
    for e in range(cfg.n_experts):
        t, j = np.nonzero((ref["idx"] == e) & kept)
        rows = ref["row_base"][t // ng, e] + ref["slot"][t, j]
        mag[t, j] = np.sqrt(np.sum((f["dy"][t] * ref["ye"][e][rows]) ** 2, axis=1))
    err = np.abs(dg - dg_ref)
    bound = tol * np.maximum(np.abs(dg_ref), mag)
    rep.add("dgate", rel_err(dg, dg_ref), float(np.max(err / np.maximum(bound, 1e-300)) * tol),
            elementwise_rel(dg, dg_ref))
    rep.write()
    assert np.all(err <= bound), f"dgate: {int(np.sum(err > bound))} elements off"
    assert rel_err(dg, dg_ref) <= tol
