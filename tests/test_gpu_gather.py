"""The dispatch fused into the expert MLP's operand loads (GPU).

vmoe_dispatch_ffn_fwd reads each expert row from the token's row of x and
never writes xe; vmoe_expert_ffn_bwd_gather reads xe's rows the same way for
the input-weight gradient. The same bf16 values reach the same products, so
every output must equal the unfused step's bit for bit; row_token must name
each kept row's token (the dispatch's permutation).
"""
import numpy as np
import pytest
import torch

from paper_2608_16188_amd import workloads as W
from paper_2608_16188_amd.layer import LayerBuffers

from .gpu_common import say, workload_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


CASES = [
    W.custom_config("bf16_ragged_g", n_tokens=300, d_model=72, d_ff=200, n_experts=5, k=2,
                    capacity_factor=0.8, n_groups=3, router_std=0.2, noise_var=0.1),
    W.custom_config("bf16_hot_empty_g", n_tokens=256, d_model=128, d_ff=384, n_experts=8, k=2,
                    capacity_factor=1.0, hot_experts=2, hot_offset=6.0),
    W.custom_config("bf16_k4_e20_g", n_tokens=400, d_model=96, d_ff=160, n_experts=20, k=4,
                    capacity_factor=1.0, n_groups=2, router_std=0.3),
    W.custom_config("bf16_ten_mtiles_g", n_tokens=2400, d_model=72, d_ff=264, n_experts=2, k=2,
                    capacity_factor=1.0, router_std=0.05),
    W.custom_config("bf16_light_tails_g", n_tokens=2240, d_model=200, d_ff=520, n_experts=16,
                    k=2, capacity_factor=1.0, hot_experts=2, hot_offset=0.8),
]
OUTS = ("a", "a_grad", "ye", "y", "dye", "dgate", "dh", "dxe", "dw1", "db1", "dw2", "db2", "dx",
        "dw_router")


def _bits(t):
    t = t.detach()
    return (t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)).cpu()


@pytest.mark.parametrize("case", CASES + ["vitb16_bf16", "vitl16_384_bf16", "multitask17_bf16"],
                         ids=lambda c: c if isinstance(c, str) else c.name)
def test_gathered_step_bit_identical(case):
    if isinstance(case, str):
        cfg, inp = workload_inputs(case)
    else:
        cfg, inp = case, W.make_inputs(case)
    say("gathered vs unfused step", cfg.name)
    L = LayerBuffers(cfg, inp)
    L.step()
    torch.cuda.synchronize()
    outs = [n for n in OUTS if getattr(L, n) is not None]
    ref = {n: _bits(getattr(L, n)) for n in outs}
    for n in outs:
        getattr(L, n).fill_(float("nan"))
    L.row_token.fill_(-7)
    L.step(gather=True)
    torch.cuda.synchronize()
    n_e = L.counts.sum(0).cpu().numpy()
    for n in outs:
        got = _bits(getattr(L, n))
        if n in ("a", "a_grad", "ye", "dye", "dh", "dxe"):
            for e, ne in enumerate(n_e):  # rows past n_e are never written
                assert torch.equal(got[e, :ne], ref[n][e, :ne]), f"{n}[{e}] differs"
        else:
            assert torch.equal(got, ref[n]), f"{n} differs"
    # row_token is the dispatch's permutation: row(t, j) holds token t
    idx, slot = L.expert_idx.cpu().numpy(), L.slot.cpu().numpy()
    rb, tok = L.row_base.cpu().numpy(), L.row_token.cpu().numpy()
    ng = cfg.n_tokens // cfg.n_groups
    t, j = np.nonzero(slot >= 0)
    e = idx[t, j]
    rows = rb[t // ng, e] + slot[t, j]
    assert np.array_equal(tok[e, rows], t)
