"""A whole layer step captured in a HIP graph (GPU).

The library allocates nothing, clears its counters with kernels and never
synchronises, so one forward + backward step (every C-ABI call of the layer
on the capturing stream) can be captured and replayed. Each replay — with
the program's own eager work and a synchronisation between replays — must
reproduce the eager step bit for bit on every output (the step is
deterministic and recomputes everything from its inputs).
"""
import pytest
import torch

from paper_2608_16188_amd import workloads as W
from paper_2608_16188_amd.layer import LayerBuffers

from .gpu_common import say, workload_inputs

pytestmark = pytest.mark.gpu

OUTS = ("logits", "probs", "expert_idx", "slot", "gate", "order", "counts", "row_base", "a",
        "a_grad", "ye", "y", "dye", "dgate", "dh", "dxe", "dw1", "db1", "dw2", "db2", "dx",
        "dw_router")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _bits(t):
    t = t.detach()
    if t.dtype in (torch.bfloat16, torch.int16):
        return t.view(torch.int16).clone()
    if t.dtype == torch.float32:
        return t.view(torch.int32).clone()
    return t.clone()


# (20 experts: the expert-MLP backward forks its dxe onto the library's side
# stream and joins it back, which the capture must record as a branch)
_E20 = W.custom_config("bf16_e20_graph", n_tokens=400, d_model=96, d_ff=160, n_experts=20, k=2,
                       capacity_factor=1.0, n_groups=2, router_std=0.3)
CASES = [("vitb16_bf16", False), ("vitb16_bf16", True), ("tiny_fp32", False),
         (W.custom_config("bf16_ragged_graph", n_tokens=300, d_model=72, d_ff=200, n_experts=5,
                          k=2, capacity_factor=0.8, n_groups=3, router_std=0.2,
                          noise_var=0.1), False),
         (_E20, False), (_E20, True)]


@pytest.mark.parametrize("case,gather", CASES,
                         ids=[(c if isinstance(c, str) else c.name) + ("-gather" if g else "")
                              for c, g in CASES])
def test_step_replays_in_a_graph(case, gather):
    if isinstance(case, str):
        cfg, inp = workload_inputs(case)
    else:
        cfg, inp = case, W.make_inputs(case)
    say("graph capture", cfg.name, "gather" if gather else "")
    L = LayerBuffers(cfg, inp)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        L.step(gather=gather)  # eager, on the stream the graph is captured from
    torch.cuda.synchronize()
    outs = [n for n in OUTS if getattr(L, n) is not None]
    ref = {n: _bits(getattr(L, n)) for n in outs}
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        L.step(gather=gather)
    torch.cuda.synchronize()
    scratch = torch.empty(1 << 20, dtype=torch.float32, device="cuda")
    for rep in range(3):
        scratch.fill_(float(rep))  # the program's own eager work between replays
        for n in ("y", "dx", "dw1", "dw2"):  # the replay must rewrite these
            getattr(L, n).view(torch.uint8).fill_(0xA5)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for n in outs:
            assert torch.equal(_bits(getattr(L, n)), ref[n]), f"replay {rep}: {n} differs"
