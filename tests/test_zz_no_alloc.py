"""The no-allocation routing entry point against vmoe_route (GPU).

vmoe_route_noalloc keeps its scratch in a static per-GPU array instead of a
caller workspace; its outputs must equal vmoe_route's bit for bit. Two calls
in a row on the same array, the second with fewer tokens (and another kernel
path: the first routes in several passes, the second in one block per
group), so a result that leaned on the first call's scratch contents would
show.
"""
import numpy as np
import pytest
import torch

from paper_2608_16188_amd import vmoe as V
from paper_2608_16188_amd import workloads as W

pytestmark = pytest.mark.gpu

OUTS = ("logits", "probs", "idx", "slot", "gate", "order", "counts", "row_base")


def _buffers(N, E, k, G):
    dev, f32, i32 = "cuda", torch.float32, torch.int32
    Nb = max(N, 1)
    return dict(logits=torch.empty(Nb, E, dtype=f32, device=dev),
                probs=torch.empty(Nb, E, dtype=f32, device=dev),
                idx=torch.empty(Nb, k, dtype=i32, device=dev),
                slot=torch.empty(Nb, k, dtype=i32, device=dev),
                gate=torch.empty(Nb, k, dtype=f32, device=dev),
                order=torch.empty(Nb, dtype=i32, device=dev),
                counts=torch.empty(G, E, dtype=i32, device=dev),
                row_base=torch.empty(G, E, dtype=i32, device=dev))


def _run(noalloc, s, x, wr, bias, noise, N, E, k, G):
    o = _buffers(N, E, k, G)
    for t in o.values():
        t.fill_(-7)  # distinct garbage, so an unwritten output shows
    args = (s, x, wr, bias, noise, 0, o["logits"], o["probs"], o["idx"], o["slot"], o["gate"],
            o["order"], o["counts"], o["row_base"])
    if noalloc:
        V.vmoe_route_noalloc(*args)
    else:
        ws = torch.empty(max(V.vmoe_route_workspace_bytes(s), 16), dtype=torch.uint8,
                         device="cuda")
        V.vmoe_route(*args, ws)
    torch.cuda.synchronize()
    return {key: o[key].cpu().numpy() for key in OUTS}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def test_route_noalloc_matches_route_twice():
    cases = [  # (N, G, d, E, k, cf, noise, bias): large multi-pass, then small one-block
        (20_000, 1, 256, 16, 2, 1.0, True, True),
        (3 * 900, 3, 128, 8, 2, 0.8, False, False),
    ]
    for i, (N, G, d, E, k, cf, with_noise, with_bias) in enumerate(cases):
        print(f"[gpu-test] route_noalloc call {i}: N={N} G={G} E={E} k={k}", flush=True)
        rng = np.random.default_rng(40 + i)
        x = torch.from_numpy(W.f32_to_bf16_bits(rng.standard_normal((N, d), np.float32))
                             .view(np.int16)).view(torch.bfloat16).cuda()
        wr = torch.from_numpy(W.f32_to_bf16_bits(0.1 * rng.standard_normal((G, E, d),
                                                                          np.float32))
                              .view(np.int16)).view(torch.bfloat16).cuda()
        noise = torch.from_numpy(0.2 * rng.standard_normal((N, E), np.float32)).cuda() \
            if with_noise else None
        bias = torch.from_numpy(np.linspace(-1, 1, E).astype(np.float32)).cuda() \
            if with_bias else None
        s = V.make_shape(N, G, d, 64, E, k, cf, V.VMOE_BF16)
        ref = _run(False, s, x, wr, bias, noise, N, E, k, G)
        got = _run(True, s, x, wr, bias, noise, N, E, k, G)
        for key in OUTS:
            a, b = got[key], ref[key]
            if a.dtype == np.float32:
                a, b = a.view(np.uint32), b.view(np.uint32)
            assert np.array_equal(a, b), f"call {i}: {key} differs from vmoe_route"
