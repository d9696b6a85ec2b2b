"""The fill-clamp-refill tile scheduler of the expert GEMMs (GPU).

- The device routine's whole-unit shares equal the host routine's
  (vmoe_fill_clamp_refill, itself pinned to the water-filling form by the
  aligning tests) for random inputs and edge cases.
- The quota-scheduled expert MLP forward and backward give bit-identical
  outputs to the default scheduling (every output tile is computed by the
  same code, whichever workgroup takes it), on small layers and at the
  ViT-L/16 skew (4 experts full, 28 with a few rows each), and the
  ViT-L/16 layer with the quota scheduler matches the oracle element by
  element (the full-size test's checks, run on its outputs).
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_2608_16188_amd import vmoe as V
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


def _host_units(m, s, c, budget):
    n = len(m)
    alloc = np.zeros(max(n, 1))
    units = np.zeros(max(n, 1), np.int32)
    rounds = ctypes.c_int32(0)
    ws = np.zeros(max(4 * n, 4), np.uint8)
    mi, si = np.ascontiguousarray(m, np.int32), np.ascontiguousarray(s, np.int32)
    ci = np.ascontiguousarray(c, np.float64)
    st = V._lib.vmoe_fill_clamp_refill(
        n, mi.ctypes.data_as(ctypes.c_void_p), si.ctypes.data_as(ctypes.c_void_p),
        ci.ctypes.data_as(ctypes.c_void_p), ctypes.c_int64(budget),
        alloc.ctypes.data_as(ctypes.c_void_p), units.ctypes.data_as(ctypes.c_void_p),
        ctypes.byref(rounds), ws.ctypes.data_as(ctypes.c_void_p), ctypes.c_size_t(ws.size))
    assert st == 0
    return units[:n]


def _device_units(m, s, c, budget):
    n = len(m)
    dm = torch.tensor(np.asarray(m, np.int32), device="cuda")
    ds = torch.tensor(np.asarray(s, np.int32), device="cuda")
    dc = torch.tensor(np.asarray(c, np.float64), device="cuda")
    du = torch.full((max(n, 1),), -1, dtype=torch.int32, device="cuda")
    V.vmoe_fill_clamp_refill_device(n, dm, ds, dc, budget, du)
    torch.cuda.synchronize()
    return du[:n].cpu().numpy()


def test_device_fill_clamp_refill_equals_host():
    rng = np.random.default_rng(3)
    cases = [([1] * 4, [10] * 4, [1.0, 2.0, 3.0, 4.0], 20),      # nothing saturates
             ([1] * 4, [2, 50, 50, 50], [100.0, 1.0, 1.0, 1.0], 40),  # clamp and refill
             ([0, 1, 1], [0, 3, 3], [0.0, 1.0, 1.0], 100),      # budget beyond saturation
             ([1, 1], [5, 5], [0.0, 0.0], 7),                   # no work: minima only
             ([1] * 3, [9] * 3, [1.0, 1.0, 1.0], 10)]           # equal fractions, ties
    for n in (1, 5, 17, 32, 64):
        for _ in range(6):
            m = rng.integers(0, 3, n)
            s = m + rng.integers(0, 40, n)
            c = rng.random(n) * rng.choice([0.0, 1.0, 1e3], n)
            budget = int(m.sum() + rng.integers(0, 300))
            cases.append((m, s, c, budget))
    # the GEMMs' own shape of input: 4 heavy and 28 light experts over 256 units
    tiles = np.array([160] * 4 + [16] * 28)
    cases.append(([1] * 32, tiles, tiles * np.array([2.0] * 4 + [1.07] * 28), 256))
    for m, s, c, budget in cases:
        assert np.array_equal(_device_units(m, s, c, budget), _host_units(m, s, c, budget)), \
            (m, s, c, budget)


QUOTA_SMALL = [
    W.custom_config("bf16_ragged_q", n_tokens=300, d_model=72, d_ff=200, n_experts=5, k=2,
                    capacity_factor=0.8, n_groups=3, router_std=0.2, noise_var=0.1),
    W.custom_config("bf16_hot_empty_q", n_tokens=256, d_model=128, d_ff=384, n_experts=8, k=2,
                    capacity_factor=1.0, hot_experts=2, hot_offset=6.0),
    W.custom_config("bf16_ten_mtiles_q", n_tokens=2400, d_model=72, d_ff=264, n_experts=2, k=2,
                    capacity_factor=1.0, router_std=0.05),
    W.custom_config("bf16_light_tails_q", n_tokens=2240, d_model=200, d_ff=520, n_experts=16,
                    k=2, capacity_factor=1.0, hot_experts=2, hot_offset=0.8),
]
OUTS = ("a", "a_grad", "ye", "y", "dye", "dgate", "dh", "dxe", "dw1", "db1", "dw2", "db2", "dx")


def _bits(t):
    t = t.detach()
    return (t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)).cpu()


@pytest.mark.parametrize("case", QUOTA_SMALL + ["vitl16_384_bf16", "vitb16_bf16"],
                         ids=lambda c: c if isinstance(c, str) else c.name)
def test_quota_schedule_bit_identical(case):
    if isinstance(case, str):
        cfg, inp = workload_inputs(case)
    else:
        cfg, inp = case, W.make_inputs(case)
    say("quota vs default schedule", cfg.name)
    L = LayerBuffers(cfg, inp)
    L.step()
    torch.cuda.synchronize()
    ref = {n: _bits(getattr(L, n)) for n in OUTS}
    for n in OUTS:
        getattr(L, n).fill_(float("nan"))
    L.step(quota=True)
    torch.cuda.synchronize()
    n_e = L.counts.sum(0).cpu().numpy()
    for n in OUTS:
        got = _bits(getattr(L, n))
        if n in ("a", "a_grad", "ye", "dye", "dh", "dxe"):
            for e, ne in enumerate(n_e):  # rows past n_e are never written
                assert torch.equal(got[e, :ne], ref[n][e, :ne]), f"{n}[{e}] differs"
        else:
            assert torch.equal(got, ref[n]), f"{n} differs"
