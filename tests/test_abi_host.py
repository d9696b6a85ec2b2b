"""Host-side checks of the C ABI (no GPU needed, nothing is launched).

The library must load, export every entry point include/vmoe.h declares, and
reject invalid arguments with the documented status before touching the GPU.
"""
import ctypes
import subprocess

import pytest

import oracle
from paper_2608_16188_amd import vmoe as V
from paper_2608_16188_amd import workloads as W

FAKE = 0x10000  # 16-byte aligned, never dereferenced: validation fails first


def test_every_declared_symbol_is_exported():
    declared = V.header_symbols()
    assert len(declared) == 27, declared
    out = subprocess.check_output(["nm", "-D", "--defined-only", V.LIB_PATH], text=True)
    exported = {line.split()[-1] for line in out.splitlines() if line.strip()}
    missing = [s for s in declared if s not in exported]
    assert not missing, missing
    for s in declared:
        assert hasattr(V._lib, s)


def test_abi_version_and_status_strings():
    assert V.vmoe_abi_version() == 1
    assert V._lib.vmoe_status_string(0) == b"ok"
    assert V._lib.vmoe_status_string(3) == b"workspace too small"
    assert V._lib.vmoe_status_string(99) == b"unknown status"


@pytest.mark.parametrize("name", list(W.CONFIGS))
def test_capacity_matches_oracle_on_workloads(name):
    c = W.CONFIGS[name]
    for rounding in (0, 1):
        s = V.make_shape(c.n_tokens, c.n_groups, c.d_model, c.d_ff, c.n_experts, c.k,
                         c.capacity_factor, 1, capacity_rounding=rounding)
        assert V.vmoe_capacity(s) == oracle.capacity(c.n_tokens, c.n_groups, c.n_experts, c.k,
                                                     c.capacity_factor, rounding)


def test_capacity_random_shapes_and_override():
    import random
    rnd = random.Random(5)
    for _ in range(300):
        G = rnd.randint(1, 20)
        N = G * rnd.randint(0, 3000)
        E = rnd.randint(1, 64)
        k = rnd.randint(1, E)
        c = rnd.choice([0.01, 0.5, 1.0, 1.05, 1.25, 2.0, 3.3])
        s = V.make_shape(N, G, 64, 64, E, k, c, 1)
        assert V.vmoe_capacity(s) == oracle.capacity(N, G, E, k, c, 0)
    s = V.make_shape(100, 1, 64, 64, 4, 2, 1.0, 1, capacity_override=7)
    assert V.vmoe_capacity(s) == 7


@pytest.mark.parametrize("kw", [
    dict(k=0), dict(k=9), dict(n_experts=65, k=2), dict(n_tokens=10, n_groups=3),
    dict(d_model=100), dict(d_ff=12), dict(capacity_factor=0.0), dict(capacity_factor=-1.0),
    dict(capacity_factor=float("inf")), dict(dtype=2), dict(n_groups=0),
    dict(n_tokens=-8), dict(capacity_rounding=2), dict(capacity_override=-1),
])
def test_invalid_shapes_rejected(kw):
    base = dict(n_tokens=64, n_groups=1, d_model=64, d_ff=128, n_experts=8, k=2,
                capacity_factor=1.0, dtype=1)
    base.update(kw)
    s = V.make_shape(**base)
    assert V.vmoe_capacity(s) == -1
    assert V.vmoe_route_workspace_bytes(s) == 0
    st = V._lib.vmoe_dispatch(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, FAKE, None)
    assert st == V.VMOE_ERR_INVALID_ARG


def _shape():
    return V.make_shape(64, 2, 64, 128, 8, 2, 1.0, 1)


def test_null_and_misaligned_pointers_rejected():
    s = _shape()
    L = V._lib
    b = ctypes.byref(s)
    assert L.vmoe_dispatch(b, None, FAKE, FAKE, FAKE, FAKE, None) == V.VMOE_ERR_INVALID_ARG
    assert L.vmoe_dispatch(b, FAKE + 8, FAKE, FAKE, FAKE, FAKE, None) == V.VMOE_ERR_INVALID_ARG
    assert L.vmoe_combine_fwd(b, FAKE, FAKE, FAKE, None, FAKE, FAKE, None) == \
        V.VMOE_ERR_INVALID_ARG
    assert L.vmoe_combine_bwd(b, *([FAKE] * 7), None, None) == V.VMOE_ERR_INVALID_ARG
    assert L.vmoe_expert_ffn_fwd(b, *([FAKE] * 8), None, None) == V.VMOE_ERR_INVALID_ARG
    assert L.vmoe_expert_ffn_bwd(b, *([FAKE] * 12), None, None) == V.VMOE_ERR_INVALID_ARG
    assert L.vmoe_dispatch_bwd(b, FAKE, FAKE, FAKE, FAKE, None, None) == V.VMOE_ERR_INVALID_ARG
    # route: missing x without LOGITS_IN, unknown flag
    r = [FAKE] * 8
    assert L.vmoe_route(b, None, FAKE, None, None, 0, *r, FAKE, 1 << 30, None) == \
        V.VMOE_ERR_INVALID_ARG
    assert L.vmoe_route(b, FAKE, FAKE, None, None, 4, *r, FAKE, 1 << 30, None) == \
        V.VMOE_ERR_INVALID_ARG
    assert L.vmoe_route(b, FAKE, FAKE, FAKE + 4, None, 0, *r, FAKE, 1 << 30, None) == \
        V.VMOE_ERR_INVALID_ARG
    # route_bwd: missing probs
    assert L.vmoe_route_bwd(b, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30,
                            None) == V.VMOE_ERR_INVALID_ARG
    # dispatch + route backward: missing dxe, then a misaligned row_base
    assert L.vmoe_dispatch_route_bwd(b, None, *([FAKE] * 10), 1 << 30, None) == \
        V.VMOE_ERR_INVALID_ARG
    assert L.vmoe_dispatch_route_bwd(b, FAKE, FAKE + 4, *([FAKE] * 9), 1 << 30, None) == \
        V.VMOE_ERR_INVALID_ARG


def test_null_pointers_rejected_with_zero_tokens():
    """An empty batch is a valid shape, but required pointers are still
    checked: sizes never waive them."""
    s = V.make_shape(0, 1, 64, 128, 8, 2, 1.0, 1)
    assert V.vmoe_capacity(s) >= 1
    b, L = ctypes.byref(s), V._lib
    r = [FAKE] * 8
    assert L.vmoe_route(b, None, FAKE, None, None, 0, *r, FAKE, 1 << 30, None) == \
        V.VMOE_ERR_INVALID_ARG
    assert L.vmoe_dispatch(b, None, FAKE, FAKE, FAKE, FAKE, None) == V.VMOE_ERR_INVALID_ARG
    assert L.vmoe_combine_bwd(b, None, *([FAKE] * 6), FAKE, None) == V.VMOE_ERR_INVALID_ARG
    assert L.vmoe_dispatch_route_bwd(b, *([FAKE] * 7), None, FAKE, FAKE, FAKE, 1 << 30,
                                     None) == V.VMOE_ERR_INVALID_ARG


def test_balance_and_dlogits_entry_points_validate():
    b, L = ctypes.byref(_shape()), V._lib
    f = [FAKE] * 4
    # logits, bias, noise, probs, noise_std, w_imp, w_load, losses, imp, load, dlogits, ws
    ok_tail = [FAKE, None, None, FAKE, FAKE, 1 << 30, None]
    assert L.vmoe_balance_loss(b, None, None, None, FAKE, 0.1, 1.0, 1.0, *ok_tail) == \
        V.VMOE_ERR_INVALID_ARG
    assert L.vmoe_balance_loss(b, FAKE, FAKE + 4, None, FAKE, 0.1, 1.0, 1.0, *ok_tail) == \
        V.VMOE_ERR_INVALID_ARG
    for bad in (0.0, -0.5, float("inf"), float("nan")):
        assert L.vmoe_balance_loss(b, FAKE, None, None, FAKE, bad, 1.0, 1.0, *ok_tail) == \
            V.VMOE_ERR_INVALID_ARG
    assert L.vmoe_balance_loss(b, FAKE, None, None, FAKE, 0.1, float("nan"), 1.0, *ok_tail) == \
        V.VMOE_ERR_INVALID_ARG
    need = V.vmoe_balance_loss_workspace_bytes(_shape())
    assert need > 0
    assert L.vmoe_balance_loss(b, FAKE, None, None, FAKE, 0.1, 1.0, 1.0, FAKE, None, None, FAKE,
                               FAKE, need - 1, None) == V.VMOE_ERR_WORKSPACE
    # the fused backward with dlogits: a NULL dlogits is an error
    assert L.vmoe_dispatch_route_bwd_dlogits(b, *([FAKE] * 8), None, FAKE, FAKE, FAKE, 1 << 30,
                                             None) == V.VMOE_ERR_INVALID_ARG
    need_b = V.vmoe_route_bwd_workspace_bytes(_shape())
    assert L.vmoe_dispatch_route_bwd_dlogits(b, *([FAKE] * 12), need_b - 1, None) == \
        V.VMOE_ERR_WORKSPACE
    del f


def test_workspace_too_small_rejected():
    s = _shape()
    b = ctypes.byref(s)
    need = V.vmoe_route_workspace_bytes(s)
    assert need > 0
    r = [FAKE] * 8
    assert V._lib.vmoe_route(b, FAKE, FAKE, None, None, 0, *r, FAKE, need - 1, None) == \
        V.VMOE_ERR_WORKSPACE
    assert V._lib.vmoe_route(b, FAKE, FAKE, None, None, 0, *r, None, need, None) == \
        V.VMOE_ERR_WORKSPACE
    need_b = V.vmoe_route_bwd_workspace_bytes(s)
    assert need_b > 0
    assert V._lib.vmoe_route_bwd(b, *([FAKE] * 8), FAKE, need_b - 1, None) == \
        V.VMOE_ERR_WORKSPACE
    assert V._lib.vmoe_dispatch_route_bwd(b, *([FAKE] * 10), FAKE, need_b - 1, None) == \
        V.VMOE_ERR_WORKSPACE


def test_workspace_sizes_are_modest_for_workloads():
    for c in W.CONFIGS.values():
        s = V.make_shape(c.n_tokens, c.n_groups, c.d_model, c.d_ff, c.n_experts, c.k,
                         c.capacity_factor, 1)
        assert 0 < V.vmoe_route_workspace_bytes(s) < 8 << 20
        assert 0 < V.vmoe_route_bwd_workspace_bytes(s) < 64 << 20


@pytest.mark.parametrize("kw", [
    # one expert's [G*C, f] activations pass 2 GiB (bf16): 350 000 rows x 4096
    dict(n_tokens=350_000, d_model=1024, d_ff=4096, n_experts=2, k=2, capacity_factor=1.0),
    # the same rows in f32 pass it at half the width
    dict(n_tokens=300_000, d_model=1024, d_ff=2048, n_experts=2, k=2, capacity_factor=1.0,
         dtype=0),
    # every expert fits, but the pooled buffers' element index passes 2^31
    dict(n_tokens=100_000, d_model=8, d_ff=4096, n_experts=64, k=8, capacity_factor=1.0),
    # one expert's [f, d] weight passes 2 GiB
    dict(n_tokens=64, d_model=32768, d_ff=32768, n_experts=2, k=1, capacity_factor=1.0),
    # every per-expert operand fits, but a 128-token f32 chunk of dx (the
    # router backward's unit) passes 2 GiB: d = 2^22
    dict(n_tokens=4, d_model=1 << 22, d_ff=8, n_experts=17, k=1, capacity_factor=1.0),
])
def test_shapes_beyond_32bit_addressing_unsupported(kw):
    """Shapes the kernels' 32-bit buffer offsets cannot address are refused
    with VMOE_ERR_UNSUPPORTED before anything is enqueued."""
    base = dict(n_groups=1, dtype=1)
    base.update(kw)
    s = V.make_shape(**base)
    b, L = ctypes.byref(s), V._lib
    assert V.vmoe_capacity(s) == -1
    assert V.vmoe_route_workspace_bytes(s) == 0
    assert L.vmoe_dispatch(b, FAKE, FAKE, FAKE, FAKE, FAKE, None) == V.VMOE_ERR_UNSUPPORTED
    assert L.vmoe_expert_ffn_fwd(b, *([FAKE] * 9), None) == V.VMOE_ERR_UNSUPPORTED
    assert L.vmoe_expert_ffn_bwd(b, *([FAKE] * 13), None) == V.VMOE_ERR_UNSUPPORTED


def test_largest_workload_within_addressing_limits():
    for c in W.CONFIGS.values():
        s = V.make_shape(c.n_tokens, c.n_groups, c.d_model, c.d_ff, c.n_experts, c.k,
                         c.capacity_factor, 1 if c.dtype == W.BF16 else 0)
        assert V.vmoe_capacity(s) > 0


def test_route_noalloc_validates_before_touching_the_gpu():
    """The no-allocation routing call checks its arguments and that the shape's
    scratch fits the static array before any HIP call."""
    L = V._lib
    r = [FAKE] * 8
    b = ctypes.byref(_shape())
    assert L.vmoe_route_noalloc(b, None, FAKE, None, None, 0, *r, None) == \
        V.VMOE_ERR_INVALID_ARG
    assert L.vmoe_route_noalloc(b, FAKE, FAKE, None, None, 4, *r, None) == \
        V.VMOE_ERR_INVALID_ARG
    # 2M tokens need about 24 MiB of routing scratch: more than the 16 MiB array
    big = V.make_shape(2_000_000, 1, 8, 8, 8, 2, 1.0, 1)
    assert V.vmoe_route_workspace_bytes(big) > 16 << 20
    assert L.vmoe_route_noalloc(ctypes.byref(big), FAKE, FAKE, None, None, 0, *r, None) == \
        V.VMOE_ERR_WORKSPACE
    for c in W.CONFIGS.values():
        s = V.make_shape(c.n_tokens, c.n_groups, c.d_model, c.d_ff, c.n_experts, c.k,
                         c.capacity_factor, 1)
        assert V.vmoe_route_workspace_bytes(s) <= 16 << 20


def test_gathered_expert_mlp_refuses_unsupported_shapes():
    """The dispatch-fused calls run bf16 layers only, with x within one
    32-bit buffer range and (backward) at most 6144 rows per expert."""
    L = V._lib
    f32 = V.make_shape(64, 1, 64, 128, 8, 2, 1.0, V.VMOE_F32)
    assert L.vmoe_dispatch_ffn_fwd(ctypes.byref(f32), *([FAKE] * 13), None) == \
        V.VMOE_ERR_UNSUPPORTED
    assert L.vmoe_expert_ffn_bwd_gather(ctypes.byref(f32), *([FAKE] * 14), None) == \
        V.VMOE_ERR_UNSUPPORTED
    many_rows = V.make_shape(40000, 1, 64, 128, 8, 2, 1.0, V.VMOE_BF16)  # C = 10000
    assert V.vmoe_capacity(many_rows) > 6144
    assert L.vmoe_expert_ffn_bwd_gather(ctypes.byref(many_rows), *([FAKE] * 14), None) == \
        V.VMOE_ERR_UNSUPPORTED
    assert L.vmoe_dispatch_ffn_fwd(ctypes.byref(_shape()), None, *([FAKE] * 12), None) == \
        V.VMOE_ERR_INVALID_ARG
