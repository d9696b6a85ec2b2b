"""Python binding of libvmoe (ctypes; argument marshalling only).

Every function has the name of the C entry point it calls and takes torch
device tensors (or None for optional pointers); every step of the layer runs
in the HIP kernels of libvmoe.so. torch is used for device memory and
streams only. There is no CPU fallback: if the library is missing this
module raises at import time.
"""
from __future__ import annotations

import ctypes
import os
import re

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libvmoe.so")
HEADER = os.path.join(os.path.dirname(_PKG), "include", "vmoe.h")

VMOE_OK, VMOE_ERR_INVALID_ARG, VMOE_ERR_UNSUPPORTED, VMOE_ERR_WORKSPACE, VMOE_ERR_HIP = range(5)
VMOE_F32, VMOE_BF16 = 0, 1
VMOE_ROUTE_LOGITS_IN = 1


class VmoeError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__(f"{fn} failed: {status} ({_lib.vmoe_status_string(status).decode()})")


class Shape(ctypes.Structure):
    _fields_ = [
        ("n_tokens", ctypes.c_int32), ("n_groups", ctypes.c_int32),
        ("d_model", ctypes.c_int32), ("d_ff", ctypes.c_int32),
        ("n_experts", ctypes.c_int32), ("k", ctypes.c_int32),
        ("capacity_factor", ctypes.c_double), ("capacity_rounding", ctypes.c_int32),
        ("capacity_override", ctypes.c_int32), ("dtype", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
    ]


def make_shape(n_tokens, n_groups, d_model, d_ff, n_experts, k, capacity_factor, dtype,
               capacity_rounding=0, capacity_override=0) -> Shape:
    return Shape(n_tokens, n_groups, d_model, d_ff, n_experts, k, float(capacity_factor),
                 capacity_rounding, capacity_override, dtype, 0)


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built: run `python -m paper_2608_16188_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    S = ctypes.POINTER(Shape)
    lib.vmoe_abi_version.restype = ctypes.c_int32
    lib.vmoe_status_string.restype = ctypes.c_char_p
    lib.vmoe_status_string.argtypes = [ctypes.c_int32]
    lib.vmoe_capacity.restype = ctypes.c_int32
    lib.vmoe_capacity.argtypes = [S]
    for name in ("vmoe_route_workspace_bytes", "vmoe_route_bwd_workspace_bytes",
                 "vmoe_balance_loss_workspace_bytes"):
        getattr(lib, name).restype = ctypes.c_size_t
        getattr(lib, name).argtypes = [S]
    sigs = {
        "vmoe_route": [S, P, P, P, P, ctypes.c_int32] + [P] * 8 + [P, ctypes.c_size_t, P],
        "vmoe_route_noalloc": [S, P, P, P, P, ctypes.c_int32] + [P] * 8 + [P],
        "vmoe_dispatch": [S] + [P] * 6,
        "vmoe_expert_ffn_fwd": [S] + [P] * 10,
        "vmoe_expert_ffn_fwd_quota": [S] + [P] * 10,
        "vmoe_dispatch_ffn_fwd": [S] + [P] * 14,
        "vmoe_expert_ffn_bwd_gather": [S] + [P] * 15,
        "vmoe_expert_ffn_bwd_quota": [S] + [P] * 14,
        "vmoe_fill_clamp_refill_device": [ctypes.c_int32, P, P, P, ctypes.c_int32, P, P],
        "vmoe_combine_fwd": [S] + [P] * 7,
        "vmoe_combine_bwd": [S] + [P] * 9,
        "vmoe_expert_ffn_bwd": [S] + [P] * 14,
        "vmoe_dispatch_bwd": [S] + [P] * 6,
        "vmoe_route_bwd": [S] + [P] * 9 + [ctypes.c_size_t, P],
        "vmoe_dispatch_route_bwd": [S] + [P] * 11 + [ctypes.c_size_t, P],
        "vmoe_dispatch_route_bwd_dlogits": [S] + [P] * 12 + [ctypes.c_size_t, P],
        "vmoe_balance_loss": [S] + [P] * 4 + [ctypes.c_float] * 3 + [P] * 5 + [ctypes.c_size_t, P],
    }
    for name, args in sigs.items():
        f = getattr(lib, name)
        f.restype = ctypes.c_int32
        f.argtypes = args
    D = ctypes.c_double
    lib.vmoe_expert_mtmp.restype = D
    lib.vmoe_expert_mtmp.argtypes = [ctypes.c_int64, ctypes.c_int32, D, D, D, D]
    lib.vmoe_group_experts_workspace_bytes.restype = ctypes.c_size_t
    lib.vmoe_group_experts_workspace_bytes.argtypes = [ctypes.c_int32, D, D, D]
    lib.vmoe_group_experts.restype = ctypes.c_int32
    lib.vmoe_group_experts.argtypes = [ctypes.c_int32, P, P, D, D, D, D, P, P, P, ctypes.c_size_t]
    lib.vmoe_fill_clamp_refill.restype = ctypes.c_int32
    lib.vmoe_fill_clamp_refill.argtypes = [ctypes.c_int32, P, P, P, ctypes.c_int64, P, P, P, P,
                                           ctypes.c_size_t]
    return lib


_lib = _load()


def header_symbols() -> list[str]:
    """Entry points declared in include/vmoe.h."""
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*[\w\s\*]+?\b(vmoe_\w+)\s*\(", text, re.M)))


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


def _check(fn, status):
    if status != VMOE_OK:
        raise VmoeError(fn, status)


def vmoe_abi_version() -> int:
    return _lib.vmoe_abi_version()


def vmoe_capacity(shape: Shape) -> int:
    return _lib.vmoe_capacity(ctypes.byref(shape))


def vmoe_route_workspace_bytes(shape: Shape) -> int:
    return _lib.vmoe_route_workspace_bytes(ctypes.byref(shape))


def vmoe_route_bwd_workspace_bytes(shape: Shape) -> int:
    return _lib.vmoe_route_bwd_workspace_bytes(ctypes.byref(shape))


def vmoe_route(shape, x, w_router, logit_bias, noise, flags, logits, probs, expert_idx, slot,
               gate, order, counts, row_base, workspace, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check("vmoe_route", _lib.vmoe_route(
        ctypes.byref(shape), _ptr(x), _ptr(w_router), _ptr(logit_bias), _ptr(noise), flags,
        _ptr(logits), _ptr(probs), _ptr(expert_idx), _ptr(slot), _ptr(gate), _ptr(order),
        _ptr(counts), _ptr(row_base), _ptr(workspace), ws_bytes, _stream(stream)))


def vmoe_route_noalloc(shape, x, w_router, logit_bias, noise, flags, logits, probs, expert_idx,
                       slot, gate, order, counts, row_base, stream=None):
    """vmoe_route with the library's static per-GPU scratch (no workspace)."""
    _check("vmoe_route_noalloc", _lib.vmoe_route_noalloc(
        ctypes.byref(shape), _ptr(x), _ptr(w_router), _ptr(logit_bias), _ptr(noise), flags,
        _ptr(logits), _ptr(probs), _ptr(expert_idx), _ptr(slot), _ptr(gate), _ptr(order),
        _ptr(counts), _ptr(row_base), _stream(stream)))


def vmoe_dispatch(shape, x, expert_idx, slot, row_base, xe, stream=None):
    _check("vmoe_dispatch", _lib.vmoe_dispatch(
        ctypes.byref(shape), _ptr(x), _ptr(expert_idx), _ptr(slot), _ptr(row_base), _ptr(xe),
        _stream(stream)))


def vmoe_expert_ffn_fwd(shape, xe, counts, w1, b1, w2, b2, act, act_grad, ye, stream=None):
    _check("vmoe_expert_ffn_fwd", _lib.vmoe_expert_ffn_fwd(
        ctypes.byref(shape), _ptr(xe), _ptr(counts), _ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2),
        _ptr(act), _ptr(act_grad), _ptr(ye), _stream(stream)))


def vmoe_dispatch_ffn_fwd(shape, x, expert_idx, slot, row_base, counts, w1, b1, w2, b2,
                          row_token, act, act_grad, ye, stream=None):
    """Dispatch fused into the expert MLP forward (no xe); writes row_token."""
    _check("vmoe_dispatch_ffn_fwd", _lib.vmoe_dispatch_ffn_fwd(
        ctypes.byref(shape), _ptr(x), _ptr(expert_idx), _ptr(slot), _ptr(row_base),
        _ptr(counts), _ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2), _ptr(row_token), _ptr(act),
        _ptr(act_grad), _ptr(ye), _stream(stream)))


def vmoe_expert_ffn_bwd_gather(shape, x, row_token, counts, w1, w2, act, act_grad, dye, dh, dxe,
                               dw1, db1, dw2, db2, stream=None):
    """Expert MLP backward reading xe's rows from x through row_token."""
    _check("vmoe_expert_ffn_bwd_gather", _lib.vmoe_expert_ffn_bwd_gather(
        ctypes.byref(shape), _ptr(x), _ptr(row_token), _ptr(counts), _ptr(w1), _ptr(w2),
        _ptr(act), _ptr(act_grad), _ptr(dye), _ptr(dh), _ptr(dxe), _ptr(dw1), _ptr(db1),
        _ptr(dw2), _ptr(db2), _stream(stream)))


def vmoe_expert_ffn_fwd_quota(shape, xe, counts, w1, b1, w2, b2, act, act_grad, ye,
                              stream=None):
    """vmoe_expert_ffn_fwd with the fill-clamp-refill tile scheduler."""
    _check("vmoe_expert_ffn_fwd_quota", _lib.vmoe_expert_ffn_fwd_quota(
        ctypes.byref(shape), _ptr(xe), _ptr(counts), _ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2),
        _ptr(act), _ptr(act_grad), _ptr(ye), _stream(stream)))


def vmoe_expert_ffn_bwd_quota(shape, xe, counts, w1, w2, act, act_grad, dye, dh, dxe, dw1, db1,
                              dw2, db2, stream=None):
    """vmoe_expert_ffn_bwd with the fill-clamp-refill tile scheduler."""
    _check("vmoe_expert_ffn_bwd_quota", _lib.vmoe_expert_ffn_bwd_quota(
        ctypes.byref(shape), _ptr(xe), _ptr(counts), _ptr(w1), _ptr(w2), _ptr(act),
        _ptr(act_grad), _ptr(dye), _ptr(dh), _ptr(dxe), _ptr(dw1), _ptr(db1), _ptr(dw2),
        _ptr(db2), _stream(stream)))


def vmoe_fill_clamp_refill_device(n, min_units, sat_units, coef, budget, alloc_units,
                                  stream=None):
    """Device fill-clamp-refill units (one wavefront), device tensors."""
    _check("vmoe_fill_clamp_refill_device", _lib.vmoe_fill_clamp_refill_device(
        int(n), _ptr(min_units), _ptr(sat_units), _ptr(coef), int(budget), _ptr(alloc_units),
        _stream(stream)))


def vmoe_combine_fwd(shape, ye, expert_idx, slot, row_base, gate, y, stream=None):
    _check("vmoe_combine_fwd", _lib.vmoe_combine_fwd(
        ctypes.byref(shape), _ptr(ye), _ptr(expert_idx), _ptr(slot), _ptr(row_base), _ptr(gate),
        _ptr(y), _stream(stream)))


def vmoe_combine_bwd(shape, dy, ye, expert_idx, slot, row_base, gate, dye, dgate, stream=None):
    _check("vmoe_combine_bwd", _lib.vmoe_combine_bwd(
        ctypes.byref(shape), _ptr(dy), _ptr(ye), _ptr(expert_idx), _ptr(slot), _ptr(row_base),
        _ptr(gate), _ptr(dye), _ptr(dgate), _stream(stream)))


def vmoe_expert_ffn_bwd(shape, xe, counts, w1, w2, act, act_grad, dye, dh, dxe, dw1, db1, dw2,
                        db2, stream=None):
    _check("vmoe_expert_ffn_bwd", _lib.vmoe_expert_ffn_bwd(
        ctypes.byref(shape), _ptr(xe), _ptr(counts), _ptr(w1), _ptr(w2), _ptr(act),
        _ptr(act_grad),
        _ptr(dye), _ptr(dh), _ptr(dxe), _ptr(dw1), _ptr(db1), _ptr(dw2), _ptr(db2),
        _stream(stream)))


def vmoe_dispatch_bwd(shape, dxe, expert_idx, slot, row_base, dx, stream=None):
    _check("vmoe_dispatch_bwd", _lib.vmoe_dispatch_bwd(
        ctypes.byref(shape), _ptr(dxe), _ptr(expert_idx), _ptr(slot), _ptr(row_base), _ptr(dx),
        _stream(stream)))


def vmoe_dispatch_route_bwd(shape, dxe, row_base, x, w_router, probs, expert_idx, slot, dgate,
                            dx, dw_router, workspace, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check("vmoe_dispatch_route_bwd", _lib.vmoe_dispatch_route_bwd(
        ctypes.byref(shape), _ptr(dxe), _ptr(row_base), _ptr(x), _ptr(w_router), _ptr(probs),
        _ptr(expert_idx), _ptr(slot), _ptr(dgate), _ptr(dx), _ptr(dw_router), _ptr(workspace),
        ws_bytes, _stream(stream)))


def vmoe_dispatch_route_bwd_dlogits(shape, dxe, row_base, x, w_router, probs, expert_idx, slot,
                                    dgate, dlogits, dx, dw_router, workspace, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check("vmoe_dispatch_route_bwd_dlogits", _lib.vmoe_dispatch_route_bwd_dlogits(
        ctypes.byref(shape), _ptr(dxe), _ptr(row_base), _ptr(x), _ptr(w_router), _ptr(probs),
        _ptr(expert_idx), _ptr(slot), _ptr(dgate), _ptr(dlogits), _ptr(dx), _ptr(dw_router),
        _ptr(workspace), ws_bytes, _stream(stream)))


def vmoe_balance_loss_workspace_bytes(shape: Shape) -> int:
    return int(_lib.vmoe_balance_loss_workspace_bytes(ctypes.byref(shape)))


def vmoe_balance_loss(shape, logits, logit_bias, noise, probs, noise_std, w_importance, w_load,
                      losses, importance, load, dlogits, workspace, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check("vmoe_balance_loss", _lib.vmoe_balance_loss(
        ctypes.byref(shape), _ptr(logits), _ptr(logit_bias), _ptr(noise), _ptr(probs),
        float(noise_std), float(w_importance), float(w_load), _ptr(losses), _ptr(importance),
        _ptr(load), _ptr(dlogits), _ptr(workspace), ws_bytes, _stream(stream)))


def vmoe_route_bwd(shape, x, w_router, probs, expert_idx, slot, dgate, dx, dw_router, workspace,
                   stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check("vmoe_route_bwd", _lib.vmoe_route_bwd(
        ctypes.byref(shape), _ptr(x), _ptr(w_router), _ptr(probs), _ptr(expert_idx), _ptr(slot),
        _ptr(dgate), _ptr(dx), _ptr(dw_router), _ptr(workspace), ws_bytes, _stream(stream)))


# ---------------------------------------------------- expert grouping (host)

def vmoe_expert_mtmp(tokens, d_k, bytes_per_elem, theta1, theta2, m_f) -> float:
    """Temporary DRAM estimate of one expert, bytes (host)."""
    return _lib.vmoe_expert_mtmp(int(tokens), int(d_k), float(bytes_per_elem), float(theta1),
                                 float(theta2), float(m_f))


def vmoe_group_experts(mtmp, lifespan, mem_budget, mem_static, eta, unit_bytes):
    """Ordered time slices of the experts (host arrays in, numpy out):
    returns (slice_of int32 [n], n_slices)."""
    import numpy as np
    m = np.ascontiguousarray(mtmp, dtype=np.float64)
    r = np.ascontiguousarray(lifespan, dtype=np.float64)
    n = int(m.size)
    if r.size != n:
        raise ValueError("mtmp and lifespan differ in length")
    ws_bytes = _lib.vmoe_group_experts_workspace_bytes(n, float(mem_budget), float(mem_static),
                                                       float(unit_bytes))
    ws = np.empty(max(ws_bytes, 8), dtype=np.uint8)
    out = np.empty(max(n, 1), dtype=np.int32)
    ns = ctypes.c_int32(0)
    _check("vmoe_group_experts", _lib.vmoe_group_experts(
        n, m.ctypes.data, r.ctypes.data, float(mem_budget), float(mem_static), float(eta),
        float(unit_bytes), out.ctypes.data, ctypes.addressof(ns), ws.ctypes.data, ws_bytes))
    return out[:n], int(ns.value)


def vmoe_fill_clamp_refill(min_units, sat_units, coef, budget):
    """Host routine: fill-clamp-refill shares of `budget` units; returns
    (alloc f64 array, alloc_units i32 array, rounds)."""
    import numpy as np
    mn = np.ascontiguousarray(min_units, dtype=np.int32)
    sat = np.ascontiguousarray(sat_units, dtype=np.int32)
    w = np.ascontiguousarray(coef, dtype=np.float64)
    n = len(mn)
    if len(sat) != n or len(w) != n:
        raise ValueError("min_units, sat_units and coef must have one entry per expert")
    alloc = np.zeros(n, np.float64)
    units = np.zeros(n, np.int32)
    ws = np.zeros(max(n, 1), np.int32)
    rounds = ctypes.c_int32(0)
    c = ctypes.c_void_p
    _check("vmoe_fill_clamp_refill", _lib.vmoe_fill_clamp_refill(
        n, c(mn.ctypes.data), c(sat.ctypes.data), c(w.ctypes.data), int(budget),
        c(alloc.ctypes.data), c(units.ctypes.data), ctypes.cast(ctypes.byref(rounds), c),
        c(ws.ctypes.data), ws.nbytes))
    return alloc, units, int(rounds.value)
