"""ctypes marshalling for the C oracle (test infrastructure only).

Every function takes and returns numpy arrays. Float inputs of the layer are
passed as float64 arrays holding values exactly representable in the layer's
dtype (the caller widens bf16 or f32 exactly); routing inputs are float32.
See vmoe_oracle.c for the definition each function computes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "vmoe_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

__all__ = [
    "capacity", "exp_spec", "router_logits", "gate", "bpr", "route", "dispatch",
    "combine_fwd", "combine_bwd", "dispatch_bwd", "ffn_fwd", "ffn_bwd_rows",
    "ffn_bwd_weights", "ffn_bwd_weight_entries", "route_bwd", "expert_rows", "layer",
]


def build(force: bool = True) -> str:
    """Compile liboracle.so with IEEE float semantics (no contraction, no fast-math),
    with OpenMP over independent outputs (results do not depend on threads)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
                               "-fopenmp", "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def load():
    global _lib
    if _lib is None:
        build(force=False)
        _lib = ctypes.CDLL(_LIB)
        _lib.orc_exp.restype = ctypes.c_float
        _lib.orc_exp.argtypes = [ctypes.c_float]
        _lib.orc_capacity.restype = ctypes.c_int
        _lib.orc_capacity.argtypes = [ctypes.c_int] * 4 + [ctypes.c_double, ctypes.c_int]
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _f32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float32)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def capacity(n_tokens, n_groups, n_experts, k, capacity_factor, rounding=0) -> int:
    return load().orc_capacity(n_tokens, n_groups, n_experts, k, float(capacity_factor), rounding)


def exp_spec(u: np.ndarray) -> np.ndarray:
    lib = load()
    u = np.asarray(u, dtype=np.float32).ravel()
    return np.array([lib.orc_exp(float(v)) for v in u], dtype=np.float32)


def router_logits(x, w_router, n_groups):
    x, wr = _f64(x), _f64(w_router)
    N, d = x.shape
    E = wr.shape[1]
    out = np.empty((N, E), np.float32)
    load().orc_router_logits(N, n_groups, d, E, _p(x), _p(wr), _p(out))
    return out


def gate(logits, k, bias=None, noise=None):
    """-> dict(z, probs, idx, prio)"""
    logits, bias, noise = _f32(logits), _f32(bias), _f32(noise)
    N, E = logits.shape
    z = np.empty((N, E), np.float32)
    probs = np.empty((N, E), np.float32)
    idx = np.empty((N, k), np.int32)
    prio = np.empty(N, np.float32)
    load().orc_gate(N, E, k, _p(logits), _p(bias), _p(noise), _p(z), _p(probs), _p(idx), _p(prio))
    return dict(z=z, probs=probs, idx=idx, prio=prio)


def bpr(probs, idx, prio, n_groups, C):
    """-> dict(order, slot, gate, counts, row_base)"""
    probs, prio, idx = _f32(probs), _f32(prio), _i32(idx)
    N, E = probs.shape
    k = idx.shape[1]
    G = n_groups
    order = np.empty(N, np.int32)
    slot = np.empty((N, k), np.int32)
    gatev = np.empty((N, k), np.float32)
    counts = np.empty((G, E), np.int32)
    row_base = np.empty((G, E), np.int32)
    load().orc_bpr(N, G, E, k, C, _p(probs), _p(idx), _p(prio), _p(order), _p(slot), _p(gatev),
                   _p(counts), _p(row_base))
    return dict(order=order, slot=slot, gate=gatev, counts=counts, row_base=row_base)


def route(logits, k, C, n_groups=1, bias=None, noise=None):
    """Gate + batch-prioritized routing from fp32 logits."""
    g = gate(logits, k, bias, noise)
    r = bpr(g["probs"], g["idx"], g["prio"], n_groups, C)
    r.update(g)
    return r


def dispatch(x, idx, slot, row_base, n_experts, C, n_groups=1):
    x = _f64(x)
    N, d = x.shape
    k = idx.shape[1]
    xe = np.full((n_experts, n_groups * C, d), np.nan)
    load().orc_dispatch(N, n_groups, d, n_experts, k, C, _p(x), _p(_i32(idx)), _p(_i32(slot)),
                        _p(_i32(row_base)), _p(xe))
    return xe


def combine_fwd(ye, idx, slot, row_base, gatev, n_tokens, C, n_groups=1):
    ye = _f64(ye)
    E, _, d = ye.shape
    k = idx.shape[1]
    y = np.empty((n_tokens, d))
    load().orc_combine_fwd(n_tokens, n_groups, d, E, k, C, _p(ye), _p(_i32(idx)), _p(_i32(slot)),
                           _p(_i32(row_base)), _p(_f32(gatev)), _p(y))
    return y


def combine_bwd(dy, ye, idx, slot, row_base, gatev, C, n_groups=1):
    dy, ye = _f64(dy), _f64(ye)
    N, d = dy.shape
    E = ye.shape[0]
    k = idx.shape[1]
    dye = np.full(ye.shape, np.nan)
    dgate = np.empty((N, k))
    load().orc_combine_bwd(N, n_groups, d, E, k, C, _p(dy), _p(ye), _p(_i32(idx)), _p(_i32(slot)),
                           _p(_i32(row_base)), _p(_f32(gatev)), _p(dye), _p(dgate))
    return dye, dgate


def dispatch_bwd(dxe, idx, slot, row_base, n_tokens, C, n_groups=1):
    dxe = _f64(dxe)
    E, _, d = dxe.shape
    k = idx.shape[1]
    dx = np.empty((n_tokens, d))
    load().orc_dispatch_bwd(n_tokens, n_groups, d, E, k, C, _p(dxe), _p(_i32(idx)),
                            _p(_i32(slot)), _p(_i32(row_base)), _p(dx))
    return dx


def ffn_fwd(xe_rows, w1, b1, w2, b2, with_grad=False):
    """One expert over the given rows -> (H, A, ye), or (H, A, G, ye) with
    G = gelu'(H) when with_grad."""
    xe, w1, b1, w2, b2 = map(_f64, (xe_rows, w1, b1, w2, b2))
    rows, d = xe.shape
    f = w1.shape[0]
    H = np.empty((rows, f))
    A = np.empty((rows, f))
    G = np.empty((rows, f)) if with_grad else None
    ye = np.empty((rows, d))
    load().orc_ffn_fwd(rows, d, f, _p(xe), _p(w1), _p(b1), _p(w2), _p(b2), _p(H), _p(A), _p(G),
                       _p(ye))
    return (H, A, G, ye) if with_grad else (H, A, ye)


def ffn_bwd_rows(xe_rows, w1, b1, w2, dye_rows):
    """One expert, per-row backward -> (dxe, dH)."""
    xe, w1, b1, w2, dye = map(_f64, (xe_rows, w1, b1, w2, dye_rows))
    rows, d = xe.shape
    f = w1.shape[0]
    dxe = np.empty((rows, d))
    dH = np.empty((rows, f))
    load().orc_ffn_bwd_rows(rows, d, f, _p(xe), _p(w1), _p(b1), _p(w2), _p(dye), _p(dxe), _p(dH))
    return dxe, dH


def ffn_bwd_weights(xe_rows, w1, b1, w2, dye_rows):
    """One expert -> (dW1 [f,d], db1 [f], dW2 [d,f], db2 [d])."""
    xe, w1, b1, w2, dye = map(_f64, (xe_rows, w1, b1, w2, dye_rows))
    rows, d = xe.shape
    f = w1.shape[0]
    dw1, db1 = np.empty((f, d)), np.empty(f)
    dw2, db2 = np.empty((d, f)), np.empty(d)
    load().orc_ffn_bwd_weights(rows, d, f, _p(xe), _p(w1), _p(b1), _p(w2), _p(dye), _p(dw1),
                               _p(db1), _p(dw2), _p(db2))
    return dw1, db1, dw2, db2


def ffn_bwd_weight_entries(xe_rows, w1, b1, w2, dye_rows, which, row, col):
    """Selected entries: which 1=dW1[row,col] 2=dW2[row,col] 3=db1[row] 4=db2[row]."""
    xe, w1, b1, w2, dye = map(_f64, (xe_rows, w1, b1, w2, dye_rows))
    rows, d = xe.shape
    f = w1.shape[0]
    which, row, col = _i32(which), _i32(row), _i32(col)
    out = np.empty(len(which))
    load().orc_ffn_bwd_weight_entries(rows, d, f, _p(xe), _p(w1), _p(b1), _p(w2), _p(dye),
                                      len(which), _p(which), _p(row), _p(col), _p(out))
    return out


def route_bwd(x, w_router, probs, idx, slot, dgate, n_groups, dx_in=None, want_dwr=True):
    """-> (dx, dw_router or None, dz); dx = dx_in + gate-path gradient."""
    x, wr = _f64(x), _f64(w_router)
    N, d = x.shape
    E = wr.shape[1]
    k = idx.shape[1]
    dx = np.zeros((N, d)) if dx_in is None else _f64(dx_in).copy()
    dwr = np.empty(wr.shape) if want_dwr else None
    dz = np.empty((N, E))
    load().orc_route_bwd(N, n_groups, d, E, k, _p(x), _p(wr), _p(_f32(probs)), _p(_i32(idx)),
                         _p(_i32(slot)), _p(_f64(dgate)), _p(dx), _p(dwr), _p(dz))
    return dx, dwr, dz


def expert_rows(counts):
    """n_e = sum over groups of counts[g, e]."""
    return np.asarray(counts).sum(axis=0)


def layer(x, w_router, w1, b1, w2, b2, dy, *, k, C, n_groups=1, bias=None, noise=None,
          logits=None, want_dwr=True, rows_only=None):
    """Whole layer, forward then backward, by chaining the functions above.

    Float inputs are float64 arrays of exactly representable values. If
    `logits` is given it replaces the router product (logits-in mode).
    rows_only: if not None, a set of experts whose weight gradients are
    computed; others are skipped (None = all experts).
    Returns a dict with every intermediate and gradient.
    """
    x, w_router, w1, b1, w2, b2, dy = map(_f64, (x, w_router, w1, b1, w2, b2, dy))
    N, d = x.shape
    E, f = w1.shape[0], w1.shape[1]
    G = n_groups
    if logits is None:
        logits = router_logits(x, w_router, G)
    r = route(logits, k, C, G, bias, noise)
    r["logits"] = logits
    n_e = expert_rows(r["counts"])
    xe = dispatch(x, r["idx"], r["slot"], r["row_base"], E, C, G)
    H = np.full((E, G * C, f), np.nan)
    A = np.full((E, G * C, f), np.nan)
    Gd = np.full((E, G * C, f), np.nan)
    ye = np.full((E, G * C, d), np.nan)
    for e in range(E):
        if n_e[e]:
            r_ = slice(0, n_e[e])
            H[e, r_], A[e, r_], Gd[e, r_], ye[e, r_] = ffn_fwd(xe[e, r_], w1[e], b1[e], w2[e],
                                                               b2[e], with_grad=True)
    y = combine_fwd(ye, r["idx"], r["slot"], r["row_base"], r["gate"], N, C, G)
    dye, dgate = combine_bwd(dy, ye, r["idx"], r["slot"], r["row_base"], r["gate"], C, G)
    dxe = np.full((E, G * C, d), np.nan)
    dH = np.full((E, G * C, f), np.nan)
    dw1, db1 = np.zeros((E, f, d)), np.zeros((E, f))
    dw2, db2 = np.zeros((E, d, f)), np.zeros((E, d))
    for e in range(E):
        if n_e[e]:
            dxe[e, :n_e[e]], dH[e, :n_e[e]] = ffn_bwd_rows(xe[e, :n_e[e]], w1[e], b1[e], w2[e],
                                                           dye[e, :n_e[e]])
        if rows_only is None or e in rows_only:
            dw1[e], db1[e], dw2[e], db2[e] = ffn_bwd_weights(xe[e, :n_e[e]], w1[e], b1[e], w2[e],
                                                             dye[e, :n_e[e]])
    dx = dispatch_bwd(dxe, r["idx"], r["slot"], r["row_base"], N, C, G)
    dx_total, dwr, dz = route_bwd(x, w_router, r["probs"], r["idx"], r["slot"], dgate, G,
                                  dx_in=dx, want_dwr=want_dwr)
    r.update(n_e=n_e, xe=xe, H=H, A=A, Gd=Gd, ye=ye, y=y, dye=dye, dgate=dgate, dxe=dxe, dH=dH,
             dw1=dw1, db1=db1, dw2=dw2, db2=db2, dx_dispatch=dx, dx=dx_total, dw_router=dwr,
             dz=dz)
    return r
