"""The whole layer, forward and backward, at full size (oracle).

TEST INFRASTRUCTURE ONLY (part of the oracle): only the tests, the smoke
check and the benchmark's CPU-baseline leg may import it.

The same chain as `oracle.layer` (routing, dispatch, expert MLP, combine and
every backward, in the order the layer defines them), with two differences
that only change cost: the expert MLP runs through oracle/dense.py (float64
matrix products) instead of the plain loops, and the per-expert tensors are
kept packed, one [n_e, width] array per expert, instead of [E, G*C, width]
buffers of mostly unused rows. Routing, dispatch, combine, their backward
and the router backward are the plain-loop C functions of vmoe_oracle.c.
"""
from __future__ import annotations

import numpy as np

from . import api, dense


def layer_packed(x, w_router, w1, b1, w2, b2, dy, *, k, C, n_groups=1, bias=None,
                 noise=None, logits=None, want_dwr=True, progress=None):
    """Float inputs: float64 arrays of values exact in the layer's dtype.
    logits (float32) replaces the router product when given (logits-in).
    Returns a dict with the routing outputs, per-expert lists xe, A, Gd
    (gelu'(H)), ye, dye, dH, dxe (each [n_e, width]), the token tensors y,
    dgate, dx, and the gradients dw1, db1, dw2, db2, dw_router."""
    say = progress or (lambda *a: None)
    N, d = x.shape
    E, f = w1.shape[0], w1.shape[1]
    G = n_groups
    if logits is None:
        logits = api.router_logits(x, w_router, G)
    r = api.route(logits, k, C, G, bias, noise)
    r["logits"] = logits
    n_e = api.expert_rows(r["counts"])
    meta = (r["idx"], r["slot"], r["row_base"])
    buf = api.dispatch(x, *meta, E, C, G)
    xe = [buf[e, :n_e[e]].copy() for e in range(E)]
    say("oracle: routing and dispatch done")
    A, Gd, ye = [], [], []
    for e in range(E):
        _, a, g, y_e = dense.ffn_fwd(xe[e], w1[e], b1[e], w2[e], b2[e])
        A.append(a)
        Gd.append(g)
        ye.append(y_e)
    say("oracle: expert MLP forward done")
    buf.fill(np.nan)
    for e in range(E):
        buf[e, :n_e[e]] = ye[e]
    y = api.combine_fwd(buf, *meta, r["gate"], N, C, G)
    dye_buf, dgate = api.combine_bwd(dy, buf, *meta, r["gate"], C, G)
    dye = [dye_buf[e, :n_e[e]].copy() for e in range(E)]
    del dye_buf
    say("oracle: combine and its backward done")
    dw1, db1 = np.zeros((E, f, d)), np.zeros((E, f))
    dw2, db2 = np.zeros((E, d, f)), np.zeros((E, d))
    dH, dxe = [], []
    buf.fill(np.nan)
    for e in range(E):
        g = dense.ffn_bwd(xe[e], A[e], Gd[e], w1[e], w2[e], dye[e])
        dH.append(g["dH"])
        dxe.append(g["dxe"])
        buf[e, :n_e[e]] = g["dxe"]
        dw1[e], db1[e], dw2[e], db2[e] = g["dw1"], g["db1"], g["dw2"], g["db2"]
    say("oracle: expert MLP backward done")
    dx_disp = api.dispatch_bwd(buf, *meta, N, C, G)
    del buf
    dx, dwr, dz = api.route_bwd(x, w_router, r["probs"], r["idx"], r["slot"], dgate, G,
                                dx_in=dx_disp, want_dwr=want_dwr)
    say("oracle: dispatch and router backward done")
    r.update(n_e=n_e, xe=xe, A=A, Gd=Gd, ye=ye, y=y, dye=dye, dgate=dgate, dH=dH, dxe=dxe,
             dw1=dw1, db1=db1, dw2=dw2, db2=db2, dx=dx, dw_router=dwr, dz=dz)
    return r
