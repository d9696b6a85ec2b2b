"""Expert MLP forward and backward in float64 by matrix products.

TEST INFRASTRUCTURE ONLY (part of the oracle): only the tests, the smoke
check and the benchmark's CPU-baseline leg may import it; the product path
never does, and it shares nothing with the HIP library.

What it computes. Each expert is an MLP block (the expertised MLP blocks
routed to by sparse gating, paper Sec. 2.1) adapted by back-propagation
(Sec. 3.1-3.2). Over an expert's packed rows xe [n, d], with w1 [f, d],
b1 [f], w2 [d, f], b2 [d] (nn.Linear layout):
    H  = xe w1^T + b1          A = gelu(H) = H Phi(H)     A' = gelu'(H)
    ye = A w2^T + b2
and, for an upstream gradient dye [n, d], by the chain rule:
    dA  = dye w2               dH = dA * A'               dxe = dH w1
    dW2 = dye^T A              db2 = sum over rows of dye
    dW1 = dH^T xe              db1 = sum over rows of dH
with the exact GELU: Phi(h) = (1 + erf(h / sqrt 2)) / 2 and
gelu'(h) = Phi(h) + h phi(h), phi the standard normal density.

This is the same definition as the plain loops of vmoe_oracle.c
(orc_ffn_fwd, orc_ffn_bwd_rows, orc_ffn_bwd_weights), written with numpy's
float64 matrix product as the one library step so that the full-size
workloads finish in seconds. Nothing is rounded below float64 and nothing is
blocked or reordered beyond what each product does internally. Inputs are
float64 arrays of values exactly representable in the layer's dtype.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
from scipy.special import erf

_SQRT2 = math.sqrt(2.0)
_INV_SQRT_2PI = 1.0 / math.sqrt(2.0 * math.pi)
_THREADS = max(1, min(16, os.cpu_count() or 1))


def _elementwise(fn, h: np.ndarray) -> np.ndarray:
    """fn applied to h, split over threads in row chunks (numpy's and scipy's
    element-wise loops release the interpreter lock)."""
    out = np.empty_like(h)
    if h.size < (1 << 20) or h.ndim != 2:
        out[...] = fn(h)
        return out
    step = max(1, -(-h.shape[0] // _THREADS))

    def part(r0):
        out[r0:r0 + step] = fn(h[r0:r0 + step])

    with ThreadPoolExecutor(_THREADS) as ex:
        list(ex.map(part, range(0, h.shape[0], step)))
    return out


def gelu(h: np.ndarray) -> np.ndarray:
    """gelu(h) = h Phi(h), exact erf form."""
    return _elementwise(lambda v: 0.5 * v * (1.0 + erf(v / _SQRT2)), h)


def gelu_grad(h: np.ndarray) -> np.ndarray:
    """d gelu / dh = Phi(h) + h phi(h)."""
    return _elementwise(lambda v: 0.5 * (1.0 + erf(v / _SQRT2))
                        + v * _INV_SQRT_2PI * np.exp(-0.5 * v * v), h)


def ffn_fwd(xe, w1, b1, w2, b2):
    """One expert over its rows -> (H, A, A', ye), all float64 [n, f] / [n, d]."""
    H = xe @ w1.T + b1
    A = gelu(H)
    G = gelu_grad(H)
    ye = A @ w2.T + b2
    return H, A, G, ye


def ffn_bwd(xe, A, G, w1, w2, dye):
    """One expert's backward from the forward's A, A' -> dict of dA, dH, dxe,
    dw1 [f, d], db1 [f], dw2 [d, f], db2 [d]. With no rows every weight and
    bias gradient is 0 (an empty sum)."""
    dA = dye @ w2
    dH = dA * G
    dxe = dH @ w1
    return dict(dA=dA, dH=dH, dxe=dxe, dw2=dye.T @ A, db2=dye.sum(axis=0),
                dw1=dH.T @ xe, db1=dH.sum(axis=0))
