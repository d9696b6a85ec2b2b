"""Pins of oracle/dense.py, the float64 matrix-product form of the expert MLP
(forward, backward, weight gradients) that the full-size parity tests use.

Each pin is outside the module: torch's own linear / exact-GELU layers and
autograd in float64, the plain-loop C oracle (the same definition summed
term by term), central finite differences, and closed forms of the GELU.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import dense


def _expert(rng, n, d, f, scale=0.5):
    return (rng.standard_normal((n, d)), rng.standard_normal((f, d)) * scale,
            rng.standard_normal(f) * scale, rng.standard_normal((d, f)) * scale,
            rng.standard_normal(d) * scale, rng.standard_normal((n, d)))


@pytest.mark.parametrize("n,d,f", [(0, 8, 16), (1, 8, 16), (37, 24, 40), (300, 64, 96)])
def test_dense_expert_mlp_vs_torch_autograd(n, d, f):
    """Forward, saved gelu', every gradient against torch (float64, CPU):
    nn.functional.linear + exact-erf gelu, gradients by autograd."""
    rng = np.random.default_rng(n + 7)
    xe, w1, b1, w2, b2, dye = _expert(rng, n, d, f)
    H, A, G, ye = dense.ffn_fwd(xe, w1, b1, w2, b2)
    g = dense.ffn_bwd(xe, A, G, w1, w2, dye)
    F = torch.nn.functional
    t = {k: torch.tensor(v, requires_grad=True) for k, v in
         dict(xe=xe, w1=w1, b1=b1, w2=w2, b2=b2).items()}
    h = F.linear(t["xe"], t["w1"], t["b1"])
    h.retain_grad()
    y = F.linear(F.gelu(h, approximate="none"), t["w2"], t["b2"])
    (y * torch.tensor(dye)).sum().backward()
    close = lambda a, b: np.allclose(a, b, rtol=1e-11, atol=1e-12)  # noqa: E731
    assert close(ye, y.detach().numpy())
    assert close(A, F.gelu(h.detach(), approximate="none").numpy())
    assert close(g["dH"], h.grad.numpy())
    assert close(g["dxe"], t["xe"].grad.numpy())
    assert close(g["dw1"], t["w1"].grad.numpy())
    assert close(g["db1"], t["b1"].grad.numpy())
    assert close(g["dw2"], t["w2"].grad.numpy())
    assert close(g["db2"], t["b2"].grad.numpy())
    if n == 0:
        for key in ("dw1", "db1", "dw2", "db2"):
            assert np.all(g[key] == 0.0)


def test_dense_matches_plain_loop_oracle():
    """The same definition summed term by term in C (vmoe_oracle.c)."""
    rng = np.random.default_rng(3)
    xe, w1, b1, w2, b2, dye = _expert(rng, 29, 40, 56)
    H, A, G, ye = dense.ffn_fwd(xe, w1, b1, w2, b2)
    Hc, Ac, Gc, yec = oracle.ffn_fwd(xe, w1, b1, w2, b2, with_grad=True)
    for a, b in ((H, Hc), (A, Ac), (G, Gc), (ye, yec)):
        assert np.allclose(a, b, rtol=1e-12, atol=1e-13)
    g = dense.ffn_bwd(xe, A, G, w1, w2, dye)
    dxe, dH = oracle.ffn_bwd_rows(xe, w1, b1, w2, dye)
    dw1, db1, dw2, db2 = oracle.ffn_bwd_weights(xe, w1, b1, w2, dye)
    for a, b in ((g["dxe"], dxe), (g["dH"], dH), (g["dw1"], dw1), (g["db1"], db1),
                 (g["dw2"], dw2), (g["db2"], db2)):
        assert np.allclose(a, b, rtol=1e-11, atol=1e-12)


def test_dense_gradients_central_differences():
    rng = np.random.default_rng(11)
    xe, w1, b1, w2, b2, dye = _expert(rng, 4, 5, 7)
    H, A, G, _ = dense.ffn_fwd(xe, w1, b1, w2, b2)
    g = dense.ffn_bwd(xe, A, G, w1, w2, dye)
    args = dict(xe=xe, w1=w1, b1=b1, w2=w2, b2=b2)

    def loss(**kw):
        return float((dense.ffn_fwd(kw["xe"], kw["w1"], kw["b1"], kw["w2"], kw["b2"])[3]
                      * dye).sum())

    h = 1e-6
    for name, grad in (("xe", g["dxe"]), ("w1", g["dw1"]), ("b1", g["db1"]), ("w2", g["dw2"]),
                       ("b2", g["db2"])):
        for flat in range(args[name].size):
            p, m = dict(args), dict(args)
            p[name] = args[name].copy()
            m[name] = args[name].copy()
            p[name].flat[flat] += h
            m[name].flat[flat] -= h
            fd = (loss(**p) - loss(**m)) / (2 * h)
            assert abs(fd - grad.flat[flat]) < 1e-6, (name, flat)


def test_gelu_closed_forms():
    h = np.array([[0.0, 40.0, -40.0, 1.0, -1.0]])
    g, dg = dense.gelu(h), dense.gelu_grad(h)
    assert g[0, 0] == 0.0 and dg[0, 0] == 0.5
    assert g[0, 1] == 40.0 and dg[0, 1] == 1.0
    assert g[0, 2] == 0.0 and abs(dg[0, 2]) < 1e-300
    # gelu(1) = Phi(1), gelu(-1) = -(1 - Phi(1)), Phi(1) = 0.841344746068543
    assert abs(g[0, 3] - 0.8413447460685429) < 1e-15
    assert abs(g[0, 4] + (1 - 0.8413447460685429)) < 1e-15
    # the derivative against a central difference of the function itself
    x = np.linspace(-6, 6, 241)[None, :]
    e = 1e-6
    fd = (dense.gelu(x + e) - dense.gelu(x - e)) / (2 * e)
    assert np.max(np.abs(fd - dense.gelu_grad(x))) < 1e-8


def test_threaded_elementwise_equals_single_pass():
    """Large inputs are split over threads; the values are those of one pass."""
    h = np.random.default_rng(5).standard_normal((2048, 700))
    one = 0.5 * h * (1.0 + __import__("scipy").special.erf(h / np.sqrt(2.0)))
    assert np.array_equal(dense.gelu(h), one)
