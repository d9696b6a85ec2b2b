"""Pins of the balance-loss oracle against mathematics it does not restate:
closed forms of CV^2, sampling of the load probability, finite differences of
the gradient, symmetry, and degenerate cases."""
import numpy as np
import pytest

from oracle import balance as B


def test_cv2_closed_forms():
    assert B.cv2([1, 1, 1, 1]) == 0.0
    assert B.cv2([4, 0, 0, 0]) == pytest.approx(3.0)   # one expert takes all: E - 1
    assert B.cv2([1, 3]) == pytest.approx(0.25)        # var 1, mean 2
    assert B.cv2([0, 0, 0]) == 0.0
    assert B.cv2([2, 4, 6]) == pytest.approx((8 / 3) / 16)
    assert np.all(B.cv2_grad([0, 0]) == 0)


def test_cv2_gradient_finite_differences():
    rng = np.random.default_rng(0)
    for E in (2, 5, 17):
        v = rng.uniform(0.1, 3.0, E)
        g = B.cv2_grad(v)
        h = 1e-6
        for e in range(E):
            a, b = v.copy(), v.copy()
            a[e] += h
            b[e] -= h
            assert (B.cv2(a) - B.cv2(b)) / (2 * h) == pytest.approx(g[e], rel=1e-6, abs=1e-9)


def test_load_probability_matches_sampling():
    """P[t, e] is the chance that e lands in the top-k when only its own noise
    is drawn again: count it by sampling."""
    rng = np.random.default_rng(1)
    N, E, k, sigma = 3, 5, 2, 0.7
    logits = rng.normal(0, 1, (N, E))
    bias = rng.normal(0, 0.3, E)
    noise = rng.normal(0, sigma, (N, E))
    P, _, _ = B.load_probability(logits, k, sigma, bias=bias, noise=noise)
    z = logits + bias + noise
    n = 200_000
    for t in range(N):
        for e in range(E):
            others = np.delete(z[t], e)
            fresh = logits[t, e] + bias[e] + rng.normal(0, sigma, n)
            beaten_by = (others[None, :] > fresh[:, None]).sum(axis=1)
            freq = (beaten_by < k).mean()
            tol = 4 * np.sqrt(max(P[t, e] * (1 - P[t, e]), 1e-4) / n) + 1e-3
            assert abs(freq - P[t, e]) < tol, (t, e, freq, P[t, e])


@pytest.mark.parametrize("E,k,G", [(6, 2, 2), (4, 1, 1), (8, 3, 3)])
def test_gradient_finite_differences(E, k, G):
    rng = np.random.default_rng(E * 10 + k)
    N, sigma = 4 * G, 0.5
    logits = rng.normal(0, 1.5, (N, E))
    bias = rng.normal(0, 0.2, E)
    noise = rng.normal(0, sigma, (N, E))
    w_imp, w_load = 0.7, 1.3
    r = B.balance_loss(logits, k, G, sigma, w_imp, w_load, bias=bias, noise=noise)
    h = 1e-6
    for t in range(N):
        for e in range(E):
            a, b = logits.copy(), logits.copy()
            a[t, e] += h
            b[t, e] -= h
            fa = B.balance_loss(a, k, G, sigma, w_imp, w_load, bias=bias, noise=noise)["total"]
            fb = B.balance_loss(b, k, G, sigma, w_imp, w_load, bias=bias, noise=noise)["total"]
            fd = (fa - fb) / (2 * h)
            assert fd == pytest.approx(r["dlogits"][t, e], rel=1e-5, abs=1e-8), (t, e)


def test_permuting_experts_permutes_gradient():
    rng = np.random.default_rng(3)
    N, E, k, sigma = 10, 7, 2, 0.4
    logits = rng.normal(0, 1, (N, E))
    noise = rng.normal(0, sigma, (N, E))
    perm = rng.permutation(E)
    r = B.balance_loss(logits, k, 2, sigma, noise=noise)
    q = B.balance_loss(logits[:, perm], k, 2, sigma, noise=noise[:, perm])
    np.testing.assert_allclose(q["losses"], r["losses"], rtol=1e-12)
    np.testing.assert_allclose(q["dlogits"], r["dlogits"][:, perm], rtol=1e-10, atol=1e-15)


def test_degenerate_cases():
    rng = np.random.default_rng(4)
    N, E = 12, 4
    logits = rng.normal(0, 1, (N, E))
    # every expert is always chosen when k = E: no load imbalance, no load gradient
    r = B.balance_loss(logits, E, 1, 0.3, w_imp=0.0, w_load=1.0)
    assert r["losses"][0, 1] == 0.0 and np.all(r["dlogits"] == 0)
    # equal logits and no noise: uniform importance and load
    r = B.balance_loss(np.zeros((N, E)), 2, 1, 0.3)
    assert r["losses"][0, 0] == pytest.approx(0.0, abs=1e-15)
    assert r["losses"][0, 1] == pytest.approx(0.0, abs=1e-15)
    # one expert dominating every token: importance CV^2 -> E - 1
    big = np.zeros((N, E))
    big[:, 0] = 60.0
    assert B.balance_loss(big, 1, 1, 0.3)["losses"][0, 0] == pytest.approx(E - 1, rel=1e-9)
    # a huge noise std makes every expert equally likely: load CV^2 -> 0
    r = B.balance_loss(logits, 2, 1, 1e6)
    assert r["losses"][0, 1] < 1e-10
    # importance sums to the group's token count (probability rows sum to one)
    r = B.balance_loss(logits, 2, 3, 0.3)
    np.testing.assert_allclose(r["imp"].sum(axis=1), N / 3, rtol=1e-12)


def test_router_mode_uses_f32_noisy_logits():
    """With the router's probabilities the threshold comes from the f32 sum
    (logits + bias) + noise; two logits equal in f32 but not in f64 rank by
    index."""
    logits = np.array([[1.0, 1.0 + 2.0 ** -30, 0.0]], dtype=np.float64)
    probs = B.softmax(logits.astype(np.float32).astype(np.float64)).astype(np.float32)
    r = B.balance_loss(logits, 1, 1, 0.5, probs=probs)
    # in f32 experts 0 and 1 tie; expert 2's threshold is the first of them
    _, _, tgt = B.load_probability(logits, 1, 0.5, f32=True)
    assert tgt[0, 2] == 0
    assert np.isfinite(r["dlogits"]).all()
