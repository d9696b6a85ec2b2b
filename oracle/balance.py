"""Oracle of the auxiliary balance losses on the gate (TEST INFRASTRUCTURE ONLY).

The paper names auxiliary balance losses (the AdaMV-MoE line of work, cited
in Sec. 1 and Sec. 2.3) as the way other systems fight load skew, without
defining them. This module restates the published noisy top-k gating
formulation of those losses (V-MoE, after the sparsely-gated MoE layer):

  importance  imp[g, e]  = sum over the group's tokens t of p[t, e], the
                           router's probability (softmax of the noisy logits
                           z = (logits + bias) + noise);
  load        load[g, e] = sum over t of P[t, e], the probability that e is
                           among the top-k of z when only e's own noise is
                           drawn again:  P = Phi((l'[t, e] - thr[t, e]) / sigma)
                           with l' = logits + bias (no noise), thr[t, e] the
                           k-th largest noisy logit among the OTHER experts
                           (-inf when fewer than k others exist), Phi the
                           standard normal CDF, sigma the noise std;
  each loss   CV^2(v)    = var(v) / mean(v)^2 over the E experts
                           (population variance; 0 when sum(v) = 0);
  objective              = sum over groups of w_imp CV^2(imp[g]) + w_load CV^2(load[g]).

Gradient with respect to the logits (dz = dlogits, as z = logits + bias +
noise): with c[g, e] = w dCV^2/dv_e = w 2 / (E mu^2) (v_e - mu - var / mu),
  importance: p[t, e] (c_imp[e] - sum_e' p[t, e'] c_imp[e'])   (softmax Jacobian)
  load:       + c_load[e] phi(u) / sigma at (t, e), and the same amount
              subtracted at (t, e*), the expert whose noisy logit is thr[t, e]
              (u = (l' - thr) / sigma, phi the standard normal density).
The threshold expert e* follows the top-k tie rule: equal noisy logits rank
the lower expert index first.

Two evaluation modes:
  * probs=None: every quantity in float64 (z = logits + bias + noise, p =
    softmax(z)); the mathematical function, for finite differences and
    sampling checks;
  * probs given (the router's stored float32 probabilities): z is rebuilt in
    float32 exactly as the router forms it, (logits + bias) + noise, so the
    threshold choice matches the device bit for bit; the rest is float64.

Shares no code with the library; only tests import it.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import ndtr


def cv2(v) -> float:
    """Squared coefficient of variation, var / mean^2 (0 for a zero sum)."""
    v = np.asarray(v, dtype=np.float64)
    if v.size == 0 or v.sum() == 0.0:
        return 0.0
    mu = v.mean()
    return float(((v - mu) ** 2).mean() / (mu * mu))


def cv2_grad(v) -> np.ndarray:
    """d CV^2 / d v_e = 2 / (E mu^2) (v_e - mu - var / mu); zeros for a zero sum."""
    v = np.asarray(v, dtype=np.float64)
    if v.size == 0 or v.sum() == 0.0:
        return np.zeros_like(v)
    E = v.size
    mu = v.mean()
    var = ((v - mu) ** 2).mean()
    return 2.0 / (E * mu * mu) * (v - mu - var / mu)


def _noisy(logits, bias, noise, f32: bool):
    l = np.asarray(logits, dtype=np.float32 if f32 else np.float64)
    dt = l.dtype
    clean = l + (np.zeros(l.shape[1], dt) if bias is None else np.asarray(bias, dtype=dt))
    z = clean + (np.zeros_like(clean) if noise is None else np.asarray(noise, dtype=dt))
    return clean.astype(np.float64), z.astype(np.float64)


def thresholds(z, k):
    """thr[t, e] = k-th largest of z[t, e'] over e' != e (lower index first on
    ties), and the expert holding it (-1, thr = -inf when E - 1 < k)."""
    N, E = z.shape
    thr = np.full((N, E), -np.inf)
    tgt = np.full((N, E), -1, dtype=np.int64)
    if E - 1 < k:
        return thr, tgt
    rows = np.arange(N)
    for e in range(E):
        others = [c for c in range(E) if c != e]
        zo = z[:, others]
        # stable sort of -z: equal values keep ascending expert order
        order = np.argsort(-zo, axis=1, kind="stable")
        pick = order[:, k - 1]
        thr[:, e] = zo[rows, pick]
        tgt[:, e] = np.asarray(others)[pick]
    return thr, tgt


def load_probability(logits, k, sigma, bias=None, noise=None, f32=False):
    """P[t, e] = Phi((l' - thr) / sigma), with u and the threshold expert."""
    clean, z = _noisy(logits, bias, noise, f32)
    thr, tgt = thresholds(z, k)
    u = (clean - thr) / sigma
    return ndtr(u), u, tgt


def softmax(z):
    m = z.max(axis=1, keepdims=True)
    w = np.exp(z - m)
    return w / w.sum(axis=1, keepdims=True)


def balance_loss(logits, k, n_groups, sigma, w_imp=1.0, w_load=1.0, bias=None, noise=None,
                 probs=None):
    """-> dict with losses [G, 2] (importance, load), imp, load [G, E],
    dlogits [N, E] (gradient of the weighted sum over groups) and total."""
    logits = np.asarray(logits)
    N, E = logits.shape
    G = n_groups
    if N % G:
        raise ValueError("tokens must split evenly into groups")
    f32 = probs is not None
    clean, z = _noisy(logits, bias, noise, f32)
    p = np.asarray(probs, dtype=np.float64) if f32 else softmax(z)
    thr, tgt = thresholds(z, k)
    u = (clean - thr) / sigma
    P = ndtr(u)
    dens = np.exp(-0.5 * u * u) / math.sqrt(2.0 * math.pi) / sigma  # phi(u) / sigma (0 at -inf)
    ng = N // G
    losses = np.zeros((G, 2))
    imp = np.zeros((G, E))
    load = np.zeros((G, E))
    dl = np.zeros((N, E))
    for g in range(G):
        s = slice(g * ng, (g + 1) * ng)
        imp[g] = p[s].sum(axis=0)
        load[g] = P[s].sum(axis=0)
        losses[g] = (cv2(imp[g]), cv2(load[g]))
        c_imp = w_imp * cv2_grad(imp[g])
        c_load = w_load * cv2_grad(load[g])
        pg = p[s]
        dl[s] = pg * (c_imp[None, :] - (pg @ c_imp)[:, None])
        a = c_load[None, :] * dens[s]
        dl[s] += a
        # the same amount leaves at each (t, e)'s threshold expert
        tt, ee = np.nonzero(tgt[s] >= 0)
        np.subtract.at(dl, (s.start + tt, tgt[s][tt, ee]), a[tt, ee])
    total = float((w_imp * losses[:, 0] + w_load * losses[:, 1]).sum())
    return dict(losses=losses, imp=imp, load=load, dlogits=dl, total=total)


def router_grad_extra(x, w_router, dlogits, n_groups):
    """The router-side products of an extra logit gradient: dx += dl W_r[g],
    dW_r[g] += dl_g^T x_g (float64)."""
    x = np.asarray(x, dtype=np.float64)
    wr = np.asarray(w_router, dtype=np.float64)
    dl = np.asarray(dlogits, dtype=np.float64)
    N = x.shape[0]
    ng = N // n_groups
    dx = np.zeros_like(x)
    dwr = np.zeros_like(wr)
    for g in range(n_groups):
        s = slice(g * ng, (g + 1) * ng)
        dx[s] = dl[s] @ wr[g]
        dwr[g] = dl[s].T @ x[s]
    return dx, dwr
