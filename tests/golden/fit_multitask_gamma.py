"""Fit the router-skew strength of the 17-task expert pool.

The drifted multi-task workload should load its 16 shared experts following a
Zipf law with exponent 1.2. The generator gives expert e a per-task logit
offset -gamma * ln(e + 1); this script bisects gamma so that the pooled
top-1 histogram, computed by the oracle's router and gate, fits
share(rank) ~ rank^-s with s = 1.2 (least squares in log-log).

Run:  python tests/golden/fit_multitask_gamma.py
and copy the printed value into workloads.MULTITASK_GAMMA.
"""
import dataclasses
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))

import oracle  # noqa: E402
from paper_2608_16188_amd import workloads as W  # noqa: E402


def zipf_exponent(cfg) -> float:
    inp = W.make_inputs(cfg, with_grad=False)
    x = W.to_f64(inp["x"], cfg.dtype)
    wr = W.to_f64(inp["w_router"], cfg.dtype)
    logits = oracle.router_logits(x, wr, cfg.n_groups)
    top1 = oracle.gate(logits, 1)["idx"][:, 0]
    share = np.bincount(top1, minlength=cfg.n_experts).astype(np.float64)
    share = np.sort(share)[::-1]
    share = share[share > 0] / share.sum()
    rank = np.arange(1, len(share) + 1)
    slope = np.polyfit(np.log(rank), np.log(share), 1)[0]
    return -slope


def main(target=1.2):
    base = W.CONFIGS["multitask17_bf16"]
    lo, hi = 0.0, 3.0
    for _ in range(14):
        mid = 0.5 * (lo + hi)
        s = zipf_exponent(dataclasses.replace(base, zipf_gamma=mid))
        print(f"gamma={mid:.4f} s={s:.4f}", flush=True)
        if s < target:
            lo = mid
        else:
            hi = mid
    gamma = round(0.5 * (lo + hi), 3)
    print(f"MULTITASK_GAMMA = {gamma:.3f}  (fitted s = "
          f"{zipf_exponent(dataclasses.replace(base, zipf_gamma=gamma)):.3f})")


if __name__ == "__main__":
    main()
