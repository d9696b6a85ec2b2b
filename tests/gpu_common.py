"""Shared helpers of the GPU parity tests (comparison metrics, input caches)."""
from __future__ import annotations

import functools
import sys

import numpy as np

import oracle
from paper_2608_16188_amd import workloads as W

# Tolerance on max|gpu - oracle| / max|oracle| per tensor: bf16 storage with
# f32 accumulation vs f32 end to end.
TOL = {W.F32: 1e-4, W.BF16: 2e-2}


def say(*a):
    """Progress line that names the case before a GPU step (flushed)."""
    print("[gpu-test]", *a, file=sys.stderr, flush=True)


def rel_err(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    scale = np.max(np.abs(ref))
    if scale == 0.0:
        return float(np.max(np.abs(got)))
    return float(np.max(np.abs(got - ref)) / scale)


def assert_close(name, got, ref, tol):
    err = rel_err(got, ref)
    assert np.all(np.isfinite(np.asarray(got, dtype=np.float64))), f"{name}: non-finite values"
    assert err <= tol, f"{name}: max rel err {err:.3e} > {tol:.1e}"
    return err


def bits_equal(a, b) -> bool:
    a, b = np.asarray(a), np.asarray(b)
    if a.shape != b.shape:
        return False
    if a.dtype == np.float32:
        return np.array_equal(a.view(np.uint32), np.asarray(b, np.float32).view(np.uint32))
    return np.array_equal(a, b)


def as_f64(arr, dtype) -> np.ndarray:
    return W.to_f64(arr, dtype)


def assert_router_logits(got, x64, wr64, n_groups, dtype):
    """GPU router logits against the oracle's (double sum rounded once to f32).

    f32 activations: bit for bit (both sides sum the exact products in double
    in increasing i). bf16 activations: the GPU adds the exact bf16 products in
    f32 on the matrix cores (in the kernel's own order, d split over four
    waves), so a logit may differ from the exactly rounded sum by at most
    gamma_(d+3) * sum_i |x_i w_i| (an f32 sum of d exact terms plus three
    partial-sum additions, Higham eq. 3.5, gamma_n ~ n 2^-24) plus the
    reference's own rounding, 2^-24 |ref|; the check allows twice that.
    """
    ref = oracle.router_logits(x64, wr64, n_groups)
    got = np.asarray(got)
    if dtype == W.F32:
        assert bits_equal(got, ref), "router logits not bit-exact"
        return ref
    N, d = x64.shape
    ng = N // n_groups
    mag = np.empty_like(got, dtype=np.float64)
    for g in range(n_groups):
        mag[g * ng:(g + 1) * ng] = np.abs(x64[g * ng:(g + 1) * ng]) @ np.abs(wr64[g]).T
    bound = 2.0 * ((d + 3) * 2.0 ** -24 * mag + 2.0 ** -24 * np.abs(ref.astype(np.float64)))
    err = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    worst = float(np.max(err - bound)) if err.size else 0.0
    assert worst <= 0.0, f"router logits off by more than the f32 summation bound ({worst:.3g})"
    return ref


@functools.lru_cache(maxsize=2)
def workload_inputs(name: str, with_experts: bool = True):
    cfg = W.CONFIGS[name]
    return cfg, W.make_inputs(cfg, with_grad=with_experts, with_experts=with_experts)


def oracle_capacity(cfg: W.LayerConfig, override: int = 0) -> int:
    if override > 0:
        return override
    return oracle.capacity(cfg.n_tokens, cfg.n_groups, cfg.n_experts, cfg.k,
                           cfg.capacity_factor, cfg.capacity_rounding)


def rows_of_expert(r: dict, e: int, C: int, G: int):
    """Tokens and (t, j) of expert e's packed rows, in row order."""
    idx, slot, row_base = r["idx"], r["slot"], r["row_base"]
    N = idx.shape[0]
    ng = N // G
    n_e = int(r["counts"][:, e].sum())
    toks = np.full(n_e, -1, np.int64)
    js = np.full(n_e, -1, np.int64)
    kept = np.argwhere((idx == e) & (slot >= 0))
    for t, j in kept:
        row = row_base[t // ng, e] + slot[t, j]
        toks[row], js[row] = t, j
    assert (toks >= 0).all()
    return toks, js


# ------------------------------------------------------------------ every element

def elementwise_rel(got, ref) -> float:
    """max over elements of |a - b| / max(|b|, 1e-3 max|b|): the element-wise
    form of the relative error, reported beside the per-tensor one."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if ref.size == 0:
        return 0.0
    floor = 1e-3 * float(np.max(np.abs(ref)))
    if floor == 0.0:
        return float(np.max(np.abs(got)))
    return float(np.max(np.abs(got - ref) / np.maximum(np.abs(ref), floor)))


class Report:
    """Per-tensor metrics of one parity case: the per-tensor error
    max|a - b| / max|b|, the worst row's error against that row's own largest
    magnitude, and the element-wise form. Tensors checked in parts (one
    expert at a time) are merged by taking the worst part."""

    def __init__(self, case: str):
        self.case = case
        self.m = {}

    def add(self, name, tensor_rel, row_rel, elem_rel):
        old = self.m.get(name)
        new = dict(tensor=tensor_rel, worst_row=row_rel, elementwise=elem_rel)
        if old is not None:
            new = {k: max(old[k], new[k]) for k in new}
        self.m[name] = new

    def write(self):
        import json
        import os
        out = os.environ.get("VMOE_PARITY_REPORT_DIR")
        if out:
            os.makedirs(out, exist_ok=True)
            with open(os.path.join(out, f"{self.case}.json"), "w") as fh:
                json.dump(self.m, fh, indent=1, sort_keys=True)
        say(self.case, " ".join(f"{k}:{v['tensor']:.1e}/{v['worst_row']:.1e}/"
                                f"{v['elementwise']:.1e}" for k, v in sorted(self.m.items())))


def assert_rows_close(name, got, ref, tol, report=None, block=1):
    """Every row (leading index) of `got` within tol of `ref`, relative to
    that row's largest reference magnitude; a row whose reference is all zero
    must be exactly zero. Catches a wrong row far below the tensor's maximum
    (a light expert's, a dropped token's), which the per-tensor metric alone
    would let pass. Also checks the per-tensor metric and finiteness.
    block > 1 takes rows `block` at a time (a weight gradient's row is the
    same few coefficients times different vectors, so a single row's scale can
    sit far below its rounding error; 32 rows is one matrix-core block)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    if ref.size == 0:
        return
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    g2 = got.reshape(got.shape[0], -1)
    r2 = ref.reshape(ref.shape[0], -1)
    scale = np.max(np.abs(r2), axis=1)
    err = np.max(np.abs(g2 - r2), axis=1)
    if block > 1:
        starts = np.arange(0, len(scale), block)
        scale = np.maximum.reduceat(scale, starts)
        err = np.maximum.reduceat(err, starts)
    zero = scale == 0.0
    assert np.all(err[zero] == 0.0), f"{name}: rows {np.nonzero(zero & (err > 0))[0][:8]} " \
                                      "should be exactly zero"
    row_rel = err[~zero] / scale[~zero]
    worst = float(np.max(row_rel)) if row_rel.size else 0.0
    tensor = rel_err(got, ref)
    if report is not None:
        report.add(name, tensor, worst, elementwise_rel(got, ref))
    assert tensor <= tol, f"{name}: max rel err {tensor:.3e} > {tol:.1e}"
    bad = np.nonzero(~zero)[0][row_rel > tol]
    assert worst <= tol, f"{name}: rows {bad[:8]} off by up to {worst:.3e} of their magnitude"
