"""Seeded synthetic inputs for one V-MoE layer's forward and backward pass.

This module only draws random numbers and packs them into the dtypes the
layer consumes. It contains none of the layer's arithmetic (no routing, no
softmax, no expert MLP), so it can feed both the HIP path and the CPU oracle
without coupling them.

The paper adapts V-MoEs on private video datasets with trained weights
(Sec. 5.1); neither is available, so every tensor here is synthetic with the
shapes of the standard ViT token grids: 197 = 14*14 + 1 tokens per 224-px
image at patch 16, 577 = 24*24 + 1 at 384 px, widths 192/768/1024 with 4x MLP.

Layouts (row-major, contiguous):
    x          [N, d]        tokens, N = images * tokens_per_image
    w_router   [G, E, d]     one router per routing group (nn.Linear layout)
    logit_bias [E] f32 or None
    noise      [N, E] f32 or None   gating noise, drawn here and passed in
    w1         [E, f, d]     expert up-projection  (nn.Linear layout)
    b1         [E, f]
    w2         [E, d, f]     expert down-projection (nn.Linear layout)
    b2         [E, d]
    dy         [N, d]        upstream gradient of the layer output
bf16 tensors are numpy uint16 arrays holding the bf16 bit patterns.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

F32 = "f32"
BF16 = "bf16"


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    name: str
    cid: int                  # seed namespace of the workload
    images: int
    tokens_per_image: int
    d_model: int
    d_ff: int
    n_experts: int
    k: int
    capacity_factor: float
    dtype: str
    n_groups: int = 1         # routing groups (one per task for the multi-task pool)
    noise_var: float = 0.0    # variance of the gating noise; 0 = no noise
    router_std: float = 0.02
    weight_std: float = 0.02
    hot_experts: int = 0      # experts given a constant logit offset
    hot_offset: float = 0.0
    task_mean_var: float = 0.0  # per-task token mean offset variance (drift)
    zipf_gamma: float = 0.0   # per-task router load skew strength
    routers_frozen: bool = False
    capacity_rounding: int = 0  # 0 = round half away from zero, 1 = ceil

    @property
    def n_tokens(self) -> int:
        return self.images * self.tokens_per_image


# Router-skew strength for the 17-task pool. Written by
# tests/golden/fit_multitask_gamma.py, which bisects it so that the pooled
# top-1 expert histogram of the oracle fits a Zipf law with exponent 1.2.
MULTITASK_GAMMA = 0.353

CONFIGS = {
    c.name: c
    for c in [
        LayerConfig("tiny_fp32", 1, images=4, tokens_per_image=197, d_model=192, d_ff=768,
                    n_experts=8, k=2, capacity_factor=1.25, dtype=F32, noise_var=1.0 / 8),
        LayerConfig("vitb16_bf16", 2, images=32, tokens_per_image=197, d_model=768, d_ff=3072,
                    n_experts=8, k=2, capacity_factor=1.05, dtype=BF16, router_std=0.1),
        LayerConfig("wide_e32_bf16", 3, images=128, tokens_per_image=197, d_model=768, d_ff=3072,
                    n_experts=32, k=2, capacity_factor=1.0, dtype=BF16, noise_var=1.0 / 32),
        LayerConfig("multitask17_bf16", 4, images=17 * 8, tokens_per_image=197, d_model=768,
                    d_ff=3072, n_experts=16, k=2, capacity_factor=1.25, dtype=BF16, n_groups=17,
                    task_mean_var=0.5, zipf_gamma=MULTITASK_GAMMA, routers_frozen=True),
        LayerConfig("vitl16_384_bf16", 5, images=64, tokens_per_image=577, d_model=1024,
                    d_ff=4096, n_experts=32, k=2, capacity_factor=1.05, dtype=BF16,
                    hot_experts=4, hot_offset=2.0),
    ]
}


def custom_config(name="custom", *, n_tokens, d_model, d_ff, n_experts, k, capacity_factor,
                  dtype=BF16, n_groups=1, cid=90, **kw) -> LayerConfig:
    """A config with arbitrary sizes (tests: ragged tails, edge cases)."""
    return LayerConfig(name, cid, images=n_tokens, tokens_per_image=1, d_model=d_model,
                       d_ff=d_ff, n_experts=n_experts, k=k, capacity_factor=capacity_factor,
                       dtype=dtype, n_groups=n_groups, **kw)


# ---------------------------------------------------------------- bf16 bits

def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); return the bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    rounding = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + rounding) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def to_dtype(a: np.ndarray, dtype: str) -> np.ndarray:
    return f32_to_bf16_bits(a) if dtype == BF16 else np.ascontiguousarray(a, dtype=np.float32)


def to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of an f32 or bf16-bit array to float64."""
    if dtype == BF16:
        return bf16_bits_to_f32(a).astype(np.float64)
    return np.asarray(a, dtype=np.float32).astype(np.float64)


# ---------------------------------------------------------------- sampling

def _seed(cfg: LayerConfig, tensor_id: int, salt: int = 0) -> int:
    return 20260000 + 100 * cfg.cid + tensor_id + 7919 * salt


def truncated_normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    """N(0, std^2) truncated at +-2 std by resampling, as float32."""
    z = rng.standard_normal(size=shape, dtype=np.float32)
    bad = np.abs(z) > 2.0
    while bad.any():
        z[bad] = rng.standard_normal(size=int(bad.sum()), dtype=np.float32)
        bad = np.abs(z) > 2.0
    return z * np.float32(std)


def make_inputs(cfg: LayerConfig, salt: int = 0, with_grad: bool = True,
                with_experts: bool = True) -> dict:
    """Draw every input of one fwd+bwd pass for `cfg`.

    Tensor ids (seed offsets): 1 x, 2 router, 3 noise, 4 w1, 5 b1, 6 w2, 7 b2,
    8 dy, 9 task means.
    """
    N, d, f, E, G = cfg.n_tokens, cfg.d_model, cfg.d_ff, cfg.n_experts, cfg.n_groups
    assert N % G == 0, "tokens must split evenly into routing groups"
    Ng = N // G

    x = np.random.default_rng(_seed(cfg, 1, salt)).standard_normal((N, d), dtype=np.float32)
    wr = truncated_normal(np.random.default_rng(_seed(cfg, 2, salt)), (G, E, d), cfg.router_std)

    if cfg.task_mean_var > 0.0:
        # Drifted multi-task inputs: each task's tokens share a mean offset mu,
        # and its router carries b_e * mu / |mu|^2 so that mu . w_e adds the
        # fixed logit offset b_e = -gamma * ln(e + 1): expert e gets load rank e+1.
        mu = np.random.default_rng(_seed(cfg, 9, salt)).standard_normal((G, d), dtype=np.float32)
        mu *= np.float32(math.sqrt(cfg.task_mean_var))
        b = (-cfg.zipf_gamma * np.log(np.arange(1, E + 1, dtype=np.float64))).astype(np.float32)
        for g in range(G):
            x[g * Ng:(g + 1) * Ng] += mu[g]
            wr[g] += np.outer(b, mu[g] / np.float32(np.dot(mu[g], mu[g])))

    bias = None
    if cfg.hot_experts > 0:
        bias = np.zeros(E, dtype=np.float32)
        bias[:cfg.hot_experts] = np.float32(cfg.hot_offset)

    noise = None
    if cfg.noise_var > 0.0:
        noise = np.random.default_rng(_seed(cfg, 3, salt)).standard_normal((N, E), dtype=np.float32)
        noise *= np.float32(math.sqrt(cfg.noise_var))

    out = dict(x=to_dtype(x, cfg.dtype), w_router=to_dtype(wr, cfg.dtype), logit_bias=bias,
               noise=noise)
    if not with_experts:
        return out
    r4 = np.random.default_rng(_seed(cfg, 4, salt))
    r6 = np.random.default_rng(_seed(cfg, 6, salt))
    w1 = np.empty((E, f, d), dtype=np.uint16 if cfg.dtype == BF16 else np.float32)
    w2 = np.empty((E, d, f), dtype=w1.dtype)
    for e in range(E):  # per expert keeps the float32 temporaries small
        w1[e] = to_dtype(truncated_normal(r4, (f, d), cfg.weight_std), cfg.dtype)
        w2[e] = to_dtype(truncated_normal(r6, (d, f), cfg.weight_std), cfg.dtype)
    b1 = truncated_normal(np.random.default_rng(_seed(cfg, 5, salt)), (E, f), cfg.weight_std)
    b2 = truncated_normal(np.random.default_rng(_seed(cfg, 7, salt)), (E, d), cfg.weight_std)

    out.update(w1=w1, b1=to_dtype(b1, cfg.dtype), w2=w2, b2=to_dtype(b2, cfg.dtype))
    if with_grad:
        dy = np.random.default_rng(_seed(cfg, 8, salt)).standard_normal((N, d), dtype=np.float32)
        out["dy"] = to_dtype(dy, cfg.dtype)
    return out


def random_logits(n_tokens: int, n_experts: int, seed: int, scale: float = 1.0,
                  tie_every: int = 0) -> np.ndarray:
    """Free-standing fp32 router logits for routing-only tests.

    tie_every > 0 copies every tie_every-th row from its predecessor and
    quantises values to multiples of 1/8 so that exact ties are frequent.
    """
    rng = np.random.default_rng(seed)
    z = (rng.standard_normal((n_tokens, n_experts)) * scale).astype(np.float32)
    if tie_every > 0:
        z = np.round(z * 8.0).astype(np.float32) / np.float32(8.0)
        z[tie_every::tie_every] = z[tie_every - 1:-1:tie_every][: len(z[tie_every::tie_every])]
    return z
