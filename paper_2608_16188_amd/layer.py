"""One V-MoE layer's forward + backward through libvmoe, with torch buffers.

`LayerBuffers` owns every device tensor of one pass (inputs, saved
activations, gradients, workspaces) for a fixed shape, allocated once so a
training step allocates nothing; `forward` / `backward` / `step` enqueue the
eight C-ABI calls on the current stream. All arithmetic runs in libvmoe.
"""
from __future__ import annotations

import numpy as np
import torch

from . import vmoe as V
from . import workloads as W


def _dev_tensor(a: np.ndarray, dtype: str | None, device) -> torch.Tensor:
    """Host numpy -> device tensor. bf16 arrays arrive as uint16 bit patterns."""
    if a is None:
        return None
    if dtype == W.BF16 and a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def to_numpy(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> numpy; bf16 comes back as uint16 bit patterns."""
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


class LayerBuffers:
    def __init__(self, cfg: W.LayerConfig, inputs: dict, device="cuda", capacity_override=0):
        self.cfg = cfg
        self.device = torch.device(device)
        dt = V.VMOE_BF16 if cfg.dtype == W.BF16 else V.VMOE_F32
        self.shape = V.make_shape(cfg.n_tokens, cfg.n_groups, cfg.d_model, cfg.d_ff,
                                  cfg.n_experts, cfg.k, cfg.capacity_factor, dt,
                                  cfg.capacity_rounding, capacity_override)
        self.C = V.vmoe_capacity(self.shape)
        if self.C < 0:
            raise ValueError("invalid layer shape")
        N, G, d, f, E, k = (cfg.n_tokens, cfg.n_groups, cfg.d_model, cfg.d_ff, cfg.n_experts,
                            cfg.k)
        R = G * self.C
        N = max(N, 1)  # zero-token layers still pass valid (unused) pointers
        act = torch.bfloat16 if dt == V.VMOE_BF16 else torch.float32
        dev = self.device
        i32, f32 = torch.int32, torch.float32

        def up(name):
            return _dev_tensor(inputs.get(name), cfg.dtype, dev)

        self.x, self.w_router = up("x"), up("w_router")
        self.w1, self.b1, self.w2, self.b2 = up("w1"), up("b1"), up("w2"), up("b2")
        self.dy = up("dy")
        if cfg.n_tokens == 0:  # an empty batch still hands over allocated rows
            self.x = torch.zeros(1, d, dtype=act, device=dev)
            self.dy = torch.zeros(1, d, dtype=act, device=dev)
        self.logit_bias = None if inputs.get("logit_bias") is None else \
            torch.from_numpy(inputs["logit_bias"]).to(dev)
        self.noise = None if inputs.get("noise") is None else \
            torch.from_numpy(inputs["noise"]).to(dev)
        # routing
        self.logits = torch.empty(N, E, dtype=f32, device=dev)
        self.probs = torch.empty(N, E, dtype=f32, device=dev)
        self.expert_idx = torch.empty(N, k, dtype=i32, device=dev)
        self.slot = torch.empty(N, k, dtype=i32, device=dev)
        self.gate = torch.empty(N, k, dtype=f32, device=dev)
        self.order = torch.empty(N, dtype=i32, device=dev)
        self.counts = torch.empty(G, E, dtype=i32, device=dev)
        self.row_base = torch.empty(G, E, dtype=i32, device=dev)
        self.route_ws = torch.empty(max(V.vmoe_route_workspace_bytes(self.shape), 16),
                                    dtype=torch.uint8, device=dev)
        # expert buffers
        self.xe = torch.empty(E, R, d, dtype=act, device=dev)
        self.row_token = torch.empty(E, max(R, 1), dtype=i32, device=dev)  # fused path
        self.a = torch.empty(E, R, f, dtype=act, device=dev)       # gelu(H)
        self.a_grad = torch.empty(E, R, f, dtype=act, device=dev)  # gelu'(H)
        self.ye = torch.empty(E, R, d, dtype=act, device=dev)
        self.y = torch.empty(N, d, dtype=act, device=dev)
        # backward
        self.dye = torch.empty(E, R, d, dtype=act, device=dev)
        self.dgate = torch.empty(N, k, dtype=f32, device=dev)
        self.dh = torch.empty(E, R, f, dtype=act, device=dev)
        self.dxe = torch.empty(E, R, d, dtype=act, device=dev)
        self.dw1 = torch.empty(E, f, d, dtype=f32, device=dev)
        self.db1 = torch.empty(E, f, dtype=f32, device=dev)
        self.dw2 = torch.empty(E, d, f, dtype=f32, device=dev)
        self.db2 = torch.empty(E, d, dtype=f32, device=dev)
        self.dx = torch.empty(N, d, dtype=f32, device=dev)
        self.dw_router = None if cfg.routers_frozen else \
            torch.empty(G, E, d, dtype=f32, device=dev)
        self.route_bwd_ws = torch.empty(max(V.vmoe_route_bwd_workspace_bytes(self.shape), 16),
                                        dtype=torch.uint8, device=dev)

    # ---------------------------------------------------------------- calls
    def route(self, logits_in: bool = False, stream=None):
        V.vmoe_route(self.shape, self.x, self.w_router, self.logit_bias, self.noise,
                     V.VMOE_ROUTE_LOGITS_IN if logits_in else 0, self.logits, self.probs,
                     self.expert_idx, self.slot, self.gate, self.order, self.counts,
                     self.row_base, self.route_ws, stream)

    def forward(self, logits_in: bool = False, stream=None, quota: bool = False,
                gather: bool = False):
        """quota: the expert MLP through the fill-clamp-refill tile scheduler
        (vmoe_expert_ffn_fwd_quota; same results); gather: the dispatch fused
        into the up-projection's loads (vmoe_dispatch_ffn_fwd; xe unused)."""
        s = self.shape
        self.route(logits_in, stream)
        if gather:
            V.vmoe_dispatch_ffn_fwd(s, self.x, self.expert_idx, self.slot, self.row_base,
                                    self.counts, self.w1, self.b1, self.w2, self.b2,
                                    self.row_token, self.a, self.a_grad, self.ye, stream)
            V.vmoe_combine_fwd(s, self.ye, self.expert_idx, self.slot, self.row_base, self.gate,
                               self.y, stream)
            return
        V.vmoe_dispatch(s, self.x, self.expert_idx, self.slot, self.row_base, self.xe, stream)
        ffn = V.vmoe_expert_ffn_fwd_quota if quota else V.vmoe_expert_ffn_fwd
        ffn(s, self.xe, self.counts, self.w1, self.b1, self.w2, self.b2, self.a, self.a_grad,
            self.ye, stream)
        V.vmoe_combine_fwd(s, self.ye, self.expert_idx, self.slot, self.row_base, self.gate,
                           self.y, stream)

    def backward(self, stream=None, fused: bool = True, quota: bool = False,
                 gather: bool = False):
        """fused: dispatch and router backward in one call (bit-identical to
        vmoe_dispatch_bwd followed by vmoe_route_bwd, which fused=False runs);
        quota: the expert MLP backward through the fill-clamp-refill tile
        scheduler."""
        s = self.shape
        V.vmoe_combine_bwd(s, self.dy, self.ye, self.expert_idx, self.slot, self.row_base,
                           self.gate, self.dye, self.dgate, stream)
        if gather:
            V.vmoe_expert_ffn_bwd_gather(s, self.x, self.row_token, self.counts, self.w1,
                                         self.w2, self.a, self.a_grad, self.dye, self.dh,
                                         self.dxe, self.dw1, self.db1, self.dw2, self.db2, stream)
        else:
            ffn = V.vmoe_expert_ffn_bwd_quota if quota else V.vmoe_expert_ffn_bwd
            ffn(s, self.xe, self.counts, self.w1, self.w2, self.a, self.a_grad, self.dye,
                self.dh, self.dxe, self.dw1, self.db1, self.dw2, self.db2, stream)
        if fused:
            V.vmoe_dispatch_route_bwd(s, self.dxe, self.row_base, self.x, self.w_router,
                                      self.probs, self.expert_idx, self.slot, self.dgate, self.dx,
                                      self.dw_router, self.route_bwd_ws, stream)
            return
        V.vmoe_dispatch_bwd(s, self.dxe, self.expert_idx, self.slot, self.row_base, self.dx,
                            stream)
        V.vmoe_route_bwd(s, self.x, self.w_router, self.probs, self.expert_idx, self.slot,
                         self.dgate, self.dx, self.dw_router, self.route_bwd_ws, stream)

    def step(self, stream=None, quota: bool = False, gather: bool = False):
        self.forward(stream=stream, quota=quota, gather=gather)
        self.backward(stream=stream, quota=quota, gather=gather)
