"""A stack of path-compositional MoE layers with residual connections, for multi-layer
decode steps (the paper's gains are measured in decoding, Section 5).

Each layer l holds its own router matrix W_r[l] [n,H], expert weights and mask [n,n]; a
step runs, per layer, the router GEMM fused with the top-k, the path table, the expansion,
the projection and combine, and the residual h += y. Every step runs in libpcomoe's
kernels; this module only owns the buffers and the order of the calls. Attention and norms
are outside the scope: the stack exercises the MoE layers and the weight streaming of a
decode step.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional

import torch

from . import binding as b


@dataclass
class StackLayer:
    w_router: torch.Tensor    # [n, H]
    w_gate: torch.Tensor      # [n, F, H]
    w_up: torch.Tensor        # [n, F, H]
    w_down: torch.Tensor      # [n, H, F]
    mask: torch.Tensor        # [n, n] uint8


class MoEStack:
    def __init__(self, layers: List[StackLayer], T: int, k: int, beta_mode: int = b.BETA_SRC_COND):
        if not layers:
            raise ValueError("a stack needs at least one layer")
        l0 = layers[0]
        n, F, H = l0.w_gate.shape
        self.layers, self.T, self.H, self.F, self.n, self.k = layers, T, H, F, n, k
        dev, dtype = l0.w_gate.device, l0.w_gate.dtype
        self.plan = b.LayerPlan(T, H, F, n, k, dtype, dev, beta_mode=beta_mode)
        dt = b.PCM_BF16 if dtype == torch.bfloat16 else b.PCM_F32
        nws = b.workspace_bytes(b.OP_ROUTE_LOGITS, T, H, 0, n, k, dt)
        self.ws_router = torch.empty((max(nws, 1),), dtype=torch.uint8, device=dev) if nws else None
        self.logits: Optional[torch.Tensor] = None

    def layer_step(self, l: int, h: torch.Tensor, keep_logits: bool = False, stream=None):
        """One layer on hidden states h [T,H] (updated in place); returns the layer output y."""
        L, p = self.layers[l], self.plan
        if keep_logits:
            with b._on(stream):
                self.logits = torch.empty((self.T, self.n), dtype=torch.float32, device=h.device)
        b.pcm_route_logits(h, L.w_router, self.k, logits=self.logits if keep_logits else None,
                           topk_ids=p.ids, topk_w=p.w, ws=self.ws_router, stream=stream)
        b.pcm_build_paths(p.ids, p.w, L.mask, p.beta_mode, out=p.paths, ws=p.ws_paths, stream=stream)
        b.pcm_expand(h, L.w_gate, L.w_up, p.paths, u=p.u, stream=stream)
        b.pcm_project_combine(p.u, L.w_down, p.paths, y=p.y, ws=p.ws_proj, stream=stream)
        b.pcm_residual_add(h, p.y, stream=stream)
        return p.y

    def forward(self, h: torch.Tensor, stream=None) -> torch.Tensor:
        for l in range(len(self.layers)):
            self.layer_step(l, h, stream=stream)
        return h

    def capture(self, h: torch.Tensor) -> "torch.cuda.CUDAGraph":
        """forward(h) as one HIP graph (binding.capture_graph): each replay runs every layer on
        h's current contents, in place. The capture's eager warm-up runs forward(h) once, so
        set h after capturing and before each replay."""
        return b.capture_graph(lambda: self.forward(h))


def random_stack(L: int, T: int, H: int, F: int, n: int, k: int, density: float, seed: int,
                 device, dtype=torch.bfloat16, native_layers: int = 2, w_std: float = 0.02) -> MoEStack:
    """Seeded synthetic weights drawn on the device (N(0, w_std)); the first `native_layers`
    layers keep only diagonal paths (mask = I), the others a random mask of the given
    off-diagonal density."""
    g = torch.Generator(device=device).manual_seed(seed)
    layers = []
    for l in range(L):
        def rnd(*shape):
            return (torch.randn(shape, generator=g, device=device, dtype=torch.float32) * w_std).to(dtype)
        if l < native_layers:
            mask = torch.eye(n, dtype=torch.uint8, device=device)
        else:
            mask = (torch.rand((n, n), generator=g, device=device) < density).to(torch.uint8)
            mask.fill_diagonal_(1)
        layers.append(StackLayer(rnd(n, H), rnd(n, F, H), rnd(n, F, H), rnd(n, H, F), mask))
    return MoEStack(layers, T, k)
