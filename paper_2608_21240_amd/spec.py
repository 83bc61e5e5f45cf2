"""Speculative prefetching (Sec. 4.1, Alg. 1): the draft rollout on the GPU and its
prefetch intents.

A rollout starts from the current layer's input hidden state and runs one depth per
future layer, each depth three library calls on the current stream:
  route      moe_route_bucket with the future layer's router; every expert is treated as
             absent with confidence 0 (< tau = 1), so every slot is LoRE and topk_w holds
             the router's probabilities;
  surrogate  moe_expert_ffn_grouped with that layer's shared block and LoRE factors:
             S(h) and B_k A_k h for every predicted expert;
  update     moe_spec_update: enqueue, confidence, halting, draft-state step.
The predictions land in pinned host memory (written by the update kernel); queue()
waits for the rollout's event and turns them into per-layer issue lists (Eq. 3).
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import torch

from . import spice
from .layer import torch_dtype


class SpecRollout:
    """Buffers for rollouts of up to `depth` future layers over T tokens."""

    def __init__(self, shape, T: int, depth: int, device: str = "cuda", trace: bool = False):
        self.shape, self.T, self.H = shape, T, depth
        s, K, N, d = shape, shape.top_k, shape.n_experts, shape.d
        self.cfg = spice.make_cfg(s, 0, tau=1.0, conf_mode=spice.SPICE_CONF_INPUT, norm_topk=0)
        i32 = dict(dtype=torch.int32, device=device)
        f32 = dict(dtype=torch.float32, device=device)
        td = torch_dtype(s.dtype)
        self.resident = torch.full((N,), -1, **i32)
        self.conf0 = torch.zeros((T, K), **f32)
        self.topk_idx = torch.empty((T, K), **i32)
        self.topk_w = torch.empty((T, K), **f32)
        self.slot_class = torch.empty((T, K), dtype=torch.uint8, device=device)
        self.offsets = torch.empty((3, N + 1), **i32)
        self.perm = torch.empty(T * K, **i32)
        self.inv_perm = torch.empty(T * K, **i32)
        self.y_slots = torch.zeros((T * K, d), **f32)
        self.y_shared = torch.zeros((T, d), **f32)  # stays 0 without a shared block
        self.ws_bytes = spice.spice_workspace_bytes(self.cfg, T)
        self.ws = torch.zeros(self.ws_bytes, dtype=torch.uint8, device=device)
        # draft states: one per depth with trace, else two buffers used in turn
        self.h = torch.empty((depth if trace else 2, T, d), dtype=td, device=device)
        self.trace = trace
        self.halted = torch.zeros(T, **i32)
        self.pred_idx = torch.empty((depth, T, K), **i32)
        self.pred_prob = torch.empty((depth, T, K), **f32)
        self.conf = torch.empty((depth, T), **f32)
        self.pred_idx_h = torch.empty((depth, T, K), dtype=torch.int32).pin_memory()
        self.pred_prob_h = torch.empty((depth, T, K), dtype=torch.float32).pin_memory()
        self.conf_h = torch.empty((depth, T), dtype=torch.float32).pin_memory()
        self.hosts = [spice.spec_host(self.pred_idx_h[j], self.pred_prob_h[j], self.conf_h[j]) for j in range(depth)]
        self.done = torch.cuda.Event(blocking=True)  # waiters sleep instead of spinning
        self.n, self.T_run = 0, T

    def state(self, j: int) -> torch.Tensor:
        """Draft state after depth j + 1 (needs trace=True for every j)."""
        return self.h[j if self.trace else j % 2]

    def run(self, layers: Sequence, x: torch.Tensor, l_min: int, tau: float, T: Optional[int] = None) -> None:
        """Rollout from x over layers[0..] (the views of layers l+1, l+2, ...: wg, bias, w13s,
        w2s, lore_A, lore_B); at most `depth` of them."""
        T = self.T if T is None else T
        n = min(len(layers), self.H)
        self.n, self.T_run = n, T
        self.halted.zero_()
        c = self.cfg
        for j in range(n):
            L = layers[j]
            h_in = x if j == 0 else self.state(j - 1)
            h_out = self.state(j)
            spice.moe_route_bucket(c, T, h_in, L.wg, L.bias, self.resident, self.conf0, None, self.topk_idx,
                                   self.topk_w, self.slot_class, self.offsets, self.perm, self.inv_perm, None,
                                   self.ws, self.ws_bytes)
            spice.moe_expert_ffn_grouped(c, T, h_in, self.perm, self.offsets, self.resident, None, None, L.w13s,
                                         L.w2s, L.lore_A, L.lore_B, self.y_slots, self.y_shared, self.ws,
                                         self.ws_bytes)
            spice.moe_spec_update(c, T, j + 1, l_min, tau, j == n - 1, h_in, h_out, self.topk_idx, self.topk_w,
                                  self.inv_perm, self.y_slots, self.y_shared, self.halted, self.pred_idx[j],
                                  self.pred_prob[j], self.conf[j], self.hosts[j], self.ws, self.ws_bytes)
        self.done.record()

    def queue(self, max_per_depth: int) -> List[List[int]]:
        """Per-depth issue lists of the last rollout (waits for it)."""
        self.done.synchronize()
        if self.n == 0:
            return []
        T = self.T_run
        return spice.moe_prefetch_queue(self.cfg, self.pred_idx_h[: self.n].view(self.n, -1)[:, : T * self.shape.top_k]
                                        .reshape(self.n, T, -1).numpy(),
                                        self.pred_prob_h[: self.n].view(self.n, -1)[:, : T * self.shape.top_k]
                                        .reshape(self.n, T, -1).numpy(), max_per_depth)

    def flags(self, clear: bool = True) -> int:
        return spice.spice_workspace_flags(self.ws, self.ws_bytes, clear)
