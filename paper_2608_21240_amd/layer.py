"""Driver of one MoE layer call through the C ABI (memory and streams only).

``HostLayer`` holds the seeded weights of one layer in NumPy; ``DeviceLayer``
puts the resident experts into an HBM slot pool, plus the router, the shared
block and every expert's LoRE factors, and keeps the non-resident experts on
the host for the exact CPU path.  ``LayerRun`` owns the per-call buffers and
runs the path in the order the paper describes (Sec. 4.3):

    stream : moe_layer_gpu: routing + shared up | bucketing + shared down + routed up | routed down
             (the bucketing block also writes x and the routing into pinned host memory, then
             a ready word)  ........................................ -> combine (reads resid over PCIe)
    host   :   wait(ready word) -> exact residual on CPU threads -> resid (pinned) ^

With layer_call=False the same layer runs as the separate calls (moe_route_bucket,
moe_expert_ffn_grouped, moe_combine) and the host waits for the routing call's event.

Every arithmetic step runs inside libspice_moe (HIP kernels or its host path).
"""
from __future__ import annotations

import os
import time
from typing import Dict, List, Optional, Sequence

import numpy as np

import torch

from . import spice, synth
from .workloads import DTYPE_BF16, WFMT_MXFP4, Workload


def torch_dtype(dtype: int) -> torch.dtype:
    return torch.bfloat16 if dtype == DTYPE_BF16 else torch.float32


def to_tensor(a: np.ndarray, dtype: int, device=None, pin: bool = False) -> torch.Tensor:
    """Storage array (float32 or bf16 bits) -> tensor of the storage dtype."""
    if dtype == DTYPE_BF16:
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    if pin:
        return t.pin_memory()
    return t.to(device) if device is not None else t


class HostLayer:
    """Seeded weights of one layer (storage arrays), drawn lazily per expert."""

    def __init__(self, wl: Workload, layer: int = 0, resident: Optional[Sequence[int]] = None):
        self.wl, self.layer, self.shape = wl, layer, wl.shape
        self.resident = list(synth.resident_experts(wl, layer) if resident is None else resident)
        self.wg = synth.gen_router(wl, layer)
        self.bias = synth.gen_bias(wl, layer)
        self.w13s, self.w2s = synth.gen_shared(wl, layer)
        self.w_sg = synth.gen_shared_gate(wl, layer)  # None: ungated shared block
        self._experts: Dict[int, tuple] = {}
        self._lore: Dict[int, tuple] = {}

    def expert(self, e: int):
        if e not in self._experts:
            self._experts[e] = synth.gen_expert(self.wl, self.layer, e)
        return self._experts[e]

    def lore(self, e: int):
        if e not in self._lore:
            self._lore[e] = synth.gen_lore(self.wl, self.layer, e)
        return self._lore[e]

    def prefetch(self, experts: Sequence[int] = (), lore_experts: Sequence[int] = (), threads: int = 0) -> None:
        """Draw the given experts' weights and LoRE factors on a thread pool (each draw has
        its own seeded stream, so the result does not depend on the order)."""
        from concurrent.futures import ThreadPoolExecutor

        todo = [(0, e) for e in experts if e not in self._experts]
        todo += [(1, e) for e in lore_experts if e not in self._lore]
        if not todo:
            return

        def draw(item):
            kind, e = item
            return item, (synth.gen_expert if kind == 0 else synth.gen_lore)(self.wl, self.layer, e)

        n = threads or min(16, os.cpu_count() or 1)
        with ThreadPoolExecutor(n) as ex:
            for (kind, e), v in ex.map(draw, todo):
                (self._experts if kind == 0 else self._lore)[e] = v

    def resident_mask(self) -> np.ndarray:
        m = np.zeros(self.shape.n_experts, np.int32)
        m[self.resident] = 1
        return m

    def tables(self, experts: Sequence[int], lore_experts: Sequence[int]):
        """Per-expert weight tables of length N (None where not requested)."""
        N = self.shape.n_experts
        w13: List = [None] * N; w2: List = [None] * N; la: List = [None] * N; lb: List = [None] * N
        for e in experts:
            w13[e], w2[e] = self.expert(e)
        for e in lore_experts:
            la[e], lb[e] = self.lore(e)
        return w13, w2, la, lb


class DeviceLayer:
    """Device copy of a layer: pool of resident experts, router, shared block, LoRE factors."""

    def __init__(self, host: HostLayer, n_slots: Optional[int] = None, device: str = "cuda",
                 host_exact: bool = True):
        s, dt = host.shape, host.shape.dtype
        self.host, self.shape = host, s
        self.C = len(host.resident) if n_slots is None else n_slots
        td = torch_dtype(dt)
        self.wg = to_tensor(host.wg, dt, device)
        self.bias = None if host.bias is None else torch.from_numpy(host.bias).to(device)
        self.w13s = to_tensor(host.w13s, dt, device)
        self.w2s = to_tensor(host.w2s, dt, device)
        self.w_sg = None if host.w_sg is None else to_tensor(host.w_sg, dt, device)
        slot = np.full(s.n_experts, -1, np.int32)
        host.prefetch(range(s.n_experts) if host_exact else host.resident,
                      range(s.n_experts) if s.lore_rank > 0 else ())
        self.wfmt = host.wl.wfmt
        if self.wfmt == WFMT_MXFP4:
            # one MXFP4 byte blob per slot: [2I][d] and [d][I] (codes, then block scales)
            b13, b2 = synth.mxfp4_bytes(2 * s.inter, s.d), synth.mxfp4_bytes(s.d, s.inter)
            self.w13_pool = torch.empty((max(self.C, 1), b13), dtype=torch.uint8, device=device)
            self.w2_pool = torch.empty((max(self.C, 1), b2), dtype=torch.uint8, device=device)
        else:
            self.w13_pool = torch.empty((max(self.C, 1), 2 * s.inter, s.d), dtype=td, device=device)
            self.w2_pool = torch.empty((max(self.C, 1), s.d, s.inter), dtype=td, device=device)
        for i, e in enumerate(host.resident):
            w13, w2 = host.expert(e)
            self.w13_pool[i].copy_(self._weights(w13))
            self.w2_pool[i].copy_(self._weights(w2))
            slot[e] = i
        self.resident_slot = torch.from_numpy(slot).to(device)
        r = max(s.lore_rank, 1)
        self.lore_A = torch.empty((s.n_experts, r, s.d), dtype=td, device=device)
        self.lore_B = torch.empty((s.n_experts, s.d, r), dtype=td, device=device)
        if s.lore_rank > 0:
            for e in range(s.n_experts):
                A, B = host.lore(e)
                self.lore_A[e].copy_(to_tensor(A, dt))
                self.lore_B[e].copy_(to_tensor(B, dt))
        # host-resident weights of the non-resident experts (the exact CPU path), pinned so
        # that fetching them to the GPU (the exact-miss split) copies asynchronously
        self.host_w13: List = [None] * s.n_experts
        self.host_w2: List = [None] * s.n_experts
        if host_exact:
            for e in range(s.n_experts):
                if slot[e] < 0:
                    w13, w2 = host.expert(e)
                    self.host_w13[e] = self._weights(w13, pin=True)
                    self.host_w2[e] = self._weights(w2, pin=True)

    def _weights(self, a: np.ndarray, pin: bool = False) -> torch.Tensor:
        """A routed expert's weight array (storage dtype, or an MXFP4 byte blob) as a tensor."""
        if self.wfmt == WFMT_MXFP4:
            t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint8))
            return t.pin_memory() if pin else t
        return to_tensor(a, self.shape.dtype, pin=pin)

    def hbm_bytes(self) -> int:
        ts = [self.wg, self.w13s, self.w2s, self.w13_pool, self.w2_pool, self.lore_A, self.lore_B]
        return sum(t.numel() * t.element_size() for t in ts)


class LayerRun:
    """Buffers and streams for layer calls with up to T tokens."""

    def __init__(self, shape, T: int, n_slots: int, tau: float = 0.5, conf_mode: int = 0, norm_topk: int = 0,
                 device: str = "cuda", keep_logits: bool = False, fetch_slots: int = 0, wfmt: int = 0,
                 layer_call: bool = True):
        self.shape, self.T = shape, T
        self.layer_call = layer_call
        self.cfg = spice.make_cfg(shape, n_slots, tau, conf_mode, norm_topk, wfmt)
        s, K, N, d = shape, shape.top_k, shape.n_experts, shape.d
        i32 = dict(dtype=torch.int32, device=device)
        f32 = dict(dtype=torch.float32, device=device)
        self.topk_idx = torch.empty((T, K), **i32)
        self.topk_w = torch.empty((T, K), **f32)
        self.slot_class = torch.empty((T, K), dtype=torch.uint8, device=device)
        self.offsets = torch.empty((3, N + 1), **i32)
        self.perm = torch.empty(T * K, **i32)
        self.inv_perm = torch.empty(T * K, **i32)
        self.logits = torch.empty((T, N), dtype=torch.float64, device=device) if keep_logits else None
        self.y_slots = torch.zeros((T * K, d), **f32)
        self.y_shared = torch.zeros((T, d), **f32)
        self.out = torch.empty((T, d), dtype=torch_dtype(s.dtype), device=device)
        self.ws_bytes = spice.spice_workspace_bytes(self.cfg, T)
        if self.ws_bytes == 0:
            raise ValueError(f"invalid configuration for the library: {spice.last_error()}")
        self.ws = torch.zeros(self.ws_bytes, dtype=torch.uint8, device=device)
        # pinned host memory of the exact CPU path: the route kernel writes x and the
        # routing here, the CPU writes the residual that the combine kernel reads
        self.x_host = torch.empty((T, d), dtype=torch_dtype(s.dtype)).pin_memory()
        self.idx_host = torch.empty((T, K), dtype=torch.int32).pin_memory()
        self.w_host = torch.empty((T, K), dtype=torch.float32).pin_memory()
        self.cls_host = torch.empty((T, K), dtype=torch.uint8).pin_memory()
        self.counts_host = torch.zeros(3, dtype=torch.int32).pin_memory()
        self.resid = torch.zeros((T, d), dtype=torch.float32).pin_memory()
        self.ready = torch.zeros(1, dtype=torch.int32).pin_memory()
        self.epoch = 0
        self.host_out = spice.host_out(self.x_host, self.idx_host, self.w_host, self.cls_host, self.counts_host,
                                       self.ready, 0)
        self.host_out_ev = spice.host_out(self.x_host, self.idx_host, self.w_host, self.cls_host, self.counts_host)
        self.e_route = torch.cuda.Event()
        self.wait_ready = False  # the host waits for the ready word (layer call) or for e_route
        # fetch pool of the exact-miss split (Eq. 12: M_fetch), if any
        self.fetch_slots = fetch_slots
        if fetch_slots:
            td = torch_dtype(s.dtype)
            self.w13_fetch = torch.empty((fetch_slots, 2 * s.inter, d), dtype=td, device=device)
            self.w2_fetch = torch.empty((fetch_slots, d, s.inter), dtype=td, device=device)
            self.fetch_expert = torch.full((fetch_slots,), -1, dtype=torch.int32, device=device)
            self.fetch_stage = torch.full((fetch_slots,), -1, dtype=torch.int32).pin_memory()
            self.copy_stream = torch.cuda.Stream(device=device)
            self.e_fetched = torch.cuda.Event()
            self.e_pool_free = torch.cuda.Event()
            self.e_pool_free.record(torch.cuda.current_stream())
        self.last_fetch: List[int] = []
        self.last_host_s = 0.0  # wall time of the last host residual call
        self.last_host_experts = 0  # distinct experts it read

    def _same_format(self, L: DeviceLayer) -> None:
        if L.wfmt != self.cfg.wfmt:
            raise ValueError(f"the layer's expert weights are in format {L.wfmt}, the run was made for {self.cfg.wfmt}")

    # -- the steps, each one C-ABI call ------------------------------------------------
    def route(self, L: DeviceLayer, x: torch.Tensor, conf: Optional[torch.Tensor], T: Optional[int] = None,
              to_host: bool = True, mark: bool = True):
        """Routing + bucketing; with to_host the kernel also fills the pinned host copies.
        e_route marks the end of the call on the stream (mark=False records no event, for
        back-to-back timing; the host then has nothing to wait on)."""
        T = self.T if T is None else T
        spice.moe_route_bucket(self.cfg, T, x, L.wg, L.bias, L.resident_slot, conf, self.logits, self.topk_idx,
                               self.topk_w, self.slot_class, self.offsets, self.perm, self.inv_perm,
                               self.host_out_ev if to_host else None, self.ws, self.ws_bytes)
        if mark:
            self.e_route.record(torch.cuda.current_stream())
        self.wait_ready = False

    def layer_gpu(self, L: DeviceLayer, x: torch.Tensor, conf: Optional[torch.Tensor], T: Optional[int] = None,
                  to_host: bool = True, fuse_lore: bool = True, resid=None, out: bool = False, mark: bool = True):
        """Routing, bucketing and the expert FFN (+ LoRE) as one library call (moe_layer_gpu);
        with to_host the routing's host copies are followed by a new ready word; with out the
        combine runs too, with resid (device or pinned host memory, or None).  mark=False
        records no event after the call (for graph capture)."""
        T = self.T if T is None else T
        ho = None
        self._same_format(L)
        if to_host:
            self.epoch = (self.epoch + 1) & 0x7FFFFFFF
            self.host_out.ready_value = self.epoch
            ho = self.host_out
        la, lb = (L.lore_A, L.lore_B) if fuse_lore else (None, None)
        spice.moe_layer_gpu(self.cfg, T, x, L.wg, L.bias, L.resident_slot, conf, L.w13_pool, L.w2_pool, L.w13s,
                            L.w2s, L.w_sg, la, lb, self.logits, self.topk_idx, self.topk_w, self.slot_class,
                            self.offsets, self.perm, self.inv_perm, self.y_slots, self.y_shared, ho, resid,
                            self.out if out else None, self.ws, self.ws_bytes)
        if mark:
            self.e_route.record(torch.cuda.current_stream())
        self.wait_ready = to_host

    def experts(self, L: DeviceLayer, x: torch.Tensor, T: Optional[int] = None, fuse_lore: bool = True):
        T = self.T if T is None else T
        self._same_format(L)
        la, lb = (L.lore_A, L.lore_B) if fuse_lore else (None, None)
        if L.w_sg is not None:
            spice.moe_expert_ffn_grouped_gated(self.cfg, T, x, self.perm, self.offsets, L.resident_slot, L.w13_pool,
                                               L.w2_pool, L.w13s, L.w2s, L.w_sg, la, lb, self.y_slots,
                                               self.y_shared, self.ws, self.ws_bytes)
        else:
            spice.moe_expert_ffn_grouped(self.cfg, T, x, self.perm, self.offsets, L.resident_slot, L.w13_pool,
                                         L.w2_pool, L.w13s, L.w2s, la, lb, self.y_slots, self.y_shared, self.ws,
                                         self.ws_bytes)

    def lore(self, L: DeviceLayer, x: torch.Tensor, T: Optional[int] = None):
        T = self.T if T is None else T
        spice.lore_surrogate_apply(self.cfg, T, x, self.perm, self.offsets, L.lore_A, L.lore_B, self.y_slots,
                                   self.ws, self.ws_bytes)

    def combine(self, resid: Optional[torch.Tensor], T: Optional[int] = None):
        T = self.T if T is None else T
        spice.moe_combine(self.cfg, T, self.topk_w, self.slot_class, self.inv_perm, self.y_slots, self.y_shared,
                          resid, self.out)

    def exact_host(self, L: DeviceLayer, T: int, n_threads: int = 0, split=None, before_residual=None):
        """Wait for the route kernel's host copies; with a split cost model, fetch the experts
        the planner picks and queue their FFN on the GPU; then the CPU residual of the other
        exact misses into self.resid."""
        if self.wait_ready:
            spice.spice_wait_ready(self.ready, self.epoch)
        else:
            self.e_route.synchronize()
        if before_residual is not None:
            before_residual()
        self.last_fetch = []
        if split is not None and self.fetch_slots:
            cls = self.cls_host[:T].numpy()
            fetch = spice.moe_split_plan(self.cfg, T, self.idx_host[:T].numpy(), cls, split, self.fetch_slots)
            if fetch:
                self.last_fetch = fetch
                with torch.cuda.stream(self.copy_stream):
                    self.copy_stream.wait_event(self.e_pool_free)  # the previous fetched FFN is done with the pool
                    spice.moe_fetch_experts(self.cfg, fetch, L.host_w13, L.host_w2, self.w13_fetch, self.w2_fetch,
                                            self.fetch_slots, self.fetch_expert, self.fetch_stage)
                    self.e_fetched.record(self.copy_stream)
                cur = torch.cuda.current_stream()
                cur.wait_event(self.e_fetched)
                spice.moe_expert_ffn_fetched(self.cfg, T, self.x_cur, self.perm, self.offsets, self.slot_class,
                                             self.fetch_expert, self.w13_fetch, self.w2_fetch, self.fetch_slots,
                                             self.y_slots, self.ws, self.ws_bytes)
                self.e_pool_free.record(cur)
        # the slots left EXACT after the plan are the host's share (timed for the benchmark)
        cls = self.cls_host[:T].numpy()
        self.last_host_experts = len(set(self.idx_host[:T].numpy()[cls == spice.SPICE_CLASS_EXACT].tolist()))
        t0 = time.perf_counter()
        spice.moe_exact_residual_host(self.cfg, T, self.x_host, self.idx_host, self.w_host, self.cls_host,
                                      L.host_w13, L.host_w2, self.resid, n_threads)
        self.last_host_s = time.perf_counter() - t0

    def forward(self, L: DeviceLayer, x: torch.Tensor, conf: Optional[torch.Tensor], T: Optional[int] = None,
                exact: bool = True, n_threads: int = 0, events: Optional[Dict[str, torch.cuda.Event]] = None,
                split=None, after_experts=None, before_residual=None):
        """One layer call: route, FFN + LoRE on the GPU overlapped with the exact CPU residual
        (and, with a split cost model, the fetched exact misses on the GPU), combine.
        after_experts (callable) queues more GPU work right after the FFN, ahead of the host
        residual, e.g. a speculative-prefetch rollout; before_residual (callable) runs on the
        host once the routing's host copies are there, just before the residual."""
        T = self.T if T is None else T
        ev = events or {}
        self.x_cur = x
        if "start" in ev:
            ev["start"].record()
        if self.layer_call:
            self.layer_gpu(L, x, conf, T, to_host=exact)
        else:
            self.route(L, x, conf, T, to_host=exact)
            if "routed" in ev:
                ev["routed"].record()
            self.experts(L, x, T, fuse_lore=True)
        if "experts" in ev:
            ev["experts"].record()
        if after_experts is not None:
            after_experts()
        if exact:
            self.exact_host(L, T, n_threads, split, before_residual)
        if "resid" in ev:
            ev["resid"].record()
        self.combine(self.resid if exact else None, T)
        if "end" in ev:
            ev["end"].record()
        return self.out[:T]

    def flags(self, clear: bool = True) -> int:
        return spice.spice_workspace_flags(self.ws, self.ws_bytes, clear)
