"""A decode stack of independent MoE layers, each with its own LRU-managed GPU
expert cache (the library's moe_cache_* handle).

Per layer: its own router, its own per-step confidences, its own slot pool and
resident_slot.  The expert, shared-block and LoRE weights are drawn once and
used by every layer; they do not change what the cache does, which depends on
routing only.  Each step feeds one x[T][d] draw to every layer (the layers are
not chained).  Per layer call: route, FFN + LoRE, exact residual on the host,
combine (LayerRun.forward), then the cache update, whose copies overlap the
following layers; optionally the speculative prefetches of the next layers.
"""
from __future__ import annotations

import threading
from types import SimpleNamespace
from typing import Dict, List, Optional

import numpy as np
import torch

from . import spice, synth
from .layer import HostLayer, LayerRun, to_tensor, torch_dtype
from .workloads import Workload


class StackModel:
    """Host and device weights of the stack (see the module docstring)."""

    def __init__(self, wl: Workload, n_layers: Optional[int] = None, device: str = "cuda"):
        s = wl.shape
        self.wl, self.shape = wl, s
        self.L = wl.layers if n_layers is None else n_layers
        self.C = wl.cache_slots
        self.base = HostLayer(wl, layer=0, resident=[])
        N, dt = s.n_experts, s.dtype
        # host experts, pinned so that admissions copy asynchronously
        self.w13_host: List[torch.Tensor] = []
        self.w2_host: List[torch.Tensor] = []
        for e in range(N):
            w13, w2 = self.base.expert(e)
            self.w13_host.append(to_tensor(w13, dt, pin=True))
            self.w2_host.append(to_tensor(w2, dt, pin=True))
        self.base._experts.clear()
        self.wg = [to_tensor(synth.gen_router(wl, l), dt, device) for l in range(self.L)]
        self.w13s = to_tensor(self.base.w13s, dt, device)
        self.w2s = to_tensor(self.base.w2s, dt, device)
        r = max(s.lore_rank, 1)
        td = torch_dtype(dt)
        self.lore_A = torch.empty((N, r, s.d), dtype=td, device=device)
        self.lore_B = torch.empty((N, s.d, r), dtype=td, device=device)
        if s.lore_rank > 0:
            for e in range(N):
                A, B = self.base.lore(e)
                self.lore_A[e].copy_(to_tensor(A, dt))
                self.lore_B[e].copy_(to_tensor(B, dt))
        self.w13_pool = [torch.empty((self.C, 2 * s.inter, s.d), dtype=td, device=device) for _ in range(self.L)]
        self.w2_pool = [torch.empty((self.C, s.d, s.inter), dtype=td, device=device) for _ in range(self.L)]
        self.resident_slot = [torch.full((N,), -1, dtype=torch.int32, device=device) for _ in range(self.L)]
        self.initial = np.tile(np.arange(self.C, dtype=np.int32), (self.L, 1))

    def host_storage(self, e: int):
        """(w13, w2) of expert e as storage arrays viewing the pinned host copies."""
        def st(t):
            return t.view(torch.int16).numpy().view(np.uint16) if self.shape.dtype else t.numpy()
        return st(self.w13_host[e]), st(self.w2_host[e])

    def layer_view(self, l: int) -> SimpleNamespace:
        """What LayerRun needs of layer l."""
        return SimpleNamespace(wg=self.wg[l], bias=None, resident_slot=self.resident_slot[l],
                               w13_pool=self.w13_pool[l], w2_pool=self.w2_pool[l], w13s=self.w13s, w2s=self.w2s,
                               lore_A=self.lore_A, lore_B=self.lore_B, host_w13=self.w13_host, host_w2=self.w2_host,
                               w_sg=None, wfmt=spice.SPICE_WFMT_DTYPE)


class StackRun:
    """Runs decode steps over the stack and records the cache's behaviour.

    prefetch (optional): dict(depth, l_min, tau, max_prefetch) turns on speculative
    prefetching (Sec. 4.1): after each layer's FFN the draft rollout of Alg. 1 runs from
    the layer's input over the next `depth` layers (overlapped with the host residual),
    and after the layer's own admissions the cache takes up to max_prefetch predicted
    experts per future layer, in issue order, from lists cut at the cache size."""

    def __init__(self, model: StackModel, max_admit: int = 4, n_threads: int = 0, prefetch: Optional[Dict] = None):
        wl, s = model.wl, model.shape
        self.m, self.max_admit, self.n_threads = model, max_admit, n_threads
        self.prefetch = prefetch
        self.spec = None
        self.spec_events: Optional[List] = None  # set to [] to time every rollout
        if prefetch:
            from .spec import SpecRollout
            self.spec = SpecRollout(s, wl.tokens, prefetch["depth"])
        self.T = wl.tokens
        self.run = LayerRun(s, self.T, model.C, tau=wl.tau, conf_mode=wl.conf_mode, norm_topk=wl.norm_topk)
        self.cfg = self.run.cfg
        L, N = model.L, s.n_experts
        self.copy_stream = torch.cuda.Stream()
        self.cache = spice.ExpertCache(
            self.cfg, L, model.initial,
            w13_host=[model.w13_host[e] for _ in range(L) for e in range(N)],
            w2_host=[model.w2_host[e] for _ in range(L) for e in range(N)],
            w13_pool=model.w13_pool, w2_pool=model.w2_pool, resident_slot=model.resident_slot, load=True)
        self.views = [model.layer_view(l) for l in range(L)]
        self.trace: List[Dict] = []

    def step(self, step: int, x: torch.Tensor, confs: List[torch.Tensor], record: bool = True,
             outputs: Optional[Dict] = None) -> None:
        """One decode step through every layer.  outputs: {layer: tensor to copy the output into}."""
        K, L = self.m.shape.top_k, self.m.L
        pf = self.prefetch
        for l in range(L):
            self.cache.wait(l)
            future = self.views[l + 1: l + 1 + pf["depth"]] if pf else []
            hook = (lambda: self._rollout(future, x)) if future else None
            box: Dict = {}
            helper = None
            if future:
                # the prefetches go out from a helper thread as soon as the rollout is done,
                # while this thread computes the layer's host residual; their copies wait
                # only for the future layers' own last calls, so they overlap this layer
                helper = threading.Thread(target=self._issue_prefetch, args=(l, step, box))
            out = self.run.forward(self.views[l], x, confs[l], self.T, n_threads=self.n_threads, after_experts=hook,
                                   before_residual=helper.start if helper else None)
            if helper is not None:
                helper.join()
                if "error" in box:
                    raise box["error"]
            if outputs is not None and l in outputs:
                outputs[l].copy_(out)
            idx = self.run.idx_host[: self.T].numpy()
            cls = self.run.cls_host[: self.T].numpy()
            adm, ev = self.cache.step(l, step, idx, cls, self.max_admit, copy_stream=self.copy_stream)
            queue, pre = box.get("queue", []), box.get("prefetched", [])
            if record:
                cnt = np.bincount(cls.ravel(), minlength=3)
                self.trace.append(dict(step=step, layer=l, idx=idx.copy(), cls=cls.copy(), admitted=adm,
                                       evicted=ev, hit=int(cnt[0]), lore=int(cnt[1]), exact=int(cnt[2]),
                                       miss_rate=float(cnt[1] + cnt[2]) / (self.T * K),
                                       lore_split=float(cnt[1]) / max(int(cnt[1] + cnt[2]), 1),
                                       queue=queue, prefetched=pre))

    def _issue_prefetch(self, l: int, step: int, box: Dict) -> None:
        """Issue lists cut at the cache size (a prefetch never evicts one of a layer's C
        most likely experts to make room for another) into the next layers' caches."""
        try:
            queue = self.spec.queue(self.m.C)
            box["queue"] = queue
            box["prefetched"] = [self.cache.prefetch(l + 1 + j, step, q, self.prefetch["max_prefetch"],
                                                     copy_stream=self.copy_stream) for j, q in enumerate(queue)]
        except BaseException as ex:  # re-raised on the calling thread
            box["error"] = ex

    def _rollout(self, future, x) -> None:
        pf = self.prefetch
        if self.spec_events is None:
            self.spec.run(future, x, pf["l_min"], pf["tau"])
            return
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        self.spec.run(future, x, pf["l_min"], pf["tau"])
        e1.record()
        self.spec_events.append((e0, e1, len(future)))

    def close(self) -> None:
        torch.cuda.synchronize()
        self.cache.close()
