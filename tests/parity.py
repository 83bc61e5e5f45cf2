"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI and
the oracle on the same seeded inputs, and compare.

Bars: routing, classes, offsets, perm and inv_perm bit-exact; gates within
fp32 rounding; float outputs within a per-token relative error
max|out - ref| / max|ref| of 1e-4 (fp32 layers) or 2e-2 (bf16 layers,
fp32 accumulation).
"""
from __future__ import annotations

import sys
from typing import Optional, Sequence

import numpy as np
import torch

import oracle as orc
from paper_2608_21240_amd import layer as LY, synth, workloads as W

HIT, LORE, EXACT = 0, 1, 2


def say(msg: str) -> None:
    print(f"[parity] {msg}", flush=True)
    sys.stdout.flush()


def tol_for(shape) -> float:
    return 1e-4 if shape.dtype == W.DTYPE_F32 else 2e-2


def rel_err(out: np.ndarray, ref: np.ndarray) -> np.ndarray:
    out = np.asarray(out, np.float64).reshape(ref.shape[0], -1)
    ref = np.asarray(ref, np.float64).reshape(ref.shape[0], -1)
    return np.abs(out - ref).max(axis=1) / np.maximum(np.abs(ref).max(axis=1), 1e-30)


def to_np(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def as_f64(a: np.ndarray, dtype: int) -> np.ndarray:
    return synth.as_f32(a, dtype).astype(np.float64)


class Case:
    """One parity case: host weights, device layer, inputs and both results."""

    def __init__(self, wl: W.Workload, T: Optional[int] = None, resident: Optional[Sequence[int]] = None,
                 host: Optional[LY.HostLayer] = None, conf: Optional[np.ndarray] = None, x: Optional[np.ndarray] = None,
                 step: int = 0, n_slots: Optional[int] = None):
        self.wl = wl
        self.shape = wl.shape
        self.T = wl.tokens if T is None else T
        self.host = host if host is not None else LY.HostLayer(wl, 0, resident)
        if resident is not None and host is not None:
            self.host.resident = list(resident)
        self.x = synth.gen_x(wl, 0, step, self.T) if x is None else x
        self.conf = synth.gen_conf(wl, 0, step, self.T) if conf is None else conf
        self.n_slots = n_slots

    # ---------------------------------------------------------------- HIP path
    def run_gpu(self, dev: Optional[LY.DeviceLayer] = None, fused: bool = True, exact: bool = True,
                run: Optional[LY.LayerRun] = None, n_threads: int = 0, split=None, fetch_slots: int = 0,
                layer_call: bool = True):
        """fused: the whole layer through LayerRun.forward (moe_layer_gpu when layer_call, else the
        separate routing and FFN calls); not fused: routing, FFN without LoRE, lore_surrogate_apply,
        the host residual and the combine as separate calls."""
        s = self.shape
        self.dev = dev if dev is not None else LY.DeviceLayer(self.host, n_slots=self.n_slots)
        self.run = run if run is not None else LY.LayerRun(s, self.T, self.dev.C, tau=self.wl.tau,
                                                            conf_mode=self.wl.conf_mode, norm_topk=self.wl.norm_topk,
                                                            keep_logits=True, fetch_slots=fetch_slots,
                                                            wfmt=self.wl.wfmt, layer_call=layer_call)
        R = self.run
        xd = LY.to_tensor(self.x, s.dtype, "cuda")
        conf = torch.from_numpy(np.ascontiguousarray(self.conf)).cuda()
        R.y_slots.zero_(); R.y_shared.zero_()
        if fused:
            R.forward(self.dev, xd, conf, self.T, exact=exact, n_threads=n_threads, split=split)
        else:
            R.route(self.dev, xd, conf, self.T, to_host=exact)
            R.experts(self.dev, xd, self.T, fuse_lore=False)
            R.lore(self.dev, xd, self.T)
            if exact:
                R.exact_host(self.dev, self.T, n_threads)
            R.combine(R.resid if exact else None, self.T)
        torch.cuda.synchronize()
        T, K = self.T, s.top_k
        self.g = dict(
            logits=to_np(R.logits[:T]), idx=to_np(R.topk_idx[:T]), w=to_np(R.topk_w[:T]),
            cls=to_np(R.slot_class[:T]), offsets=to_np(R.offsets), perm=to_np(R.perm[: T * K]),
            inv_perm=to_np(R.inv_perm[: T * K]), y_slots=to_np(R.y_slots[: T * K]),
            y_shared=to_np(R.y_shared[:T]), resid=to_np(R.resid[:T]), out=to_np(R.out[:T]),
            flags=R.flags(clear=True))
        return self.g

    # ------------------------------------------------------------------ oracle
    def run_oracle(self, tokens: Optional[Sequence[int]] = None):
        s, wl = self.shape, self.wl
        cfg = orc.make_cfg(s, tau=wl.tau, conf_mode=wl.conf_mode, norm_topk=wl.norm_topk, wfmt=wl.wfmt)
        self.cfg = cfg
        res = self.host.resident_mask()
        r = orc.route(cfg, self.x, self.host.wg, self.host.bias, res, self.conf)
        toks = list(range(self.T)) if tokens is None else list(tokens)
        need = sorted(set(r["idx"][toks][r["cls"][toks] != LORE].tolist()))
        need_l = sorted(set(r["idx"][toks][r["cls"][toks] == LORE].tolist()))
        w13, w2, la, lb = self.host.tables(need, need_l)
        out = np.empty((len(toks), s.d)); ys = np.empty((len(toks), s.d)); yslot = np.empty((len(toks), s.top_k, s.d))
        for i, t in enumerate(toks):
            out[i], ys[i], yslot[i] = orc.token_output(cfg, self.x[t], r["idx"][t], r["g"][t], r["cls"][t], w13, w2,
                                                       self.host.w13s, self.host.w2s, la, lb, self.host.w_sg)
        r.update(out=out, y_shared=ys, y_slot=yslot, tokens=np.array(toks))
        exact_e = sorted(set(r["idx"][toks][r["cls"][toks] == EXACT].tolist()))
        e13, e2, _, _ = self.host.tables(exact_e, [])
        sub = np.where(np.isin(np.arange(self.T), toks)[:, None], r["cls"], LORE).astype(np.uint8)
        r["resid"] = orc.exact_residual(cfg, self.x, r["idx"], r["g"], sub, e13, e2)[toks]
        self.o = r
        return r

    # ----------------------------------------------------------------- checks
    def check_routing(self):
        g, o, s = self.g, self.o, self.shape
        # logits within the summation-rounding bound of fp64 (both sides)
        bound = 2.0 * s.d * 2.0 ** -53 * o["zabs"] + 1e-300
        assert np.all(np.abs(g["logits"] - o["z"]) <= 2 * bound + 1e-12 * np.abs(o["z"])), "logits"
        # certification: the oracle's order among the first K+1 logits cannot flip
        zs = -np.sort(-o["z"], axis=1)[:, : s.top_k + 1]
        gaps = np.abs(np.diff(zs, axis=1))
        certified = np.all((gaps > 4 * bound.max(axis=1, keepdims=True)) | (gaps == 0), axis=1)
        assert certified.all(), f"{(~certified).sum()} uncertified tokens"
        assert np.array_equal(g["idx"], o["idx"]), "topk_idx"
        assert np.allclose(g["w"], o["g"].astype(np.float32), rtol=2e-7, atol=0), "topk_w"
        assert np.array_equal(g["cls"], o["cls"]), "slot_class"
        assert np.array_equal(g["offsets"], o["offsets"]), "offsets"
        assert np.array_equal(g["perm"], o["perm"]), "perm"
        assert np.array_equal(g["inv_perm"], o["inv_perm"]), "inv_perm"
        assert g["flags"] == 0, f"device flags {g['flags']}"

    def check_outputs(self, exact: bool = True):
        g, o, s = self.g, self.o, self.shape
        tol = tol_for(s)
        toks = o["tokens"]
        errs = {}
        errs["y_shared"] = rel_err(g["y_shared"][toks], o["y_shared"])
        rows, refs = [], []
        for i, t in enumerate(toks):
            for k in range(s.top_k):
                if o["cls"][t, k] in (HIT, LORE):
                    rows.append(g["y_slots"][g["inv_perm"][t * s.top_k + k]])
                    refs.append(o["y_slot"][i, k])
        if rows:
            errs["y_slots"] = rel_err(np.array(rows), np.array(refs))
        if exact:
            has = (o["cls"][toks] == EXACT).any(axis=1)
            if has.any():
                errs["resid"] = rel_err(g["resid"][toks][has], o["resid"][has])
            out = g["out"][toks]
            outf = synth.as_f32(out, s.dtype) if s.dtype == W.DTYPE_BF16 else out
            errs["out"] = rel_err(outf, o["out"])
        summary = {k: (float(np.median(v)), float(v.max())) for k, v in errs.items()}
        say(f"rel errors (median, max): {summary}")
        for k, v in errs.items():
            assert v.max() <= tol, f"{k}: max rel err {v.max():.3e} > {tol}"
        return summary
