"""Python access to the reference oracle (``liboracle.so``, built from spice_oracle.c).

TEST INFRASTRUCTURE ONLY: a plain fp64 CPU implementation of the SPICE MoE-layer
forward, written from the paper (Sec. 2.1-2.2, 4.2, 4.3; Eq. 1, 6, 7, 9, 11).
Only the tests, the package smoke check and the benchmark's CPU-baseline leg
may import it.  It shares no code with the HIP library.

Each wrapper passes NumPy arrays (fp32, or bf16 bits as uint16) to one C step
and returns NumPy results; ``route`` and ``layer`` run the steps in the order
the paper states them.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "spice_oracle.c")
_LIB_PATH = os.environ.get("SPICE_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")

HIT, LORE, EXACT = 0, 1, 2
CONF_INPUT, CONF_GATE, CONF_GATE_RENORM = 0, 1, 2


def build(force: bool = True) -> str:
    """Compile liboracle.so with gcc (plain -O2, no fast-math, no FMA contraction)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                        "-fno-fast-math", "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        _lib = ctypes.CDLL(_LIB_PATH)
        _declare(_lib)
    return _lib


class Cfg(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int32), ("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32),
                ("inter", ctypes.c_int32), ("shared_inter", ctypes.c_int32), ("lore_rank", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("norm_topk", ctypes.c_int32), ("conf_mode", ctypes.c_int32),
                ("tau", ctypes.c_float), ("wfmt", ctypes.c_int32)]


MXFP4 = 2  # routed experts' weights as MXFP4 blobs (see spice_oracle.h)


def make_cfg(shape, tau: float = 0.5, conf_mode: int = CONF_INPUT, norm_topk: int = 0, wfmt: int = 0) -> Cfg:
    return Cfg(shape.d, shape.n_experts, shape.top_k, shape.inter, shape.shared_inter,
               shape.lore_rank, shape.dtype, norm_topk, conf_mode, tau, wfmt)


def expert_dtype(cfg: Cfg) -> int:
    """Storage of the routed experts' weights: the cfg dtype, or MXFP4."""
    return MXFP4 if cfg.wfmt == MXFP4 else cfg.dtype


_P = ctypes.c_void_p
_I = ctypes.c_int32


def _declare(L: ctypes.CDLL) -> None:
    cp = ctypes.POINTER(Cfg)
    L.orc_router_logits.argtypes = [cp, _I, _P, _P, _P, _P, _P]
    L.orc_gates_topk.argtypes = [cp, _I, _P, _P, _P, _P]
    L.orc_confidence.argtypes = [cp, _I, _P, _P, _P]
    L.orc_classify.argtypes = [cp, _I, _P, _P, _P, _P]
    L.orc_bucket.argtypes = [cp, _I, _P, _P, _P, _P, _P, _P]
    L.orc_swiglu.argtypes = [_I, _I, _I, _P, _P, _P, _P]
    L.orc_lore_delta.argtypes = [_I, _I, _I, _P, _P, _P, _P]
    L.orc_token_output.argtypes = [cp, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]
    L.orc_token_output.restype = _I
    L.orc_token_output_sg.argtypes = [cp, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]
    L.orc_token_output_sg.restype = _I
    L.orc_shared_gate.argtypes = [_I, _I, _P, _P]
    L.orc_shared_gate.restype = ctypes.c_double
    L.orc_mxfp4_elem.argtypes = [_P, _I, _I, _I, _I]
    L.orc_mxfp4_elem.restype = ctypes.c_double
    L.orc_exact_residual.argtypes = [cp, _I, _P, _P, _P, _P, _P, _P, _P]
    L.orc_exact_residual.restype = _I
    L.orc_lru_step.argtypes = [_I, _I, _P, _P, _I, _I, _I, _P, _P, _I, _P, _P]
    L.orc_lru_step.restype = _I
    L.orc_round_to.argtypes = [_I, ctypes.c_double]
    L.orc_round_to.restype = ctypes.c_double
    L.orc_spec_step.argtypes = [cp, _I, _I, _I, ctypes.c_double, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                _P, _P]
    L.orc_spec_step.restype = _I
    L.orc_h_min.argtypes = [ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.c_double, _I,
                            ctypes.c_double]
    L.orc_h_min.restype = _I
    L.orc_prefetch_queue.argtypes = [_I, _I, _I, _I, _P, _P, _I, _P, _P]
    L.orc_lru_prefetch.argtypes = [_I, _I, _P, _P, _I, _I, _P, _I, _P, _P]
    L.orc_lru_prefetch.restype = _I


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def _c(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


def _store(a: np.ndarray, dtype: int) -> np.ndarray:
    if dtype == MXFP4:
        return _c(a, np.uint8)
    return _c(a, np.uint16 if dtype == 1 else np.float32)


def _table(arrs: Sequence[Optional[np.ndarray]], dtype: int):
    keep = [None if a is None else _store(a, dtype) for a in arrs]
    tab = (ctypes.c_void_p * len(keep))(*[None if a is None else a.ctypes.data for a in keep])
    return tab, keep


def router_logits(cfg: Cfg, x, wg, bias=None):
    T = x.shape[0]
    x, wg = _store(x, cfg.dtype), _store(wg, cfg.dtype)
    b = None if bias is None else _c(bias, np.float32)
    z = np.empty((T, cfg.n_experts)); zabs = np.empty((T, cfg.n_experts))
    lib().orc_router_logits(ctypes.byref(cfg), T, _ptr(x), _ptr(wg), _ptr(b), _ptr(z), _ptr(zabs))
    return z, zabs


def gates_topk(cfg: Cfg, z):
    z = _c(z, np.float64)
    T = z.shape[0]
    idx = np.empty((T, cfg.top_k), np.int32); g = np.empty((T, cfg.top_k))
    probs = np.empty((T, cfg.n_experts))
    lib().orc_gates_topk(ctypes.byref(cfg), T, _ptr(z), _ptr(idx), _ptr(g), _ptr(probs))
    return idx, g, probs


def confidence(cfg: Cfg, g, conf_in=None):
    g = _c(g, np.float64)
    T = g.shape[0]
    ci = None if conf_in is None else _c(conf_in, np.float32)
    conf = np.empty((T, cfg.top_k), np.float32)
    lib().orc_confidence(ctypes.byref(cfg), T, _ptr(g), _ptr(ci), _ptr(conf))
    return conf


def classify(cfg: Cfg, idx, resident_mask, conf):
    idx = _c(idx, np.int32); res = _c(resident_mask, np.int32); conf = _c(conf, np.float32)
    cls = np.empty(idx.shape, np.uint8)
    lib().orc_classify(ctypes.byref(cfg), idx.shape[0], _ptr(idx), _ptr(res), _ptr(conf), _ptr(cls))
    return cls


def bucket(cfg: Cfg, idx, cls):
    idx = _c(idx, np.int32); cls = _c(cls, np.uint8)
    T = idx.shape[0]
    S = T * cfg.top_k
    offsets = np.empty((3, cfg.n_experts + 1), np.int32)
    perm = np.empty(S, np.int32); inv = np.empty(S, np.int32); counts = np.empty(3, np.int32)
    lib().orc_bucket(ctypes.byref(cfg), T, _ptr(idx), _ptr(cls), _ptr(offsets), _ptr(perm), _ptr(inv),
                     _ptr(counts))
    return offsets, perm, inv, counts


def mxfp4_elem(blob, rows: int, K: int, r: int, c: int) -> float:
    b = _c(blob, np.uint8)
    return lib().orc_mxfp4_elem(_ptr(b), rows, K, r, c)


def swiglu(d: int, inter: int, dtype: int, w13, w2, x64):
    w13, w2 = _store(w13, dtype), _store(w2, dtype)
    x64 = _c(x64, np.float64); y = np.empty(d)
    lib().orc_swiglu(d, inter, dtype, _ptr(w13), _ptr(w2), _ptr(x64), _ptr(y))
    return y


def lore_delta(d: int, r: int, dtype: int, A, B, x64):
    A, B = _store(A, dtype), _store(B, dtype)
    x64 = _c(x64, np.float64); y = np.empty(d)
    lib().orc_lore_delta(d, r, dtype, _ptr(A), _ptr(B), _ptr(x64), _ptr(y))
    return y


def shared_gate(cfg: Cfg, x_row, w_sg) -> float:
    """The shared block's output gate sigmoid(w_sg . x) for one token."""
    x_row = _store(x_row, cfg.dtype); w = _store(w_sg, cfg.dtype)
    return lib().orc_shared_gate(cfg.d, cfg.dtype, _ptr(x_row), _ptr(w))


def token_output(cfg: Cfg, x_row, idx_t, g_t, cls_t, w13, w2, w13s, w2s, lA, lB, w_sg=None):
    """Per-token layer output.  w13/w2/lA/lB: length-N sequences (None where unused);
    w_sg: the shared block's gate vector [d], or None for an ungated shared block."""
    x_row = _store(x_row, cfg.dtype)
    idx_t = _c(idx_t, np.int32); g_t = _c(g_t, np.float64); cls_t = _c(cls_t, np.uint8)
    t13, k1 = _table(w13, expert_dtype(cfg)); t2, k2 = _table(w2, expert_dtype(cfg))
    tA, k3 = _table(lA, cfg.dtype); tB, k4 = _table(lB, cfg.dtype)
    s13, s2 = _store(w13s, cfg.dtype), _store(w2s, cfg.dtype)
    sg = None if w_sg is None else _store(w_sg, cfg.dtype)
    out = np.empty(cfg.d); ys = np.empty(cfg.d); yslot = np.empty((cfg.top_k, cfg.d))
    rc = lib().orc_token_output_sg(ctypes.byref(cfg), _ptr(x_row), _ptr(idx_t), _ptr(g_t), _ptr(cls_t),
                                   t13, t2, _ptr(s13), _ptr(s2), _ptr(sg), tA, tB, _ptr(out), _ptr(ys),
                                   _ptr(yslot))
    if rc != 0:
        raise ValueError("oracle: a needed expert weight was not supplied")
    return out, ys, yslot


def exact_residual(cfg: Cfg, x, idx, g, cls, w13, w2):
    T = x.shape[0]
    x = _store(x, cfg.dtype); idx = _c(idx, np.int32); g = _c(g, np.float64); cls = _c(cls, np.uint8)
    t13, k1 = _table(w13, expert_dtype(cfg)); t2, k2 = _table(w2, expert_dtype(cfg))
    resid = np.empty((T, cfg.d))
    rc = lib().orc_exact_residual(ctypes.byref(cfg), T, _ptr(x), _ptr(idx), _ptr(g), _ptr(cls), t13, t2,
                                  _ptr(resid))
    if rc != 0:
        raise ValueError("oracle: a needed expert weight was not supplied")
    return resid


class LRUState:
    """Per-layer cache state: slot_expert[C], last_use[C]."""

    def __init__(self, n_experts: int, C: int, initial=None):
        self.N, self.C = n_experts, C
        init = list(range(C)) if initial is None else list(initial)
        self.slot_expert = np.array(init, dtype=np.int32)
        self.last_use = np.full(C, -1, dtype=np.int32)

    def step(self, step: int, idx, cls, max_admit: int):
        idx = _c(idx, np.int32); cls = _c(cls, np.uint8)
        T, K = idx.shape
        adm = np.empty(max(max_admit, 1), np.int32); ev = np.empty(max(max_admit, 1), np.int32)
        n = lib().orc_lru_step(self.N, self.C, _ptr(self.slot_expert), _ptr(self.last_use), step, T, K,
                               _ptr(idx), _ptr(cls), max_admit, _ptr(adm), _ptr(ev))
        return adm[:n].copy(), ev[:n].copy()

    def prefetch(self, step: int, experts, max_prefetch: int):
        """Speculative admissions (the prefetch queue of one future layer)."""
        ex = _c(experts, np.int32).reshape(-1)
        adm = np.empty(max(max_prefetch, 1), np.int32); ev = np.empty(max(max_prefetch, 1), np.int32)
        n = lib().orc_lru_prefetch(self.N, self.C, _ptr(self.slot_expert), _ptr(self.last_use), step, len(ex),
                                   _ptr(ex), max_prefetch, _ptr(adm), _ptr(ev))
        return adm[:n].copy(), ev[:n].copy()

    def resident_mask(self) -> np.ndarray:
        m = np.zeros(self.N, np.int32)
        m[self.slot_expert[self.slot_expert >= 0]] = 1
        return m


def route(cfg: Cfg, x, wg, bias, resident_mask, conf_in=None) -> Dict[str, np.ndarray]:
    """Routing, gating, confidence, classification and bucketing for all tokens."""
    z, zabs = router_logits(cfg, x, wg, bias)
    idx, g, probs = gates_topk(cfg, z)
    conf = confidence(cfg, g, conf_in)
    cls = classify(cfg, idx, resident_mask, conf)
    offsets, perm, inv, counts = bucket(cfg, idx, cls)
    return dict(z=z, zabs=zabs, idx=idx, g=g, probs=probs, conf=conf, cls=cls, offsets=offsets,
                perm=perm, inv_perm=inv, counts=counts)


def layer(cfg: Cfg, x, wg, bias, resident_mask, conf_in, w13, w2, w13s, w2s, lA, lB,
          tokens: Optional[Sequence[int]] = None, w_sg=None) -> Dict[str, np.ndarray]:
    """Whole layer: routing for all tokens, outputs for ``tokens`` (default: all); w_sg
    gates the shared block (None: ungated)."""
    r = route(cfg, x, wg, bias, resident_mask, conf_in)
    T = x.shape[0]
    toks = list(range(T)) if tokens is None else list(tokens)
    out = np.empty((len(toks), cfg.d)); ys = np.empty((len(toks), cfg.d))
    yslot = np.empty((len(toks), cfg.top_k, cfg.d))
    for i, t in enumerate(toks):
        out[i], ys[i], yslot[i] = token_output(cfg, x[t], r["idx"][t], r["g"][t], r["cls"][t],
                                               w13, w2, w13s, w2s, lA, lB, w_sg)
    r.update(out=out, y_shared=ys, y_slot=yslot, tokens=np.array(toks, np.int32))
    return r


# ---- speculative prefetching (Sec. 4.1, Eq. 2-5, Alg. 1) -----------------------------------

def round_to(dtype: int, v: float) -> float:
    return lib().orc_round_to(dtype, float(v))


def spec_step(cfg: Cfg, h_in, delta: int, l_min: int, tau: float, last: bool, wg, bias, w13s, w2s, lA, lB,
              halted):
    """One depth of the draft rollout (Alg. 1) for every token.  h_in: storage array [T][d];
    halted: int32 [T], updated in place.  Returns (pred_idx, pred_prob, conf, h_out)."""
    h_in = _store(h_in, cfg.dtype)
    T = h_in.shape[0]
    wg = _store(wg, cfg.dtype)
    b = None if bias is None else _c(bias, np.float32)
    tA, k1 = _table(lA, cfg.dtype); tB, k2 = _table(lB, cfg.dtype)
    s13, s2 = _store(w13s, cfg.dtype), _store(w2s, cfg.dtype)
    assert halted.dtype == np.int32 and halted.flags.c_contiguous
    pidx = np.empty((T, cfg.top_k), np.int32); pprob = np.empty((T, cfg.top_k)); conf = np.empty(T)
    h_out = np.empty_like(h_in)
    rc = lib().orc_spec_step(ctypes.byref(cfg), T, delta, l_min, tau, int(last), _ptr(h_in), _ptr(wg), _ptr(b),
                             _ptr(s13), _ptr(s2), tA, tB, _ptr(halted), _ptr(pidx), _ptr(pprob), _ptr(conf),
                             _ptr(h_out))
    if rc != 0:
        raise ValueError("oracle: a needed LoRE factor was not supplied")
    return pidx, pprob, conf, h_out


def spec_rollout(cfg: Cfg, x, layers, l_min: int, tau: float):
    """Alg. 1 from anchor x over len(layers) future layers; layers[j] = dict(wg, bias, w13s,
    w2s, lA, lB) of layer l + 1 + j.  Returns per-depth predictions, confidences, the draft
    states after each depth, and each token's last enqueued depth."""
    T = x.shape[0]
    halted = np.zeros(T, np.int32)
    h = _store(x, cfg.dtype)
    out = dict(idx=[], prob=[], conf=[], h=[])
    depth = np.zeros(T, np.int32)
    for j, L in enumerate(layers):
        delta = j + 1
        was = halted.copy()
        pidx, pprob, conf, h = spec_step(cfg, h, delta, l_min, tau, delta == len(layers), L["wg"], L.get("bias"),
                                         L["w13s"], L["w2s"], L["lA"], L["lB"], halted)
        depth[was == 0] = delta
        out["idx"].append(pidx); out["prob"].append(pprob); out["conf"].append(conf); out["h"].append(h)
    return {k: np.stack(v) for k, v in out.items()} | dict(depth=depth)


def h_min(P: float, M_e: float, B: float, t_attn: float, K: int, t_expert: float) -> int:
    return lib().orc_h_min(P, M_e, B, t_attn, K, t_expert)


def prefetch_queue(n_experts: int, pred_idx, pred_prob, max_per_depth: int):
    """Per-depth issue lists of the prefetch intents (Eq. 3)."""
    pidx = _c(pred_idx, np.int32); pprob = _c(pred_prob, np.float64)
    D, T, K = pidx.shape
    ex = np.empty((D, max(max_per_depth, 1)), np.int32); cnt = np.empty(D, np.int32)
    lib().orc_prefetch_queue(n_experts, D, T, K, _ptr(pidx), _ptr(pprob), max_per_depth, _ptr(ex), _ptr(cnt))
    return [ex[i, :cnt[i]].tolist() for i in range(D)]


# ---- LoRE calibration fit (Sec. 4.2, Eq. 8-10) ---------------------------------------------

def lore_fit(X, Y, r: int):
    """The minimiser of Eq. 10, sum_t || y_t - B A x_t ||^2 over A [r][d], B [d][r], in fp64.

    X [n][d] calibration hidden states (rows), Y [n][d] their residual targets
    E_e(x) - S(x) (Eq. 8).  This is reduced-rank regression: the least-squares map
    W_ols = Y^T (X^T)^+ (minimum norm), its fitted values F = W_ols X^T, and the best rank-r
    approximation of F from its r leading left singular vectors U_r (Eckart-Young), so
    B A = U_r U_r^T W_ols with B = U_r, A = U_r^T W_ols.  Returns (A, B, loss)."""
    X = np.asarray(X, np.float64)
    Y = np.asarray(Y, np.float64)
    Xt, Yt = X.T, Y.T  # columns are tokens
    W_ols = Yt @ np.linalg.pinv(Xt)
    F = W_ols @ Xt
    U, _, _ = np.linalg.svd(F, full_matrices=False)
    Ur = U[:, :r]
    B = Ur
    A = Ur.T @ W_ols
    R = Yt - B @ (A @ Xt)
    return A, B, float((R * R).sum())


def lore_loss(X, Y, A, B) -> float:
    """Eq. 10's objective for given factors."""
    X = np.asarray(X, np.float64); Y = np.asarray(Y, np.float64)
    R = Y.T - np.asarray(B, np.float64) @ (np.asarray(A, np.float64) @ X.T)
    return float((R * R).sum())
