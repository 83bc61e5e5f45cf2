"""ctypes binding of libspice_moe.so: the C-ABI entry points under the same names.

Argument marshalling only.  Buffers may be passed as torch tensors (their
data_ptr() is used), NumPy arrays (host buffers), raw integer addresses or
None.  Streams default to torch's current HIP stream.  A non-zero status
raises SpiceError with the library's message.  There is no fallback: if the
library is missing, loading raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libspice_moe.so")

SPICE_OK, SPICE_ERR_INVALID, SPICE_ERR_UNSUPPORTED, SPICE_ERR_HIP, SPICE_ERR_WORKSPACE, SPICE_ERR_INTERNAL = (
    0, -1, -2, -3, -4, -5)
SPICE_F32, SPICE_BF16 = 0, 1
SPICE_CONF_INPUT, SPICE_CONF_GATE, SPICE_CONF_GATE_RENORM = 0, 1, 2
SPICE_WFMT_DTYPE, SPICE_WFMT_MXFP4 = 0, 2
SPICE_CLASS_HIT, SPICE_CLASS_LORE, SPICE_CLASS_EXACT, SPICE_CLASS_EXACT_GPU = 0, 1, 2, 3
SPICE_MAX_EXPERTS, SPICE_MAX_TOKENS, SPICE_MAX_LORE_RANK = 256, 65536, 256
SPICE_WS_CONTROL_BYTES = 131072
SPICE_FLAG_BAD_SLOT, SPICE_FLAG_BAD_INDEX = 1, 2

# Every function the header declares (checked against include/spice_moe.h by the tests).
EXPORTS = (
    "spice_workspace_bytes", "spice_workspace_init", "spice_workspace_flags",
    "moe_route_bucket", "moe_expert_ffn_grouped", "moe_expert_ffn_grouped_gated", "lore_surrogate_apply",
    "moe_combine", "moe_layer_gpu", "moe_layer_gpu_noalloc",
    "moe_exact_residual_host", "moe_cache_create", "moe_cache_step", "moe_cache_wait", "moe_cache_state",
    "moe_cache_destroy", "moe_split_plan", "moe_fetch_experts", "moe_expert_ffn_fetched",
    "moe_spec_update", "moe_prefetch_h_min", "moe_prefetch_queue", "moe_cache_prefetch",
    "spice_lore_fit_workspace_bytes", "moe_lore_fit",
    "spice_wait_ready", "spice_status_string", "spice_last_error",
)


class SpiceError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn}: status {status}: {msg}")
        self.status = status


class spice_moe_cfg_t(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int32), ("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32),
                ("inter", ctypes.c_int32), ("shared_inter", ctypes.c_int32), ("lore_rank", ctypes.c_int32),
                ("n_slots", ctypes.c_int32), ("dtype", ctypes.c_int32), ("norm_topk", ctypes.c_int32),
                ("conf_mode", ctypes.c_int32), ("tau", ctypes.c_float), ("wfmt", ctypes.c_int32)]


class spice_split_cost_t(ctypes.Structure):
    _fields_ = [("cpu_bytes_per_s", ctypes.c_double), ("cpu_flops_per_s", ctypes.c_double),
                ("pcie_bytes_per_s", ctypes.c_double), ("gpu_fixed_s", ctypes.c_double),
                ("margin", ctypes.c_double)]


class spice_spec_host_t(ctypes.Structure):
    _fields_ = [("pred_idx", ctypes.c_void_p), ("pred_prob", ctypes.c_void_p), ("conf", ctypes.c_void_p)]


class spice_host_out_t(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("topk_idx", ctypes.c_void_p), ("topk_w", ctypes.c_void_p),
                ("slot_class", ctypes.c_void_p), ("class_counts", ctypes.c_void_p), ("ready", ctypes.c_void_p),
                ("ready_value", ctypes.c_uint32)]


def host_out(x=None, topk_idx=None, topk_w=None, slot_class=None, class_counts=None, ready=None,
             ready_value: int = 0) -> spice_host_out_t:
    """Pinned host buffers (tensors, arrays or addresses) for the routing's host copies."""
    return spice_host_out_t(_p(x), _p(topk_idx), _p(topk_w), _p(slot_class), _p(class_counts), _p(ready),
                            ready_value & 0xFFFFFFFF)


def make_cfg(shape, n_slots: int, tau: float = 0.5, conf_mode: int = SPICE_CONF_INPUT,
             norm_topk: int = 0, wfmt: int = 0) -> spice_moe_cfg_t:
    return spice_moe_cfg_t(shape.d, shape.n_experts, shape.top_k, shape.inter, shape.shared_inter,
                           shape.lore_rank, n_slots, shape.dtype, norm_topk, conf_mode, tau, wfmt)


_lib: Optional[ctypes.CDLL] = None
_P, _I, _Z = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2608_21240_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        C = ctypes.POINTER(spice_moe_cfg_t)
        sig = {
            "spice_workspace_bytes": (_Z, [C, _I]),
            "spice_workspace_init": (_I, [_P, _Z, _P]),
            "spice_workspace_flags": (_I, [_P, _Z, ctypes.POINTER(ctypes.c_uint32), _I, _P]),
            "moe_route_bucket": (_I, [C, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                      ctypes.POINTER(spice_host_out_t), _P, _Z, _P]),
            "moe_expert_ffn_grouped": (_I, [C, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _Z, _P]),
            "moe_expert_ffn_grouped_gated": (_I, [C, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _Z,
                                                  _P]),
            "lore_surrogate_apply": (_I, [C, _I, _P, _P, _P, _P, _P, _P, _P, _Z, _P]),
            "moe_combine": (_I, [C, _I, _P, _P, _P, _P, _P, _P, _P, _P]),
            "moe_layer_gpu": (_I, [C, _I] + [_P] * 21 + [ctypes.POINTER(spice_host_out_t), _P, _P, _P, _Z, _P]),
            "moe_layer_gpu_noalloc": (_I, [C, _I] + [_P] * 21 + [ctypes.POINTER(spice_host_out_t), _P, _P, _P]),
            "moe_exact_residual_host": (_I, [C, _I, _P, _P, _P, _P, _P, _P, _P, _I]),
            "moe_cache_create": (_I, [C, _I, _P, _P, _P, _P, _P, _P, _I, _P, ctypes.POINTER(_P)]),
            "moe_cache_step": (_I, [_P, _I, _I, _I, _P, _P, _I, _P, _P, ctypes.POINTER(_I), _P, _P]),
            "moe_cache_wait": (_I, [_P, _I, _P]),
            "moe_cache_state": (_I, [_P, _I, _P, _P]),
            "moe_cache_destroy": (None, [_P]),
            "moe_split_plan": (_I, [C, _I, _P, _P, ctypes.POINTER(spice_split_cost_t), _I, _P,
                                    ctypes.POINTER(_I)]),
            "moe_fetch_experts": (_I, [C, _I, _P, _P, _P, _P, _P, _I, _P, _P, _P]),
            "moe_expert_ffn_fetched": (_I, [C, _I, _P, _P, _P, _P, _P, _P, _P, _I, _P, _P, _Z, _P]),
            "moe_spec_update": (_I, [C, _I, _I, _I, ctypes.c_float, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                     ctypes.POINTER(spice_spec_host_t), _P, _Z, _P]),
            "moe_prefetch_h_min": (_I, [ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.c_double, _I,
                                        ctypes.c_double]),
            "moe_prefetch_queue": (_I, [C, _I, _I, _P, _P, _I, _P, _P]),
            "moe_cache_prefetch": (_I, [_P, _I, _I, _I, _P, _I, _P, _P, _P, _P, _P]),
            "spice_lore_fit_workspace_bytes": (_Z, [C, _I, _I]),
            "moe_lore_fit": (_I, [C, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.POINTER(ctypes.c_double), _P, _Z,
                                  _P]),
            "spice_wait_ready": (_I, [_P, ctypes.c_uint32, ctypes.c_int64]),
            "spice_status_string": (ctypes.c_char_p, [_I]),
            "spice_last_error": (ctypes.c_char_p, []),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype, f.argtypes = res, args
        _lib = L
    return _lib


def _p(a):
    """Address of a buffer argument."""
    if a is None:
        return None
    if isinstance(a, int):
        return a
    if hasattr(a, "data_ptr"):
        return a.data_ptr()
    if hasattr(a, "ctypes"):
        return a.ctypes.data
    if isinstance(a, ctypes.Array):
        return ctypes.addressof(a)
    raise TypeError(f"cannot pass {type(a).__name__} as a buffer")


def _stream(s):
    if s is None:
        import torch

        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else None
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _check(fn: str, st: int) -> None:
    if st != SPICE_OK:
        raise SpiceError(fn, st, lib().spice_last_error().decode())


def _matrix_bytes(cfg, rows: int, K: int) -> int:
    """Bytes of one routed-expert matrix [rows][K] in the cfg's weight format (the MXFP4 blob
    holds rows*K/2 code bytes and rows*K/32 scale bytes)."""
    if cfg.wfmt == SPICE_WFMT_MXFP4:
        return rows * K // 2 + rows * K // 32
    return rows * K * (2 if cfg.dtype == SPICE_BF16 else 4)


def _check_pools(fn: str, cfg, w13_pool, w2_pool) -> None:
    """Reject pool tensors smaller than cfg.n_slots experts in the cfg's weight format (for
    instance MXFP4 blobs passed with a cfg that says bf16): the kernels index the slots from
    the cfg alone, so a short pool would be read past its end.  Raw addresses pass unchecked."""
    for name, buf, rows, K in (("w13_pool", w13_pool, 2 * cfg.inter, cfg.d), ("w2_pool", w2_pool, cfg.d, cfg.inter)):
        if buf is None or not hasattr(buf, "element_size"):
            continue
        need = max(cfg.n_slots, 0) * _matrix_bytes(cfg, rows, K)
        have = buf.numel() * buf.element_size()
        if have < need:
            raise ValueError(f"{fn}: {name} holds {have} bytes, the cfg (n_slots {cfg.n_slots}, wfmt {cfg.wfmt}, "
                             f"dtype {cfg.dtype}) needs {need}")


def last_error() -> str:
    return lib().spice_last_error().decode()


def spice_status_string(status: int) -> str:
    return lib().spice_status_string(status).decode()


def spice_wait_ready(ready, value: int, timeout_us: int = 0) -> None:
    """Wait on the host until the pinned word `ready` holds `value`."""
    _check("spice_wait_ready", lib().spice_wait_ready(_p(ready), value & 0xFFFFFFFF, timeout_us))


def spice_workspace_bytes(cfg: spice_moe_cfg_t, T: int) -> int:
    return lib().spice_workspace_bytes(ctypes.byref(cfg), T)


def spice_workspace_init(ws, ws_bytes: int, stream=None) -> None:
    _check("spice_workspace_init", lib().spice_workspace_init(_p(ws), ws_bytes, _stream(stream)))


def spice_workspace_flags(ws, ws_bytes: int, clear: bool = False, stream=None) -> int:
    f = ctypes.c_uint32(0)
    _check("spice_workspace_flags",
           lib().spice_workspace_flags(_p(ws), ws_bytes, ctypes.byref(f), int(clear), _stream(stream)))
    return f.value


def moe_route_bucket(cfg, T, x, w_gate, logit_bias, resident_slot, conf, logits, topk_idx, topk_w, slot_class,
                     offsets, perm, inv_perm, host_out: Optional[spice_host_out_t], ws, ws_bytes,
                     stream=None) -> None:
    _check("moe_route_bucket", lib().moe_route_bucket(
        ctypes.byref(cfg), T, _p(x), _p(w_gate), _p(logit_bias), _p(resident_slot), _p(conf), _p(logits),
        _p(topk_idx), _p(topk_w), _p(slot_class), _p(offsets), _p(perm), _p(inv_perm),
        None if host_out is None else ctypes.byref(host_out), _p(ws), ws_bytes, _stream(stream)))


def moe_expert_ffn_grouped(cfg, T, x, perm, offsets, resident_slot, w13_pool, w2_pool, w13_shared, w2_shared,
                           lore_A, lore_B, y_slots, y_shared, ws, ws_bytes, stream=None) -> None:
    _check_pools("moe_expert_ffn_grouped", cfg, w13_pool, w2_pool)
    _check("moe_expert_ffn_grouped", lib().moe_expert_ffn_grouped(
        ctypes.byref(cfg), T, _p(x), _p(perm), _p(offsets), _p(resident_slot), _p(w13_pool), _p(w2_pool),
        _p(w13_shared), _p(w2_shared), _p(lore_A), _p(lore_B), _p(y_slots), _p(y_shared), _p(ws), ws_bytes,
        _stream(stream)))


def moe_expert_ffn_grouped_gated(cfg, T, x, perm, offsets, resident_slot, w13_pool, w2_pool, w13_shared, w2_shared,
                                 w_shared_gate, lore_A, lore_B, y_slots, y_shared, ws, ws_bytes, stream=None) -> None:
    _check_pools("moe_expert_ffn_grouped_gated", cfg, w13_pool, w2_pool)
    _check("moe_expert_ffn_grouped_gated", lib().moe_expert_ffn_grouped_gated(
        ctypes.byref(cfg), T, _p(x), _p(perm), _p(offsets), _p(resident_slot), _p(w13_pool), _p(w2_pool),
        _p(w13_shared), _p(w2_shared), _p(w_shared_gate), _p(lore_A), _p(lore_B), _p(y_slots), _p(y_shared),
        _p(ws), ws_bytes, _stream(stream)))


def lore_surrogate_apply(cfg, T, x, perm, offsets, lore_A, lore_B, y_slots, ws, ws_bytes, stream=None) -> None:
    _check("lore_surrogate_apply", lib().lore_surrogate_apply(
        ctypes.byref(cfg), T, _p(x), _p(perm), _p(offsets), _p(lore_A), _p(lore_B), _p(y_slots), _p(ws),
        ws_bytes, _stream(stream)))


def moe_combine(cfg, T, topk_w, slot_class, inv_perm, y_slots, y_shared, resid, out, stream=None) -> None:
    _check("moe_combine", lib().moe_combine(
        ctypes.byref(cfg), T, _p(topk_w), _p(slot_class), _p(inv_perm), _p(y_slots), _p(y_shared), _p(resid),
        _p(out), _stream(stream)))


def moe_layer_gpu(cfg, T, x, w_gate, logit_bias, resident_slot, conf, w13_pool, w2_pool, w13_shared, w2_shared,
                  w_shared_gate, lore_A, lore_B, logits, topk_idx, topk_w, slot_class, offsets, perm, inv_perm,
                  y_slots, y_shared, host_out: Optional[spice_host_out_t], resid, out, ws, ws_bytes,
                  stream=None) -> None:
    _check_pools("moe_layer_gpu", cfg, w13_pool, w2_pool)
    _check("moe_layer_gpu", lib().moe_layer_gpu(
        ctypes.byref(cfg), T, _p(x), _p(w_gate), _p(logit_bias), _p(resident_slot), _p(conf), _p(w13_pool),
        _p(w2_pool), _p(w13_shared), _p(w2_shared), _p(w_shared_gate), _p(lore_A), _p(lore_B), _p(logits),
        _p(topk_idx), _p(topk_w), _p(slot_class), _p(offsets), _p(perm), _p(inv_perm), _p(y_slots), _p(y_shared),
        None if host_out is None else ctypes.byref(host_out), _p(resid), _p(out), _p(ws), ws_bytes,
        _stream(stream)))


SPICE_NOALLOC_SCRATCH_BYTES = 32 << 20


def moe_layer_gpu_noalloc(cfg, T, x, w_gate, logit_bias, resident_slot, conf, w13_pool, w2_pool, w13_shared,
                          w2_shared, w_shared_gate, lore_A, lore_B, logits, topk_idx, topk_w, slot_class, offsets,
                          perm, inv_perm, y_slots, y_shared, host_out: Optional[spice_host_out_t], resid, out,
                          stream=None) -> None:
    _check_pools("moe_layer_gpu_noalloc", cfg, w13_pool, w2_pool)
    _check("moe_layer_gpu_noalloc", lib().moe_layer_gpu_noalloc(
        ctypes.byref(cfg), T, _p(x), _p(w_gate), _p(logit_bias), _p(resident_slot), _p(conf), _p(w13_pool),
        _p(w2_pool), _p(w13_shared), _p(w2_shared), _p(w_shared_gate), _p(lore_A), _p(lore_B), _p(logits),
        _p(topk_idx), _p(topk_w), _p(slot_class), _p(offsets), _p(perm), _p(inv_perm), _p(y_slots), _p(y_shared),
        None if host_out is None else ctypes.byref(host_out), _p(resid), _p(out), _stream(stream)))


def moe_exact_residual_host(cfg, T, x_host, topk_idx_host, topk_w_host, slot_class_host,
                            w13_host: Sequence, w2_host: Sequence, resid_host, n_threads: int = 0) -> None:
    """w13_host / w2_host: length-N sequences of host buffers (or None)."""
    t13 = (ctypes.c_void_p * len(w13_host))(*[_p(w) for w in w13_host])
    t2 = (ctypes.c_void_p * len(w2_host))(*[_p(w) for w in w2_host])
    _check("moe_exact_residual_host", lib().moe_exact_residual_host(
        ctypes.byref(cfg), T, _p(x_host), _p(topk_idx_host), _p(topk_w_host), _p(slot_class_host), t13, t2,
        _p(resid_host), n_threads))


def _table(items, n: int):
    """ctypes array of n addresses (None -> NULL)."""
    items = list(items)
    if len(items) != n:
        raise ValueError(f"table needs {n} entries, got {len(items)}")
    return (ctypes.c_void_p * n)(*[_p(a) for a in items])


class ExpertCache:
    """Handle of moe_cache_create (bookkeeping only when w13_pool is None)."""

    def __init__(self, cfg: spice_moe_cfg_t, n_layers: int, initial_experts, w13_host=None, w2_host=None,
                 w13_pool=None, w2_pool=None, resident_slot=None, load: bool = False, stream=None):
        import numpy as np

        self.cfg, self.L, self.C = cfg, n_layers, cfg.n_slots
        self.device = w13_pool is not None
        init = np.ascontiguousarray(initial_experts, dtype=np.int32).reshape(n_layers, cfg.n_slots)
        self._keep = [init]
        args = [None] * 5
        if w13_pool is not None:
            LN = n_layers * cfg.n_experts
            args = [_table(w13_host, LN), _table(w2_host, LN), _table(w13_pool, n_layers),
                    _table(w2_pool, n_layers), _table(resident_slot, n_layers)]
            self._keep += [w13_host, w2_host, w13_pool, w2_pool, resident_slot, args]
        h = ctypes.c_void_p(None)
        _check("moe_cache_create", lib().moe_cache_create(
            ctypes.byref(cfg), n_layers, args[0], args[1], args[2], args[3], args[4], init.ctypes.data, int(load),
            _stream(stream) if w13_pool is not None else None, ctypes.byref(h)))
        self.h = h.value

    def step(self, layer: int, step: int, idx, cls, max_admit: int, copy_stream=None, compute_stream=None):
        """-> (admitted, evicted) as lists."""
        import numpy as np

        idx = np.ascontiguousarray(idx, dtype=np.int32)
        cls = np.ascontiguousarray(cls, dtype=np.uint8)
        T = idx.shape[0] if idx.ndim == 2 else idx.size // self.cfg.top_k
        n = ctypes.c_int32(0)
        adm = np.empty(max(max_admit, 1), np.int32)
        ev = np.empty(max(max_admit, 1), np.int32)
        dev = self.device
        _check("moe_cache_step", lib().moe_cache_step(
            self.h, layer, step, T, idx.ctypes.data, cls.ctypes.data, max_admit,
            _stream(copy_stream) if dev else None, _stream(compute_stream) if dev else None, ctypes.byref(n),
            adm.ctypes.data, ev.ctypes.data))
        return adm[:n.value].tolist(), ev[:n.value].tolist()

    def prefetch(self, layer: int, step: int, experts, max_prefetch: int, copy_stream=None, compute_stream=None):
        """Speculative admissions of the listed experts (issue order) -> (admitted, evicted)."""
        import numpy as np

        ex = np.ascontiguousarray(experts, dtype=np.int32).reshape(-1)
        n = ctypes.c_int32(0)
        adm = np.empty(max(max_prefetch, 1), np.int32)
        ev = np.empty(max(max_prefetch, 1), np.int32)
        dev = self.device
        _check("moe_cache_prefetch", lib().moe_cache_prefetch(
            self.h, layer, step, ex.size, ex.ctypes.data if ex.size else None, max_prefetch,
            _stream(copy_stream) if dev else None, _stream(compute_stream) if dev else None, ctypes.byref(n),
            adm.ctypes.data, ev.ctypes.data))
        return adm[:n.value].tolist(), ev[:n.value].tolist()

    def wait(self, layer: int, stream=None) -> None:
        _check("moe_cache_wait", lib().moe_cache_wait(self.h, layer, _stream(stream)))

    def state(self, layer: int):
        import numpy as np

        se = np.empty(self.C, np.int32)
        lu = np.empty(self.C, np.int32)
        _check("moe_cache_state", lib().moe_cache_state(self.h, layer, se.ctypes.data, lu.ctypes.data))
        return se, lu

    def close(self) -> None:
        if getattr(self, "h", None):
            lib().moe_cache_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def moe_split_plan(cfg, T, topk_idx_host, slot_class_host, cost: spice_split_cost_t, max_fetch: int):
    """-> list of experts to fetch; slot_class_host (uint8 array) is relabelled in place."""
    import numpy as np

    out = np.empty(max(max_fetch, 1), np.int32)
    n = ctypes.c_int32(0)
    _check("moe_split_plan", lib().moe_split_plan(
        ctypes.byref(cfg), T, _p(topk_idx_host), _p(slot_class_host), ctypes.byref(cost), max_fetch, _p(out),
        ctypes.byref(n)))
    return out[:n.value].tolist()


def moe_fetch_experts(cfg, experts: Sequence[int], w13_host: Sequence, w2_host: Sequence, w13_fetch, w2_fetch,
                      n_slots: int, fetch_expert, fetch_expert_stage, copy_stream=None) -> None:
    ex = (ctypes.c_int32 * max(len(experts), 1))(*experts)
    t13 = (ctypes.c_void_p * len(w13_host))(*[_p(w) for w in w13_host])
    t2 = (ctypes.c_void_p * len(w2_host))(*[_p(w) for w in w2_host])
    _check("moe_fetch_experts", lib().moe_fetch_experts(
        ctypes.byref(cfg), len(experts), ex, t13, t2, _p(w13_fetch), _p(w2_fetch), n_slots, _p(fetch_expert),
        _p(fetch_expert_stage), _stream(copy_stream)))


def moe_expert_ffn_fetched(cfg, T, x, perm, offsets, slot_class, fetch_expert, w13_fetch, w2_fetch, n_slots,
                           y_slots, ws, ws_bytes, stream=None) -> None:
    _check("moe_expert_ffn_fetched", lib().moe_expert_ffn_fetched(
        ctypes.byref(cfg), T, _p(x), _p(perm), _p(offsets), _p(slot_class), _p(fetch_expert), _p(w13_fetch),
        _p(w2_fetch), n_slots, _p(y_slots), _p(ws), ws_bytes, _stream(stream)))


def spec_host(pred_idx=None, pred_prob=None, conf=None) -> spice_spec_host_t:
    """Pinned host copies of one depth's predictions (CPU tensors from pin_memory())."""
    return spice_spec_host_t(_p(pred_idx), _p(pred_prob), _p(conf))


def moe_spec_update(cfg, T, depth, l_min, tau, last, h_in, h_out, topk_idx, topk_w, inv_perm, y_slots, y_shared,
                    halted, pred_idx, pred_prob, conf, host_out=None, ws=None, ws_bytes=0, stream=None) -> None:
    _check("moe_spec_update", lib().moe_spec_update(
        ctypes.byref(cfg), T, depth, l_min, tau, int(last), _p(h_in), _p(h_out), _p(topk_idx), _p(topk_w),
        _p(inv_perm), _p(y_slots), _p(y_shared), _p(halted), _p(pred_idx), _p(pred_prob), _p(conf),
        None if host_out is None else ctypes.byref(host_out), _p(ws), ws_bytes, _stream(stream)))


def moe_prefetch_h_min(P, expert_bytes, pcie_bytes_per_s, t_attn_s, K, t_expert_s) -> int:
    return lib().moe_prefetch_h_min(P, expert_bytes, pcie_bytes_per_s, t_attn_s, K, t_expert_s)


def moe_prefetch_queue(cfg, pred_idx_host, pred_prob_host, max_per_depth: int):
    """Per-depth issue lists from host predictions [n_depth][T][K]."""
    import numpy as np

    pidx = np.ascontiguousarray(pred_idx_host, dtype=np.int32)
    pprob = np.ascontiguousarray(pred_prob_host, dtype=np.float32)
    D, T = pidx.shape[0], pidx.shape[1]
    ex = np.empty((D, max(max_per_depth, 1)), np.int32)
    cnt = np.zeros(max(D, 1), np.int32)
    _check("moe_prefetch_queue", lib().moe_prefetch_queue(
        ctypes.byref(cfg), T, D, pidx.ctypes.data, pprob.ctypes.data, max_per_depth, ex.ctypes.data,
        cnt.ctypes.data))
    return [ex[i, :cnt[i]].tolist() for i in range(D)]


def moe_lore_fit(cfg, n, r, x, w13, w2, w13s, w2s, A_out, B_out, y_out=None, ws=None, ws_bytes=0,
                 stream=None) -> float:
    """LoRE calibration fit of one expert (Eq. 10); returns the minimum loss."""
    loss = ctypes.c_double(0.0)
    _check("moe_lore_fit", lib().moe_lore_fit(
        ctypes.byref(cfg), n, r, _p(x), _p(w13), _p(w2), _p(w13s), _p(w2s), _p(A_out), _p(B_out), _p(y_out),
        ctypes.byref(loss), _p(ws), ws_bytes, _stream(stream)))
    return loss.value
