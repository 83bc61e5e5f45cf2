"""The C-ABI library without a GPU: it loads, exports every function the header
declares, and rejects bad arguments on the host before touching HIP."""
import ctypes
import os
import re

import pytest

from paper_2608_21240_amd import spice, workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "spice_moe.h")
DUMMY = 0x1000  # never dereferenced: every case below fails validation first


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(?:spice_status_t|size_t|int32_t|void|const char\*)\s+(\w+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    L = spice.lib()
    names = declared_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(spice.EXPORTS)


def cfg(**kw):
    c = spice.make_cfg(W.DSV2, n_slots=32)
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def route(c, T=4, ws_bytes=None, conf=DUMMY, host_out=None, **ptrs):
    p = dict(x=DUMMY, w_gate=DUMMY, resident_slot=DUMMY, topk_idx=DUMMY, topk_w=DUMMY, slot_class=DUMMY,
             offsets=DUMMY, perm=DUMMY, inv_perm=DUMMY, ws=DUMMY)
    p.update(ptrs)
    if ws_bytes is None:
        ws_bytes = spice.spice_workspace_bytes(c, T) if spice.spice_workspace_bytes(c, T) else 1 << 40
    return spice.lib().moe_route_bucket(ctypes.byref(c), T, p["x"], p["w_gate"], None, p["resident_slot"], conf,
                                        None, p["topk_idx"], p["topk_w"], p["slot_class"], p["offsets"], p["perm"],
                                        p["inv_perm"], None if host_out is None else ctypes.byref(host_out),
                                        p["ws"], ws_bytes, None)


@pytest.mark.parametrize("field,value,status", [
    ("top_k", 0, spice.SPICE_ERR_INVALID),
    ("top_k", 65, spice.SPICE_ERR_INVALID),            # K > N
    ("n_experts", 0, spice.SPICE_ERR_INVALID),
    ("n_experts", 300, spice.SPICE_ERR_UNSUPPORTED),
    ("d", 0, spice.SPICE_ERR_INVALID),
    ("d", 2044, spice.SPICE_ERR_UNSUPPORTED),           # not a multiple of 8 for bf16
    ("inter", 1404, spice.SPICE_ERR_UNSUPPORTED),
    ("lore_rank", -1, spice.SPICE_ERR_INVALID),
    ("lore_rank", 260, spice.SPICE_ERR_UNSUPPORTED),
    ("n_slots", -1, spice.SPICE_ERR_INVALID),
    ("dtype", 7, spice.SPICE_ERR_UNSUPPORTED),
    ("conf_mode", 3, spice.SPICE_ERR_INVALID),
    ("norm_topk", 2, spice.SPICE_ERR_INVALID),
])
def test_bad_configuration_is_rejected(field, value, status):
    assert route(cfg(**{field: value})) == status
    assert spice.last_error()
    assert spice.spice_workspace_bytes(cfg(**{field: value}), 4) == 0


def test_token_count_rules():
    assert route(cfg(), T=-1) == spice.SPICE_ERR_INVALID
    assert route(cfg(), T=spice.SPICE_MAX_TOKENS + 1) == spice.SPICE_ERR_UNSUPPORTED
    # T == 0 is a no-op even with NULL buffers
    z = spice.lib().moe_route_bucket(ctypes.byref(cfg()), 0, None, None, None, None, None, None, None, None, None,
                                     None, None, None, None, None, 0, None)
    assert z == spice.SPICE_OK


def test_null_pointers_and_missing_confidence():
    assert route(cfg(), x=None) == spice.SPICE_ERR_INVALID
    assert route(cfg(), perm=None) == spice.SPICE_ERR_INVALID
    assert route(cfg(), conf=None) == spice.SPICE_ERR_INVALID
    assert "conf" in spice.last_error()


def test_small_workspace_is_rejected():
    c = cfg()
    need = spice.spice_workspace_bytes(c, 4)
    assert need >= spice.SPICE_WS_CONTROL_BYTES
    assert route(c, T=4, ws_bytes=need - 1) == spice.SPICE_ERR_WORKSPACE
    assert spice.spice_workspace_bytes(c, 64) > need


def test_ffn_lore_combine_validation():
    c = cfg()
    L = spice.lib()
    ws = spice.spice_workspace_bytes(c, 4)
    # missing pool pointers
    st = L.moe_expert_ffn_grouped(ctypes.byref(c), 4, DUMMY, DUMMY, DUMMY, DUMMY, None, None, DUMMY, DUMMY, None,
                                  None, DUMMY, DUMMY, DUMMY, ws, None)
    assert st == spice.SPICE_ERR_INVALID
    st = L.lore_surrogate_apply(ctypes.byref(c), 4, DUMMY, DUMMY, DUMMY, None, DUMMY, DUMMY, DUMMY, ws, None)
    assert st == spice.SPICE_ERR_INVALID
    # outputs that alias
    st = L.moe_expert_ffn_grouped(ctypes.byref(c), 4, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY,
                                  None, None, 0x200000, 0x200000, DUMMY, ws, None)
    assert st == spice.SPICE_ERR_INVALID
    st = L.moe_combine(ctypes.byref(c), 4, DUMMY, DUMMY, DUMMY, 0x100000, 0x900000, None, 0x100000, None)
    assert st == spice.SPICE_ERR_INVALID
    st = L.moe_combine(ctypes.byref(c), 4, DUMMY, DUMMY, DUMMY, DUMMY, None, None, 0x900000, None)
    assert st == spice.SPICE_ERR_INVALID


def test_short_pools_are_rejected_by_the_binding():
    """MXFP4 pool blobs handed over with a cfg that says bf16 are a quarter of the size the
    kernels would index; the binding refuses them before any library call."""
    import torch

    s = W.DSV2
    mx = spice.make_cfg(s, n_slots=2, wfmt=spice.SPICE_WFMT_MXFP4)
    bf = spice.make_cfg(s, n_slots=2)
    p13 = torch.empty((2, (2 * s.inter * s.d) * 17 // 32), dtype=torch.uint8)
    p2 = torch.empty((2, (s.d * s.inter) * 17 // 32), dtype=torch.uint8)
    spice._check_pools("t", mx, p13, p2)  # the right size for MXFP4
    with pytest.raises(ValueError, match="w13_pool"):
        spice.moe_expert_ffn_grouped(bf, 4, DUMMY, DUMMY, DUMMY, DUMMY, p13, p2, DUMMY, DUMMY, None, None, DUMMY,
                                     DUMMY, DUMMY, 1 << 30)
    with pytest.raises(ValueError, match="w2_pool"):
        spice._check_pools("t", mx, p13, p2[:1])
    three = spice.make_cfg(s, n_slots=3, wfmt=spice.SPICE_WFMT_MXFP4)  # more slots than the pool
    with pytest.raises(ValueError, match="n_slots 3"):
        spice.moe_layer_gpu(three, 4, *([DUMMY] * 5), p13, p2, *([DUMMY] * 19), None)
    bf_pool = torch.empty((2, 2 * s.inter, s.d), dtype=torch.bfloat16)
    spice._check_pools("t", bf, bf_pool, torch.empty((2, s.d, s.inter), dtype=torch.bfloat16))


def test_gated_ffn_validation():
    c = cfg()
    L = spice.lib()
    ws = spice.spice_workspace_bytes(c, 4)
    # the gate row is required when the layer has a shared block
    st = L.moe_expert_ffn_grouped_gated(ctypes.byref(c), 4, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY,
                                        None, None, None, 0x100000, 0x900000, DUMMY, ws, None)
    assert st == spice.SPICE_ERR_INVALID
    assert "w_shared_gate" in spice.last_error()
    # and the usual checks still apply (missing pools)
    st = L.moe_expert_ffn_grouped_gated(ctypes.byref(c), 4, DUMMY, DUMMY, DUMMY, DUMMY, None, None, DUMMY, DUMMY,
                                        DUMMY, None, None, 0x100000, 0x900000, DUMMY, ws, None)
    assert st == spice.SPICE_ERR_INVALID
    # the workspace holds the gate values: one fp32 per token beyond the ungated layout
    assert spice.spice_workspace_bytes(c, 64) >= spice.spice_workspace_bytes(c, 4) + 60 * 4


def test_status_strings():
    assert spice.spice_status_string(spice.SPICE_ERR_WORKSPACE) == "SPICE_ERR_WORKSPACE"
    assert spice.spice_status_string(12345) == "unknown spice_status_t"


def test_pageable_host_copies_are_rejected():
    """The route kernel writes host copies over PCIe: pageable memory would fault, so it is refused."""
    import numpy as np

    buf = np.zeros(1 << 16, np.uint8)
    for field in ("x", "topk_idx", "topk_w", "slot_class", "class_counts"):
        ho = spice.host_out(**{field: buf})
        assert route(cfg(), host_out=ho) == spice.SPICE_ERR_INVALID
        assert "host_out." + field in spice.last_error()


def test_spec_update_validates_on_the_host():
    L = spice.lib()
    c = cfg()
    D = DUMMY
    ws = spice.spice_workspace_bytes(c, 4)

    def call(T=4, depth=1, l_min=1, tau=0.5, h_in=D, h_out=D, **kw):
        p = dict(topk_idx=D, topk_w=D, inv_perm=D, y_slots=D, y_shared=D, halted=D, pred_idx=D, pred_prob=D,
                 conf=D, ws=D)
        p.update(kw)
        return L.moe_spec_update(ctypes.byref(c), T, depth, l_min, tau, 0, h_in, h_out, p["topk_idx"],
                                 p["topk_w"], p["inv_perm"], p["y_slots"], p["y_shared"], p["halted"],
                                 p["pred_idx"], p["pred_prob"], p["conf"], None, p["ws"], ws, None)

    assert call(depth=0) == spice.SPICE_ERR_INVALID
    assert call(l_min=-1) == spice.SPICE_ERR_INVALID
    assert call(tau=float("nan")) == spice.SPICE_ERR_INVALID
    assert call(tau=float("inf")) == spice.SPICE_ERR_INVALID
    assert call(tau=-0.1) == spice.SPICE_ERR_INVALID
    for k in ("topk_idx", "topk_w", "inv_perm", "y_shared", "halted", "pred_idx", "pred_prob", "conf"):
        assert call(**{k: None}) == spice.SPICE_ERR_INVALID, k
    assert call(h_in=None) == spice.SPICE_ERR_INVALID
    assert call(h_out=D + 64) == spice.SPICE_ERR_INVALID  # overlaps h_in without being it
    assert call(ws=None) == spice.SPICE_ERR_INVALID
    assert call(T=0, depth=1) == spice.SPICE_OK


def test_lore_fit_validates_on_the_host():
    L = spice.lib()
    c = cfg()
    D = DUMMY
    ws = spice.spice_workspace_bytes(c, 8) * 8

    def call(n=8, r=4, x=D, w13=D, w2=D, ws_=D, ws_bytes=ws):
        return L.moe_lore_fit(ctypes.byref(c), n, r, x, w13, w2, D, D, D, D, None, None, ws_, ws_bytes, None)

    assert call(n=0) == spice.SPICE_ERR_INVALID
    assert call(n=c.d + 1) in (spice.SPICE_ERR_UNSUPPORTED, spice.SPICE_ERR_INVALID)
    assert call(n=1025) in (spice.SPICE_ERR_UNSUPPORTED, spice.SPICE_ERR_INVALID)
    assert call(r=0) == spice.SPICE_ERR_INVALID
    assert call(r=c.d + 1) == spice.SPICE_ERR_INVALID
    assert call(x=None) == spice.SPICE_ERR_INVALID
    assert call(w2=None) == spice.SPICE_ERR_INVALID
    assert call(ws_=None) == spice.SPICE_ERR_INVALID
    assert call(ws_bytes=16) == spice.SPICE_ERR_WORKSPACE
    assert L.spice_lore_fit_workspace_bytes(ctypes.byref(c), 0, 4) == 0
    assert L.spice_lore_fit_workspace_bytes(ctypes.byref(c), 2000, 4) == 0
    assert L.spice_lore_fit_workspace_bytes(ctypes.byref(c), 512, 32) > 512 * 512 * 16
