"""LoRE calibration fit on the GPU (Sec. 4.2, Eq. 8-10) against the oracle.

Two checks per case: the residual targets the GPU computes, E_e(x) - S(x), against the
oracle's expert and shared-block outputs (the FFN tolerance of the dtype); and the fit
itself with teacher forcing, the oracle's reduced-rank regression run on the GPU's own
targets: the maps B A and the minimum losses must agree to fp32 rounding.
"""
import numpy as np
import pytest
import torch

from paper_2608_21240_amd import layer as LY, spice, synth, workloads as W
from paper_2608_21240_amd.workloads import MoEShape, Workload

from parity import rel_err, say, tol_for

pytestmark = pytest.mark.gpu

F32, BF16 = W.DTYPE_F32, W.DTYPE_BF16

CASES = [
    (MoEShape(192, 8, 2, 96, 160, 8, BF16), 64, 8),
    (MoEShape(128, 8, 2, 64, 96, 16, F32), 100, 16),
    (MoEShape(256, 8, 2, 128, 0, 16, BF16), 40, 12),    # no shared block
    (MoEShape(192, 8, 2, 96, 160, 8, BF16), 24, 32),    # r >= n: exact fit
    (MoEShape(2048, 64, 6, 1408, 2816, 32, BF16), 512, 32),  # DSV2-Lite expert, GEMM path
]


def _fit(shape, n, r, seed):
    wl = Workload("fit", shape, tokens=n, resident=0, skew=False, seed=seed)
    d, dt = shape.d, shape.dtype
    w13, w2 = synth.gen_expert(wl, 0, 3)
    w13s, w2s = synth.gen_shared(wl, 0)
    X = synth.gen_x(wl, 0, 0, n)
    dev = lambda a: LY.to_tensor(a, dt, "cuda")  # noqa: E731
    cfg = spice.make_cfg(shape, 1)
    A = torch.empty((r, d), dtype=torch.float32, device="cuda")
    B = torch.empty((d, r), dtype=torch.float32, device="cuda")
    Y = torch.empty((n, d), dtype=torch.float32, device="cuda")
    wsb = spice.lib().spice_lore_fit_workspace_bytes(spice.ctypes.byref(cfg), n, r)
    assert wsb > 0
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    loss = spice.moe_lore_fit(cfg, n, r, dev(X), dev(w13), dev(w2), dev(w13s) if shape.shared_inter else None,
                              dev(w2s) if shape.shared_inter else None, A, B, Y, ws, wsb)
    return dict(wl=wl, X=X, w13=w13, w2=w2, w13s=w13s, w2s=w2s, A=A.cpu().numpy().astype(np.float64),
                B=B.cpu().numpy().astype(np.float64), Y=Y.cpu().numpy().astype(np.float64), loss=loss)


def _oracle_targets(orc, shape, g, X, tokens=None):
    """E_e(x) - S(x) by the oracle for the rows `tokens` of X (all by default)."""
    Xf = synth.as_f32(X, shape.dtype).astype(np.float64)
    toks = range(X.shape[0]) if tokens is None else tokens
    Y = np.zeros_like(Xf)
    for t in toks:
        e = np.empty(shape.d); s = np.zeros(shape.d)
        orc.lib().orc_swiglu(shape.d, shape.inter, shape.dtype, orc._store(g["w13"], shape.dtype).ctypes.data,
                             orc._store(g["w2"], shape.dtype).ctypes.data, Xf[t].ctypes.data, e.ctypes.data)
        if shape.shared_inter:
            orc.lib().orc_swiglu(shape.d, shape.shared_inter, shape.dtype,
                                 orc._store(g["w13s"], shape.dtype).ctypes.data,
                                 orc._store(g["w2s"], shape.dtype).ctypes.data, Xf[t].ctypes.data, s.ctypes.data)
        Y[t] = e - s
    return Xf, Y


@pytest.mark.parametrize("shape,n,r", CASES)
def test_lore_fit_matches_oracle(orc, shape, n, r):
    say(f"lore fit d={shape.d} I={shape.inter} Is={shape.shared_inter} n={n} r={r} dtype={shape.dtype}")
    g = _fit(shape, n, r, seed=n)
    toks = np.arange(n) if n <= 128 else np.linspace(0, n - 1, 32).astype(int)
    Xf, Yo = _oracle_targets(orc, shape, g, g["X"], toks)
    ey = rel_err(g["Y"][toks], Yo[toks])
    say(f"residual targets rel err (median, max): {np.median(ey):.2e}, {ey.max():.2e}")
    assert ey.max() <= tol_for(shape)
    # the fit on the GPU's own targets
    A_o, B_o, loss_o = orc.lore_fit(Xf, g["Y"], min(r, shape.d))
    W_g, W_o = g["B"] @ g["A"], B_o @ A_o
    total = float((g["Y"] ** 2).sum())
    say(f"loss gpu {g['loss']:.6e} oracle {loss_o:.6e} (|Y|^2 {total:.4e})")
    assert abs(g["loss"] - loss_o) <= 1e-6 * loss_o + 1e-9 * total
    if r >= n:
        assert g["loss"] <= 1e-9 * total
    ew = np.linalg.norm(W_g - W_o) / np.linalg.norm(W_o)
    say(f"B A rel Frobenius err {ew:.2e}")
    assert ew <= 1e-4
    # the loss the GPU reports is the loss of the factors it wrote
    assert orc.lore_loss(Xf, g["Y"], g["A"], g["B"]) == pytest.approx(g["loss"], rel=1e-4, abs=1e-7 * total)

