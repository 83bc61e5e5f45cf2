"""The library's host-side exact residual (Sec. 4.3, M_cpu) against the oracle, on the CPU."""
import numpy as np
import pytest

from paper_2608_21240_amd import spice, synth, workloads as W

HIT, LORE, EXACT = 0, 1, 2


def rel_err(out, ref):
    """Per-token max |out - ref| / max |ref|, the tolerance metric of the parity tests."""
    num = np.abs(out - ref).max(axis=1)
    den = np.maximum(np.abs(ref).max(axis=1), 1e-30)
    return num / den


def setup(orc, shape, T, seed, exact_frac=0.6, resident_frac=0.3, wfmt=0):
    wl = W.Workload("t", shape, tokens=T, resident=0, skew=False, seed=seed, wfmt=wfmt)
    r = np.random.default_rng(seed)
    N = shape.n_experts
    resident = np.zeros(N, np.int32)
    resident[r.permutation(N)[: int(resident_frac * N)]] = 1
    x = synth.gen_x(wl)
    wg = synth.gen_router(wl)
    conf = np.where(r.random((T, shape.top_k)) < exact_frac, 0.9, 0.1).astype(np.float32)
    cfg = orc.make_cfg(shape, wfmt=wfmt)
    rt = orc.route(cfg, x, wg, None, resident, conf)
    experts = sorted(set(rt["idx"][rt["cls"] == EXACT].tolist()))
    w13 = [None] * N
    w2 = [None] * N
    for e in experts:
        w13[e], w2[e] = synth.gen_expert(wl, 0, e)
    return wl, cfg, x, rt, w13, w2


@pytest.mark.parametrize("shape,T,seed", [
    (W.TINY, 4, 0),
    (W.small_shape(dtype=W.DTYPE_F32), 9, 1),
    (W.small_shape(), 13, 2),
    (W.MoEShape(2048, 64, 6, 1408, 2816, 32, W.DTYPE_BF16), 3, 3),
])
def test_exact_residual_matches_oracle(orc, shape, T, seed):
    wl, cfg, x, rt, w13, w2 = setup(orc, shape, T, seed)
    ref = orc.exact_residual(cfg, x, rt["idx"], rt["g"], rt["cls"], w13, w2)
    c = spice.make_cfg(shape, n_slots=0)
    out = np.full((T, shape.d), np.nan, np.float32)
    gw = rt["g"].astype(np.float32)
    spice.moe_exact_residual_host(c, T, x, rt["idx"], gw, rt["cls"], w13, w2, out, n_threads=4)
    has = (rt["cls"] == EXACT).any(axis=1)
    assert has.any()
    assert (out[~has] == 0).all()
    tol = 1e-4  # fp32 arithmetic on exact inputs, for fp32 and bf16 storage alike
    assert rel_err(out[has], ref[has]).max() < tol


@pytest.mark.parametrize("shape,T,seed", [
    (W.small_shape(), 13, 4),
    (W.MoEShape(2048, 64, 6, 1408, 2816, 32, W.DTYPE_BF16), 2, 6),
])
def test_exact_residual_mxfp4_matches_oracle(orc, shape, T, seed):
    """MXFP4 expert weights: the host path decodes the same blobs the oracle reads."""
    wl, cfg, x, rt, w13, w2 = setup(orc, shape, T, seed, wfmt=W.WFMT_MXFP4)
    assert all(a is None or a.dtype == np.uint8 for a in w13)
    ref = orc.exact_residual(cfg, x, rt["idx"], rt["g"], rt["cls"], w13, w2)
    c = spice.make_cfg(shape, n_slots=0, wfmt=spice.SPICE_WFMT_MXFP4)
    gw = rt["g"].astype(np.float32)
    outs = []
    for nt in (1, 5):
        out = np.full((T, shape.d), np.nan, np.float32)
        spice.moe_exact_residual_host(c, T, x, rt["idx"], gw, rt["cls"], w13, w2, out, n_threads=nt)
        outs.append(out)
    assert np.array_equal(outs[0], outs[1])
    has = (rt["cls"] == EXACT).any(axis=1)
    assert has.any() and (outs[0][~has] == 0).all()
    assert rel_err(outs[0][has], ref[has]).max() < 1e-4


def test_mxfp4_config_rules():
    bad = spice.make_cfg(W.small_shape(dtype=W.DTYPE_F32), n_slots=0, wfmt=spice.SPICE_WFMT_MXFP4)
    assert spice.spice_workspace_bytes(bad, 4) == 0  # MXFP4 needs bf16 activations
    odd = spice.make_cfg(W.MoEShape(200, 16, 4, 104, 168, 24, W.DTYPE_BF16), n_slots=0, wfmt=spice.SPICE_WFMT_MXFP4)
    assert spice.spice_workspace_bytes(odd, 4) == 0  # d and inter multiples of 32
    unknown = spice.make_cfg(W.small_shape(), n_slots=0, wfmt=1)
    assert spice.spice_workspace_bytes(unknown, 4) == 0
    wide = spice.make_cfg(W.MoEShape(4128, 16, 4, 128, 128, 8, W.DTYPE_BF16), n_slots=0, wfmt=spice.SPICE_WFMT_MXFP4)
    assert spice.spice_workspace_bytes(wide, 4) == 0  # d above the MXFP4 limit (4096)
    assert "SPICE_MXFP4_MAX_K" in spice.last_error()
    edge = spice.make_cfg(W.MoEShape(4096, 16, 4, 4096, 128, 8, W.DTYPE_BF16), n_slots=0, wfmt=spice.SPICE_WFMT_MXFP4)
    assert spice.spice_workspace_bytes(edge, 4) > 0
    ok = spice.make_cfg(W.small_shape(), n_slots=0, wfmt=spice.SPICE_WFMT_MXFP4)
    assert spice.spice_workspace_bytes(ok, 4) > 0


def test_result_is_independent_of_thread_count(orc):
    shape = W.small_shape()
    wl, cfg, x, rt, w13, w2 = setup(orc, shape, 21, 5)
    c = spice.make_cfg(shape, n_slots=0)
    outs = []
    for nt in (1, 2, 3, 8):
        out = np.empty((21, shape.d), np.float32)
        spice.moe_exact_residual_host(c, 21, x, rt["idx"], rt["g"].astype(np.float32), rt["cls"], w13, w2, out,
                                      n_threads=nt)
        outs.append(out)
    for o in outs[1:]:
        assert np.array_equal(o, outs[0])


def test_degenerate_inputs(orc):
    shape = W.small_shape()
    wl, cfg, x, rt, w13, w2 = setup(orc, shape, 6, 6)
    c = spice.make_cfg(shape, n_slots=0)
    out = np.full((6, shape.d), 7.0, np.float32)
    # T == 0: nothing is touched
    spice.moe_exact_residual_host(c, 0, x, rt["idx"], rt["g"].astype(np.float32), rt["cls"], w13, w2, out)
    assert (out == 7.0).all()
    # no exact slot: zero residual, no weights needed
    cls = np.where(rt["cls"] == EXACT, LORE, rt["cls"]).astype(np.uint8)
    spice.moe_exact_residual_host(c, 6, x, rt["idx"], rt["g"].astype(np.float32), cls, [None] * 16, [None] * 16,
                                  out)
    assert (out == 0).all()
    # an exact-miss expert without weights, a bad class, a bad expert id
    with pytest.raises(spice.SpiceError) as e:
        spice.moe_exact_residual_host(c, 6, x, rt["idx"], rt["g"].astype(np.float32), rt["cls"], [None] * 16,
                                      [None] * 16, out)
    assert e.value.status == spice.SPICE_ERR_INVALID
    bad = rt["cls"].copy(); bad[0, 0] = 4
    with pytest.raises(spice.SpiceError):
        spice.moe_exact_residual_host(c, 6, x, rt["idx"], rt["g"].astype(np.float32), bad, w13, w2, out)
    badi = rt["idx"].copy(); badi[rt["cls"] == EXACT] = 99
    with pytest.raises(spice.SpiceError):
        spice.moe_exact_residual_host(c, 6, x, badi, rt["g"].astype(np.float32), rt["cls"], w13, w2, out)


def test_exact_gpu_slots_are_left_to_the_gpu(orc):
    """Slots relabelled EXACT_GPU (fetched experts, Eq. 12's M_fetch) are skipped: the
    residual equals the oracle's over the remaining EXACT slots only."""
    shape = W.small_shape()
    wl, cfg, x, rt, w13, w2 = setup(orc, shape, 9, 5)
    c = spice.make_cfg(shape, n_slots=0)
    cls = rt["cls"].copy()
    ex = np.argwhere(cls == EXACT)
    assert len(ex) >= 2
    for t, k in ex[::2]:
        cls[t, k] = spice.SPICE_CLASS_EXACT_GPU
    out = np.empty((9, shape.d), np.float32)
    spice.moe_exact_residual_host(c, 9, x, rt["idx"], rt["g"].astype(np.float32), cls, w13, w2, out)
    only = np.where(cls == EXACT, EXACT, LORE).astype(np.uint8)
    ref = orc.exact_residual(orc.make_cfg(shape), x, rt["idx"], rt["g"], only, w13, w2)
    err = np.abs(out - ref).max() / max(np.abs(ref).max(), 1e-30)
    assert err < 1e-4 if shape.dtype == 0 else err < 2e-2


def test_exact_residual_mxfp4_scale_bytes(orc):
    """E8M0 edge bytes on the host path: 0 is 2^-127 (tiny, not zero, as in the oracle), 1 is
    2^-126, 255 is NaN, 100 an ordinary small scale; the oracle's decode of the same blobs
    is the reference.  (Large scales overflow fp32 in SwiGLU, as they would in any fp32
    evaluation, so they are not a parity case.)"""
    shape = W.small_shape()
    wl, cfg, x, rt, w13, w2 = setup(orc, shape, 7, 8, wfmt=W.WFMT_MXFP4)
    c = spice.make_cfg(shape, n_slots=0, wfmt=spice.SPICE_WFMT_MXFP4)
    gw = rt["g"].astype(np.float32)
    has = (rt["cls"] == EXACT).any(axis=1)
    assert has.any()
    n13 = 2 * shape.inter * shape.d // 2
    for byte in (0, 1, 100, 255):
        a13 = [None if b is None else b.copy() for b in w13]
        for b in a13:
            if b is not None:
                b[n13:] = byte  # every W1/W3 block scale
        out = np.full((7, shape.d), np.nan, np.float32)
        spice.moe_exact_residual_host(c, 7, x, rt["idx"], gw, rt["cls"], a13, w2, out, n_threads=3)
        ref = orc.exact_residual(cfg, x, rt["idx"], rt["g"], rt["cls"], a13, w2)
        if byte == 255:
            assert np.isnan(out[has]).all() and np.isnan(ref[has]).all()
            continue
        assert np.isfinite(out[has]).all() and np.isfinite(ref[has]).all()
        if byte <= 1:  # SiLU(g) u with g, u ~ 1e-38: below 1e-70, zero in fp32
            assert np.abs(ref[has]).max() < 1e-60 and (np.abs(out[has]) < 1e-30).all()
        else:
            assert rel_err(out[has], ref[has]).max() < 1e-4
