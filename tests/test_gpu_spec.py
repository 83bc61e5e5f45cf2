"""Speculative prefetching on the GPU (Sec. 4.1, Alg. 1) against the oracle.

The rollout is checked depth by depth with teacher forcing: the oracle's step starts
from the GPU's own draft state and halted set before that depth, so each depth is
compared on identical inputs.  Integer outputs (predicted experts, halting) must match
exactly wherever the decision is certified (the oracle's top-K logit gaps exceed the
fp64 summation bound; the confidence is clear of tau by more than fp32 rounding of the
gates), probabilities and confidences to fp32 rounding, and the draft state to the
dtype's tolerance.  The device cache's speculative admissions are checked for landing
the right weights in the right slots.
"""
import numpy as np
import pytest
import torch

from paper_2608_21240_amd import layer as LY, spice, synth, workloads as W
from paper_2608_21240_amd.spec import SpecRollout
from paper_2608_21240_amd.workloads import MoEShape, Workload

from parity import rel_err, say, tol_for

pytestmark = pytest.mark.gpu

F32, BF16 = W.DTYPE_F32, W.DTYPE_BF16


def _weights(shape, n, seed):
    wl = Workload("spec", shape, tokens=1, resident=0, skew=False, seed=seed)
    out = []
    for j in range(n):
        w13s, w2s = synth.gen_shared(wl, j)
        lore = [synth.gen_lore(wl, j, e) for e in range(shape.n_experts)]
        out.append(dict(wg=synth.gen_router(wl, j), w13s=w13s, w2s=w2s, lA=[a for a, _ in lore],
                        lB=[b for _, b in lore]))
    return out


def _views(shape, ws):
    from types import SimpleNamespace
    dt = shape.dtype
    vs = []
    for w in ws:
        r = max(shape.lore_rank, 1)
        A = torch.stack([LY.to_tensor(a, dt) for a in w["lA"]]).cuda() if shape.lore_rank else None
        B = torch.stack([LY.to_tensor(b, dt) for b in w["lB"]]).cuda() if shape.lore_rank else None
        vs.append(SimpleNamespace(wg=LY.to_tensor(w["wg"], dt, "cuda"), bias=None,
                                  w13s=LY.to_tensor(w["w13s"], dt, "cuda"), w2s=LY.to_tensor(w["w2s"], dt, "cuda"),
                                  lore_A=A if A is not None else torch.zeros((shape.n_experts, r, shape.d)).cuda(),
                                  lore_B=B if B is not None else torch.zeros((shape.n_experts, shape.d, r)).cuda(),
                                  w_sg=None))
    return vs


def _np(t):
    from parity import to_np
    return to_np(t)


def _certified(orc, cfg, h, wg, K, d):
    z, zabs = orc.router_logits(cfg, h, wg)
    bound = 2.0 * d * 2.0 ** -53 * zabs
    zs = -np.sort(-z, axis=1)[:, : K + 1]
    gaps = np.abs(np.diff(zs, axis=1))
    return np.all((gaps > 4 * bound.max(axis=1, keepdims=True)) | (gaps == 0), axis=1)


# random routers give confidences near K/N-ish levels (about 0.3-0.4 here): tau 0 never
# halts (every depth moves every token), tau near the median halts some tokens per depth
CASES = [
    (MoEShape(192, 16, 4, 96, 160, 8, BF16), 13, 4, 2, 0.34),
    (MoEShape(128, 12, 3, 64, 96, 8, F32), 7, 3, 1, 0.0),
    (MoEShape(128, 12, 3, 64, 96, 8, F32), 19, 4, 1, 0.33),
    (MoEShape(256, 24, 6, 128, 0, 16, BF16), 33, 5, 1, 0.36),   # no shared block
    (MoEShape(2048, 64, 6, 1408, 2816, 32, BF16), 32, 4, 2, 0.0),  # DSV2-Lite shapes
    (MoEShape(2048, 64, 6, 1408, 2816, 32, BF16), 32, 4, 1, 0.33),
]


@pytest.mark.parametrize("shape,T,n,l_min,tau", CASES)
def test_rollout_depth_by_depth_matches_oracle(orc, shape, T, n, l_min, tau):
    say(f"spec rollout d={shape.d} N={shape.n_experts} K={shape.top_k} Is={shape.shared_inter} r={shape.lore_rank} "
        f"T={T} depths={n} l_min={l_min} tau={tau}")
    K, d = shape.top_k, shape.d
    ws = _weights(shape, n, seed=T)
    views = _views(shape, ws)
    x = synth.to_storage(np.random.default_rng(T).standard_normal((T, d)).astype(np.float32), shape.dtype)
    R = SpecRollout(shape, T, n, trace=True)
    R.run(views, LY.to_tensor(x, shape.dtype, "cuda"), l_min, tau)
    torch.cuda.synchronize()
    g_idx, g_prob, g_conf = _np(R.pred_idx), _np(R.pred_prob), _np(R.conf)
    g_h = [_np(R.state(j)) for j in range(n)]
    assert R.flags() == 0
    # the pinned host copies are the device outputs
    assert np.array_equal(R.pred_idx_h.numpy(), g_idx) and np.array_equal(R.pred_prob_h.numpy(), g_prob)
    assert np.array_equal(R.conf_h.numpy(), g_conf, equal_nan=True)
    cfg = orc.make_cfg(shape)
    h_in = x
    uncertified = 0
    for j in range(n):
        before = (g_idx[j][:, 0] == -1).astype(np.int32)  # halted before this depth, per the GPU
        halted = before.copy()
        L = ws[j]
        p_idx, p_prob, conf, h_out = orc.spec_step(cfg, h_in, j + 1, l_min, tau, j == n - 1, L["wg"], None,
                                                   L["w13s"], L["w2s"], L["lA"], L["lB"], halted)
        live = before == 0
        cert = _certified(orc, cfg, h_in, L["wg"], K, d) & live
        uncertified += int((live & ~cert).sum())
        assert np.array_equal(g_idx[j][cert], p_idx[cert]), f"depth {j + 1}: predicted experts"
        assert (g_idx[j][~live] == -1).all() and np.isnan(g_conf[j][~live]).all()
        same = live & (g_idx[j] == p_idx).all(axis=1)
        assert np.allclose(g_prob[j][same], p_prob[same], rtol=1e-6, atol=1e-12)
        assert np.allclose(g_conf[j][same], conf[same], rtol=1e-6, atol=1e-12)
        # halting: the GPU's halted set before the next depth (or at the end)
        after = (g_idx[j + 1][:, 0] == -1) if j + 1 < n else (_np(R.halted) == 1)
        clear = same & (np.abs(conf - tau) > 1e-5)
        assert np.array_equal(after[clear], halted[clear] == 1), f"depth {j + 1}: halting"
        # the draft state: tokens the GPU moved match the oracle's step to tolerance; the
        # others (halted before or now, or the last depth) are copied bit for bit
        moved = live & ~after if j < n - 1 else np.zeros(T, bool)
        assert np.array_equal(g_h[j][~moved], h_in[~moved])
        check = moved & same & (halted == 0)
        if check.any():
            err = rel_err(synth.as_f32(g_h[j][check], shape.dtype), synth.as_f32(h_out[check], shape.dtype))
            assert err.max() <= tol_for(shape), f"depth {j + 1}: draft state rel err {err.max():.3e}"
        mc = float(g_conf[j][live].mean()) if live.any() else float("nan")
        say(f"depth {j + 1}: live {int(live.sum())}/{T}, halted now {int(((halted == 1) & live).sum())}, "
            f"moved {int(moved.sum())}, mean conf {mc:.3f}")
        h_in = g_h[j]
    say(f"uncertified token-depths: {uncertified}")


def test_rollout_queue_is_the_oracle_queue_of_the_gpu_predictions(orc):
    shape = MoEShape(192, 16, 4, 96, 160, 8, BF16)
    T, n = 21, 4
    views = _views(shape, _weights(shape, n, seed=3))
    x = synth.to_storage(np.random.default_rng(4).standard_normal((T, shape.d)).astype(np.float32), shape.dtype)
    R = SpecRollout(shape, T, n)
    R.run(views, LY.to_tensor(x, shape.dtype, "cuda"), 1, 0.5)
    q = R.queue(6)
    want = orc.prefetch_queue(shape.n_experts, R.pred_idx_h.numpy(), R.pred_prob_h.numpy().astype(np.float64), 6)
    assert q == want and len(q) == n
    # a smaller T reuses the buffers
    R.run(views, LY.to_tensor(x[:5], shape.dtype, "cuda"), 1, 0.5, T=5)
    q5 = R.queue(16)
    want5 = orc.prefetch_queue(shape.n_experts, R.pred_idx_h.numpy()[:, :5], R.pred_prob_h.numpy()[:, :5]
                               .astype(np.float64), 16)
    assert q5 == want5


def test_cache_prefetch_copies_land_in_the_pools():
    shape = MoEShape(128, 12, 3, 64, 96, 8, BF16)
    wl = Workload("spec", shape, tokens=1, resident=0, skew=False)
    N, C, L = shape.n_experts, 4, 2
    dt = shape.dtype
    host = [synth.gen_expert(wl, 0, e) for e in range(N)]
    h13 = [LY.to_tensor(w13, dt, pin=True) for w13, _ in host]
    h2 = [LY.to_tensor(w2, dt, pin=True) for _, w2 in host]
    td = LY.torch_dtype(dt)
    p13 = [torch.zeros((C, 2 * shape.inter, shape.d), dtype=td, device="cuda") for _ in range(L)]
    p2 = [torch.zeros((C, shape.d, shape.inter), dtype=td, device="cuda") for _ in range(L)]
    res = [torch.full((N,), -1, dtype=torch.int32, device="cuda") for _ in range(L)]
    cfg = spice.make_cfg(shape, C)
    cache = spice.ExpertCache(cfg, L, [[0, 1, 2, 3], [4, 5, -1, 6]], w13_host=h13 * L, w2_host=h2 * L,
                              w13_pool=p13, w2_pool=p2, resident_slot=res, load=True)
    cs = torch.cuda.Stream()
    adm, ev = cache.prefetch(1, 0, [9, 5, 10, 11], 2, copy_stream=cs)
    assert adm == [9, 10] and ev == [-1, 4]
    adm2, _ = cache.prefetch(1, 0, [7], 1, copy_stream=cs)  # a second batch on the same layer
    cache.wait(1)
    torch.cuda.synchronize()
    se, _ = cache.state(1)
    want_res = np.full(N, -1, np.int32)
    for s, e in enumerate(se):
        if e >= 0:
            want_res[e] = s
            assert torch.equal(p13[1][s].cpu(), h13[e]) and torch.equal(p2[1][s].cpu(), h2[e]), (s, e)
    assert np.array_equal(res[1].cpu().numpy(), want_res)
    cache.close()
