"""Pins for the oracle's expert FFN, LoRE correction, substitution and combine
(Eq. 6, 7, 9, 11 and the gate-weighted aggregation of Sec. 2.1), and the exact
CPU residual of Sec. 4.3.

References used here are independent of the oracle's code: torch fp64 matmuls
for the dense MoE, closed forms, and algebraic special cases (all resident,
exact full-rank LoRE factors, zero factors, zero down projections,
permutation equivariance).
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from paper_2608_21240_amd import synth, workloads as W

HIT, LORE, EXACT = 0, 1, 2


def _rand(r, shape, dtype, std):
    return synth.to_storage(r.standard_normal(shape).astype(np.float32) * np.float32(std), dtype)


def make_layer(seed=0, dtype=W.DTYPE_F32, d=32, N=6, K=2, I=16, Is=24, r=4, T=5):
    rg = np.random.default_rng(seed)
    shp = W.MoEShape(d=d, n_experts=N, top_k=K, inter=I, shared_inter=Is, lore_rank=r, dtype=dtype)
    L = dict(
        shape=shp,
        x=_rand(rg, (T, d), dtype, 1.0),
        wg=_rand(rg, (N, d), dtype, 0.3),
        w13=[_rand(rg, (2 * I, d), dtype, 0.2) for _ in range(N)],
        w2=[_rand(rg, (d, I), dtype, 0.2) for _ in range(N)],
        w13s=_rand(rg, (2 * Is, d), dtype, 0.2),
        w2s=_rand(rg, (d, Is), dtype, 0.2),
        lA=[_rand(rg, (r, d), dtype, 0.2) for _ in range(N)],
        lB=[_rand(rg, (d, r), dtype, 0.2) for _ in range(N)],
        conf=rg.random((T, K)).astype(np.float32),
    )
    return L


def f64(a, dtype):
    return torch.from_numpy(synth.as_f32(a, dtype).astype(np.float64))


def t_swiglu(x, w13, w2, I):
    return (F.silu(x @ w13[:I].T) * (x @ w13[I:].T)) @ w2.T


def dense_moe(L, idx, g):
    """torch fp64 dense MoE: S(x) + sum_k g_k E_{idx_k}(x) for every token."""
    s, dt = L["shape"], L["shape"].dtype
    x = f64(L["x"], dt)
    out = t_swiglu(x, f64(L["w13s"], dt), f64(L["w2s"], dt), s.shared_inter)
    for t in range(x.shape[0]):
        for k in range(s.top_k):
            e = int(idx[t, k])
            out[t] += float(g[t, k]) * t_swiglu(x[t:t + 1], f64(L["w13"][e], dt), f64(L["w2"][e], dt), s.inter)[0]
    return out.numpy()


def run_layer(orc, L, resident, conf=None, tau=0.5, **kw):
    cfg = orc.make_cfg(L["shape"], tau=tau)
    return orc.layer(cfg, L["x"], L["wg"], None, resident, L["conf"] if conf is None else conf,
                     L["w13"], L["w2"], L["w13s"], L["w2s"], L["lA"], L["lB"], **kw)


@pytest.mark.parametrize("dtype", [W.DTYPE_F32, W.DTYPE_BF16])
def test_swiglu_matches_torch(orc, dtype):
    L = make_layer(1, dtype)
    s = L["shape"]
    x64 = synth.as_f32(L["x"], dtype).astype(np.float64)
    for e in range(3):
        y = orc.swiglu(s.d, s.inter, dtype, L["w13"][e], L["w2"][e], x64[e])
        ref = t_swiglu(torch.from_numpy(x64[e:e + 1]), f64(L["w13"][e], dtype), f64(L["w2"][e], dtype), s.inter)
        assert np.allclose(y, ref.numpy()[0], rtol=1e-12, atol=1e-14)


def test_silu_closed_form(orc):
    # d = 1, I = 1: y = w2 * silu(a) * b with gate weight a and up weight b.
    w13 = np.array([[1.5], [-2.0]], np.float32)
    w2 = np.array([[0.25]], np.float32)
    for xv in (0.0, 1.0, -3.0):
        y = orc.swiglu(1, 1, W.DTYPE_F32, w13, w2, np.array([xv]))
        a, b = 1.5 * xv, -2.0 * xv
        assert math.isclose(y[0], 0.25 * (a / (1 + math.exp(-a))) * b, rel_tol=1e-15, abs_tol=1e-300)


@pytest.mark.parametrize("dtype", [W.DTYPE_F32, W.DTYPE_BF16])
def test_lore_delta_matches_torch(orc, dtype):
    L = make_layer(2, dtype)
    s = L["shape"]
    x64 = synth.as_f32(L["x"], dtype).astype(np.float64)
    for e in range(2):
        dl = orc.lore_delta(s.d, s.lore_rank, dtype, L["lA"][e], L["lB"][e], x64[0])
        ref = f64(L["lB"][e], dtype) @ (f64(L["lA"][e], dtype) @ torch.from_numpy(x64[0]))
        assert np.allclose(dl, ref.numpy(), rtol=1e-12, atol=1e-14)


def test_concatenated_shared_experts_equal_their_sum(orc):
    # Two shared experts (I each) form one SwiGLU block of 2I by stacking
    # [gate_a; gate_b; up_a; up_b] and [W2_a W2_b].
    r = np.random.default_rng(3)
    d, I = 24, 10
    ga, gb, ua, ub = (r.standard_normal((I, d)).astype(np.float32) * 0.3 for _ in range(4))
    wa, wb = (r.standard_normal((d, I)).astype(np.float32) * 0.3 for _ in range(2))
    x = r.standard_normal(d)
    ya = orc.swiglu(d, I, 0, np.vstack([ga, ua]), wa, x)
    yb = orc.swiglu(d, I, 0, np.vstack([gb, ub]), wb, x)
    yc = orc.swiglu(d, 2 * I, 0, np.vstack([ga, gb, ua, ub]), np.hstack([wa, wb]), x)
    assert np.allclose(yc, ya + yb, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("dtype", [W.DTYPE_F32, W.DTYPE_BF16])
def test_all_resident_is_the_dense_moe(orc, dtype):
    L = make_layer(4, dtype)
    N = L["shape"].n_experts
    r = run_layer(orc, L, np.ones(N, np.int32))
    assert (r["cls"] == HIT).all()
    assert np.allclose(r["out"], dense_moe(L, r["idx"], r["g"]), rtol=1e-11, atol=1e-12)


def test_all_exact_is_the_dense_moe_and_the_cpu_residual(orc):
    L = make_layer(5)
    N = L["shape"].n_experts
    conf = np.ones_like(L["conf"])  # every miss has conf >= tau
    r = run_layer(orc, L, np.zeros(N, np.int32), conf=conf)
    assert (r["cls"] == EXACT).all()
    dense = dense_moe(L, r["idx"], r["g"])
    assert np.allclose(r["out"], dense, rtol=1e-11, atol=1e-12)
    cfg = orc.make_cfg(L["shape"])
    resid = orc.exact_residual(cfg, L["x"], r["idx"], r["g"], r["cls"], L["w13"], L["w2"])
    assert np.allclose(r["y_shared"] + resid, dense, rtol=1e-11, atol=1e-12)


def test_exact_residual_is_zero_without_exact_slots(orc):
    L = make_layer(6)
    N = L["shape"].n_experts
    r = run_layer(orc, L, np.zeros(N, np.int32), conf=np.zeros_like(L["conf"]))
    assert (r["cls"] == LORE).all()
    cfg = orc.make_cfg(L["shape"])
    resid = orc.exact_residual(cfg, L["x"], r["idx"], r["g"], r["cls"], [None] * N, [None] * N)
    assert (resid == 0).all()


def test_full_rank_lore_factors_reproduce_the_expert(orc):
    # With n <= r independent calibration tokens H (d x n) and residuals
    # R = [E(h_i) - S(h_i)], A = [pinv(H); 0] and B = [R 0] reach zero loss in
    # Eq. 10, so B A h_i = E(h_i) - S(h_i) and an all-LoRE layer equals the dense MoE.
    L = make_layer(7, d=32, N=5, K=2, I=12, Is=20, r=8, T=4)
    s = L["shape"]
    x = f64(L["x"], 0)
    S = t_swiglu(x, f64(L["w13s"], 0), f64(L["w2s"], 0), s.shared_inter)
    Hp = torch.linalg.pinv(x.T)  # n x d
    for e in range(s.n_experts):
        R = (t_swiglu(x, f64(L["w13"][e], 0), f64(L["w2"][e], 0), s.inter) - S).T  # d x n
        A = torch.zeros(s.lore_rank, s.d, dtype=torch.float64); A[: x.shape[0]] = Hp
        B = torch.zeros(s.d, s.lore_rank, dtype=torch.float64); B[:, : x.shape[0]] = R
        L["lA"][e] = A.numpy().astype(np.float32)
        L["lB"][e] = B.numpy().astype(np.float32)
    r = run_layer(orc, L, np.zeros(s.n_experts, np.int32), conf=np.zeros_like(L["conf"]))
    assert (r["cls"] == LORE).all()
    dense = dense_moe(L, r["idx"], r["g"])
    err = np.abs(r["out"] - dense).max() / np.abs(dense).max()
    assert err < 1e-5  # factors are stored in fp32


def test_zero_factors_leave_the_shared_expert(orc):
    # B = 0 makes every LoRE term S(x), so out = (1 + sum_k g_k) S(x) for an all-LoRE token.
    L = make_layer(8)
    N = L["shape"].n_experts
    L["lB"] = [np.zeros_like(b) for b in L["lB"]]
    r = run_layer(orc, L, np.zeros(N, np.int32), conf=np.zeros_like(L["conf"]))
    coef = 1.0 + r["g"].sum(1, keepdims=True)
    assert np.allclose(r["out"], coef * r["y_shared"], rtol=1e-14, atol=1e-15)
    assert (r["y_slot"] == 0).all()


def test_zero_down_projections_leave_shared_and_lore_terms(orc):
    # W2_e = 0 for every routed expert: out = (1 + sum_LORE g) S + sum_LORE g * B A x.
    L = make_layer(9, N=8, K=3)
    s = L["shape"]
    L["w2"] = [np.zeros_like(w) for w in L["w2"]]
    resident = np.array([1, 0, 1, 0, 0, 1, 0, 0], np.int32)
    r = run_layer(orc, L, resident)
    x64 = synth.as_f32(L["x"], 0).astype(np.float64)
    for t in range(x64.shape[0]):
        expect = r["y_shared"][t].copy()
        for k in range(s.top_k):
            if r["cls"][t, k] == LORE:
                e = r["idx"][t, k]
                dl = (f64(L["lB"][e], 0) @ (f64(L["lA"][e], 0) @ torch.from_numpy(x64[t]))).numpy()
                expect += r["g"][t, k] * (r["y_shared"][t] + dl)
        assert np.allclose(r["out"][t], expect, rtol=1e-12, atol=1e-13)
    assert set(np.unique(r["cls"])) >= {HIT}


def test_token_permutation_is_equivariant(orc):
    L = make_layer(10, T=7)
    N = L["shape"].n_experts
    resident = np.array([1, 0, 1, 0, 1, 0], np.int32)
    r1 = run_layer(orc, L, resident)
    pi = np.random.default_rng(11).permutation(7)
    L2 = dict(L, x=L["x"][pi], conf=L["conf"][pi])
    r2 = run_layer(orc, L2, resident)
    assert np.array_equal(r2["idx"], r1["idx"][pi])
    assert np.array_equal(r2["cls"], r1["cls"][pi])
    assert np.allclose(r2["out"], r1["out"][pi], rtol=0, atol=0)


def test_expert_relabeling_is_invariant(orc):
    L = make_layer(12)
    N = L["shape"].n_experts
    resident = np.array([1, 1, 0, 0, 1, 0], np.int32)
    r1 = run_layer(orc, L, resident)
    sigma = np.random.default_rng(13).permutation(N)  # new id j holds old expert sigma[j]
    L2 = dict(L, wg=L["wg"][sigma], w13=[L["w13"][j] for j in sigma], w2=[L["w2"][j] for j in sigma],
              lA=[L["lA"][j] for j in sigma], lB=[L["lB"][j] for j in sigma])
    r2 = run_layer(orc, L2, resident[sigma])
    assert np.array_equal(sigma[r2["idx"]], r1["idx"])
    assert np.array_equal(r2["cls"], r1["cls"])
    assert np.allclose(r2["out"], r1["out"], rtol=1e-15, atol=1e-15)


def test_worked_example_closed_form(orc):
    """Hand-worked layer: d=2, N=3, K=2, I=I_s=r=1, one token x=(1,0).

    Router rows (0,0),(1,0),(2,0) give logits 0,1,2: top-2 = experts 2,1 with
    gates e^2/Z and e/Z, Z = 1 + e + e^2.  Expert 2 (resident) has gate row
    (1,0), up row (2,0), down column (1,0): y2 = (2 silu(1), 0).  The shared
    block has gate (1,0), up (1,0), down (1,1): S = (silu(1), silu(1)).
    Expert 1 is missing with confidence 0.25 < 0.5, so it is replaced by
    S + B A x with A = (1,0), B = (0.5,-1): B A x = (0.5, -1).
    """
    shp = W.MoEShape(d=2, n_experts=3, top_k=2, inter=1, shared_inter=1, lore_rank=1, dtype=0)
    cfg = orc.make_cfg(shp, tau=0.5)
    f = lambda *a: np.array(a, np.float32)
    x = f([1, 0])
    wg = f([0, 0], [1, 0], [2, 0])
    w13 = [f([1, 0], [1, 0]), f([1, 0], [1, 0]), f([1, 0], [2, 0])]
    w2 = [f([1], [0]), f([1], [0]), f([1], [0])]
    lA = [f([1, 0])] * 3
    lB = [f([0.5], [-1])] * 3
    resident = np.array([0, 0, 1], np.int32)
    r = orc.layer(cfg, x, wg, None, resident, f([0.25, 0.25]), w13, w2, f([1, 0], [1, 0]), f([1], [1]), lA, lB)
    e = math.e
    Z = 1 + e + e * e
    g2, g1 = e * e / Z, e / Z
    s1 = 1 / (1 + math.exp(-1))
    assert r["idx"].tolist() == [[2, 1]]
    assert r["cls"].tolist() == [[HIT, LORE]]
    assert np.allclose(r["g"][0], [g2, g1], rtol=1e-15)
    expect = np.array([s1 + g2 * 2 * s1 + g1 * (s1 + 0.5), s1 + g1 * (s1 - 1.0)])
    assert np.allclose(r["out"][0], expect, rtol=1e-15, atol=1e-16)
    # bucketing: slot 0 (expert 2, HIT) first, then slot 1 (expert 1, LORE)
    assert r["perm"].tolist() == [0, 1]
    assert r["offsets"].tolist() == [[0, 0, 0, 1], [1, 1, 2, 2], [2, 2, 2, 2]]
