"""Pins for the oracle's routing steps (Eq. 1 router + TopK, gate scores,
confidence, the hit / low-confidence / exact rule, and slot bucketing).

Each check comes from something other than the oracle's own code: a library
matmul, a full sort, closed forms, or invariants the definitions force.
"""
import math

import numpy as np
import pytest
import torch

from paper_2608_21240_amd import synth, workloads as W

HIT, LORE, EXACT = 0, 1, 2


def _shape(d, N, K, dtype=W.DTYPE_F32):
    return W.MoEShape(d=d, n_experts=N, top_k=K, inter=8, shared_inter=8, lore_rank=2, dtype=dtype)


def _rand(seed, shape, dtype, std=1.0):
    a = np.random.default_rng(seed).standard_normal(shape).astype(np.float32) * np.float32(std)
    return synth.to_storage(a, dtype)


@pytest.mark.parametrize("dtype", [W.DTYPE_F32, W.DTYPE_BF16])
def test_router_logits_match_library_matmul(orc, dtype):
    shp = _shape(48, 12, 3, dtype)
    cfg = orc.make_cfg(shp)
    x = _rand(1, (5, 48), dtype)
    wg = _rand(2, (12, 48), dtype, 0.3)
    bias = np.random.default_rng(3).standard_normal(12).astype(np.float32)
    z, zabs = orc.router_logits(cfg, x, wg, bias)
    xt = torch.from_numpy(synth.as_f32(x, dtype).astype(np.float64))
    wt = torch.from_numpy(synth.as_f32(wg, dtype).astype(np.float64))
    ref = (xt @ wt.T).numpy() + bias.astype(np.float64)
    assert np.allclose(z, ref, rtol=0, atol=1e-12)
    assert np.allclose(zabs, (xt.abs() @ wt.abs().T).numpy(), rtol=1e-12, atol=0)


@pytest.mark.parametrize("seed", range(20))
def test_topk_equals_full_sort(orc, seed):
    r = np.random.default_rng(100 + seed)
    N = int(r.integers(1, 17))
    K = int(r.integers(1, N + 1))
    cfg = orc.make_cfg(_shape(4, N, K))
    z = r.standard_normal((6, N))
    z[:, : N // 2] = np.round(z[:, : N // 2])  # plant exact ties
    idx, g, probs = orc.gates_topk(cfg, z)
    for t in range(6):
        order = sorted(range(N), key=lambda e: (-z[t, e], e))
        assert list(idx[t]) == order[:K]
        ex = np.exp(z[t] - z[t].max())
        assert np.allclose(g[t], (ex / ex.sum())[order[:K]], rtol=1e-14, atol=0)


def test_zero_input_is_an_exact_tie(orc):
    N, K = 8, 3
    shp = _shape(16, N, K)
    cfg = orc.make_cfg(shp)
    x = np.zeros((2, 16), np.float32)
    wg = _rand(5, (N, 16), W.DTYPE_F32)
    r = orc.route(cfg, x, wg, None, np.zeros(N, np.int32), np.full((2, K), 0.9, np.float32))
    assert (r["z"] == 0).all()
    assert (r["idx"] == np.arange(K)).all()
    assert (r["g"] == 1.0 / N).all()


def test_bias_only_logits_give_popularity(orc):
    # x = 0 and b_e = ln p_e: the softmax returns p itself; ties (p equal) keep the lower id.
    p = np.array([0.1, 0.3, 0.05, 0.3, 0.25], np.float64)
    cfg = orc.make_cfg(_shape(8, 5, 3))
    bias = np.log(p).astype(np.float32)
    z, _ = orc.router_logits(cfg, np.zeros((1, 8), np.float32), np.zeros((5, 8), np.float32), bias)
    idx, g, probs = orc.gates_topk(cfg, z)
    assert list(idx[0]) == [1, 3, 4]
    pb = np.exp(bias.astype(np.float64)); pb /= pb.sum()
    assert np.allclose(probs[0], pb, rtol=1e-14)
    assert np.allclose(probs[0], p, rtol=1e-6)


def test_two_experts_reduce_to_sigmoid(orc):
    cfg = orc.make_cfg(_shape(4, 2, 1))
    z = np.array([[0.7, -0.4], [-2.0, 1.5]])
    idx, g, _ = orc.gates_topk(cfg, z)
    assert list(idx[:, 0]) == [0, 1]
    for t in range(2):
        gap = abs(z[t, 0] - z[t, 1])
        assert math.isclose(g[t, 0], 1.0 / (1.0 + math.exp(-gap)), rel_tol=1e-15)


@pytest.mark.parametrize("norm", [0, 1])
def test_gate_invariants(orc, norm):
    shp = _shape(32, 16, 5)
    cfg = orc.make_cfg(shp, norm_topk=norm)
    z = np.random.default_rng(9).standard_normal((50, 16)) * 2
    idx, g, probs = orc.gates_topk(cfg, z)
    assert np.allclose(probs.sum(1), 1.0, atol=16 * 2.0 ** -52)
    assert (np.diff(g, axis=1) <= 0).all()
    assert (g > 0).all()
    if norm:
        assert np.allclose(g.sum(1), 1.0, atol=1e-15)
        raw = np.take_along_axis(probs, idx.astype(np.int64), 1)
        assert np.allclose(g, raw / raw.sum(1, keepdims=True), rtol=1e-15)
    else:
        assert (g.sum(1) <= 1.0 + 1e-15).all()
        assert np.array_equal(g, np.take_along_axis(probs, idx.astype(np.int64), 1))


def test_router_row_permutation_relabels_experts(orc):
    N, K = 10, 4
    cfg = orc.make_cfg(_shape(24, N, K))
    x = _rand(11, (7, 24), W.DTYPE_F32)
    wg = _rand(12, (N, 24), W.DTYPE_F32)
    sigma = np.random.default_rng(13).permutation(N)  # new expert j = old expert sigma[j]
    z1, _ = orc.router_logits(cfg, x, wg)
    z2, _ = orc.router_logits(cfg, x, wg[sigma])
    i1, g1, _ = orc.gates_topk(cfg, z1)
    i2, g2, _ = orc.gates_topk(cfg, z2)
    assert np.array_equal(sigma[i2], i1)
    assert np.allclose(g1, g2, rtol=1e-14, atol=0)  # the softmax sum runs in another order


def test_confidence_modes(orc):
    shp = _shape(8, 6, 3)
    g = np.array([[0.4, 0.2, 0.1], [0.3, 0.3, 0.05]])
    cin = np.array([[0.9, 0.1, 0.5], [0.2, 0.7, 0.4]], np.float32)
    assert np.array_equal(orc.confidence(orc.make_cfg(shp, conf_mode=0), g, cin), cin)
    assert np.array_equal(orc.confidence(orc.make_cfg(shp, conf_mode=1), g), g.astype(np.float32))
    ren = orc.confidence(orc.make_cfg(shp, conf_mode=2), g)
    assert np.allclose(ren, (g / g.sum(1, keepdims=True)).astype(np.float32), rtol=0, atol=0)
    assert np.allclose(ren.sum(1), 1.0, atol=1e-6)


def test_classification_rule(orc):
    shp = _shape(8, 6, 3)
    cfg = orc.make_cfg(shp, tau=0.5)
    idx = np.array([[0, 1, 2], [3, 4, 5], [1, 3, 5]], np.int32)
    resident = np.array([1, 0, 0, 1, 0, 0], np.int32)
    conf = np.array([[0.0, 0.49, 0.5], [0.99, np.nan, 0.5000001], [0.1, 0.9, -1.0]], np.float32)
    cls = orc.classify(cfg, idx, resident, conf)
    assert cls.tolist() == [[HIT, LORE, EXACT], [HIT, EXACT, EXACT], [LORE, HIT, LORE]]


@pytest.mark.parametrize("seed", range(10))
def test_bucketing_is_the_stable_sort_by_class_then_expert(orc, seed):
    r = np.random.default_rng(200 + seed)
    N = int(r.integers(1, 20)); K = int(r.integers(1, N + 1)); T = int(r.integers(0, 40))
    cfg = orc.make_cfg(_shape(8, N, K))
    idx = np.stack([r.permutation(N)[:K] for _ in range(T)]).astype(np.int32) if T else np.zeros((0, K), np.int32)
    cls = r.integers(0, 3, size=(T, K)).astype(np.uint8)
    offsets, perm, inv, counts = orc.bucket(cfg, idx, cls)
    S = T * K
    flat_i, flat_c = idx.reshape(-1), cls.reshape(-1)
    expect = sorted(range(S), key=lambda s: (int(flat_c[s]), int(flat_i[s]), s))
    assert perm.tolist() == expect
    assert (inv[perm] == np.arange(S)).all() and (perm[inv] == np.arange(S)).all()
    hist = np.zeros((3, N), np.int64)
    np.add.at(hist, (flat_c.astype(np.int64), flat_i.astype(np.int64)), 1)
    flat_off = np.concatenate([[0], np.cumsum(hist.reshape(-1))])
    for c in range(3):
        assert offsets[c, :N].tolist() == flat_off[c * N:(c + 1) * N].tolist()
        assert offsets[c, N] == flat_off[(c + 1) * N]
        assert counts[c] == hist[c].sum()
    assert counts.sum() == S
