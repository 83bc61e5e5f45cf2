"""Pins of the oracle's speculative-prefetching functions (Sec. 4.1, Eq. 2-5, Alg. 1).

Each check compares the oracle with something it does not compute itself: a brute-force
rounding, the closed form of Eq. 4 on exact binary inputs, the oracle's own routing and
layer output (separately pinned), or hand-worked queues and cache traces.
"""
import numpy as np
import pytest

from paper_2608_21240_amd import synth
from paper_2608_21240_amd.workloads import MoEShape, Workload

F32, BF16 = 0, 1


def _bf16_brute(v: float) -> float:
    """Nearest bf16 value by enumeration of the bit patterns around v, ties to an even mantissa."""
    f = np.array([v], np.float32).view(np.uint32)[0] >> 16
    best = None
    for b in range(max(int(f) - 2, 0), min(int(f) + 3, 0xFFFF) + 1):
        c = float(np.array([b << 16], np.uint32).view(np.float32)[0])
        if not np.isfinite(c) or np.sign(c) != np.sign(v):
            continue
        key = (abs(c - v), b & 1)
        if best is None or key < best[0]:
            best = (key, c)
    return best[1]


def test_round_to_matches_brute_force(orc):
    r = np.random.default_rng(0)
    vals = np.concatenate([r.standard_normal(400) * 10.0 ** r.integers(-6, 6, 400),
                           [1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 3.0 * 2 ** -9]])
    for v in vals:
        assert orc.round_to(BF16, v) == _bf16_brute(float(v)), v
        assert orc.round_to(F32, v) == float(np.float32(v))
    # double rounding through fp32 would differ here: just above a bf16 tie
    v = 1 + 2 ** -8 + 2 ** -40
    assert orc.round_to(BF16, v) == 1 + 2 ** -7


def test_h_min_closed_form(orc):
    # exact binary inputs: P * 2^20 / (2^30 * (2^-11 + 2 * 2^-12)) = P exactly
    for P in (0, 1, 3, 7):
        assert orc.h_min(P, 2.0 ** 20, 2.0 ** 30, 2.0 ** -11, 2, 2.0 ** -12) == P
    # a DSV2 expert (17,301,504 B), 4 per layer, 25 GB/s, 0.1 ms attention + 6 x 0.05 ms experts:
    # 69,206,016 / (25e9 * 4e-4) = 6.92 -> 7
    assert orc.h_min(4, 17301504, 25e9, 1e-4, 6, 5e-5) == 7
    # just over an integer rounds up
    assert orc.h_min(1, 2.0 ** 20 + 1, 2.0 ** 30, 2.0 ** -11, 2, 2.0 ** -12) == 2
    assert orc.h_min(1, 1.0, 1.0, 0.0, 4, 0.0) == -1
    assert orc.h_min(1, 1.0, 0.0, 1.0, 4, 1.0) == -1


def _layers(shape, n, seed, zero=False):
    """Weights of n future layers (router, shared block, LoRE factors of every expert)."""
    wl = Workload("spec", shape, tokens=1, resident=0, skew=False, seed=seed)
    out = []
    for j in range(n):
        w13s, w2s = synth.gen_shared(wl, j)
        lore = [synth.gen_lore(wl, j, e) for e in range(shape.n_experts)]
        lA = [a for a, _ in lore]
        lB = [b for _, b in lore]
        if zero:
            w13s, w2s = np.zeros_like(w13s), np.zeros_like(w2s)
            lA = [np.zeros_like(a) for a in lA]
            lB = [np.zeros_like(b) for b in lB]
        out.append(dict(wg=synth.gen_router(wl, j), bias=None, w13s=w13s, w2s=w2s, lA=lA, lB=lB))
    return out


SMALL = MoEShape(d=64, n_experts=12, top_k=3, inter=32, shared_inter=48, lore_rank=8, dtype=F32)


def _x(shape, T, seed):
    r = np.random.default_rng(seed)
    return synth.to_storage(r.standard_normal((T, shape.d)).astype(np.float32), shape.dtype)


@pytest.mark.parametrize("dtype", [F32, BF16])
def test_confidence_is_top_k_softmax_mass(orc, dtype):
    shape = MoEShape(64, 12, 3, 32, 48, 8, dtype)
    cfg = orc.make_cfg(shape)
    L = _layers(shape, 1, 1)[0]
    x = _x(shape, 9, 2)
    halted = np.zeros(9, np.int32)
    pidx, pprob, conf, _ = orc.spec_step(cfg, x, 1, 1, 0.0, True, L["wg"], None, L["w13s"], L["w2s"], L["lA"],
                                         L["lB"], halted)
    xf = synth.as_f32(x, dtype).astype(np.float64)
    wf = synth.as_f32(L["wg"], dtype).astype(np.float64)
    z = xf @ wf.T
    p = np.exp(z - z.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    order = np.lexsort((np.arange(12)[None, :].repeat(9, 0), -z), axis=1)[:, :3]
    assert np.array_equal(pidx, order)
    assert np.allclose(pprob, np.take_along_axis(p, order, 1), rtol=1e-12, atol=0)
    assert np.allclose(conf, np.take_along_axis(p, order, 1).sum(1), rtol=1e-12, atol=0)


@pytest.mark.parametrize("l_min,tau", [(1, 0.0), (1, 2.0), (3, 2.0), (2, 0.6), (1, 0.5)])
def test_zero_surrogates_keep_the_state_and_route_each_future_layer(orc, l_min, tau):
    """With S = 0 and B A = 0 the draft state never moves, so depth j predicts exactly the
    oracle's routing of x by layer l+j's router; halting follows Eq. 5 and Alg. 1 step 3."""
    shape = SMALL
    cfg = orc.make_cfg(shape)
    n, T = 5, 11
    layers = _layers(shape, n, 3, zero=True)
    x = _x(shape, T, 4)
    res = orc.spec_rollout(cfg, x, layers, l_min, tau)
    stop = np.full(T, n)
    for j, L in enumerate(layers):
        z, _ = orc.router_logits(cfg, x, L["wg"])
        ridx, rg, _ = orc.gates_topk(cfg, z)
        rt = dict(idx=ridx, g=rg)
        assert np.array_equal(res["h"][j], x)
        live = stop >= j + 1
        assert np.array_equal(res["idx"][j][live], rt["idx"][live])
        assert (res["idx"][j][~live] == -1).all() and np.isnan(res["conf"][j][~live]).all()
        cf = rt["g"].sum(1)
        assert np.allclose(res["conf"][j][live], cf[live], rtol=1e-12)
        newly = live & (j + 1 >= l_min) & (cf < tau)
        stop[newly] = j + 1
    assert np.array_equal(res["depth"], stop)


@pytest.mark.parametrize("dtype", [F32, BF16])
def test_one_depth_update_is_the_all_lore_layer_output_minus_the_shared_term(orc, dtype):
    """h' = x + sum_k pi_k (S(x) + B_k A_k x); the oracle's layer output with every slot LoRE
    and gates pi is S(x) + sum_k pi_k (S(x) + B_k A_k x), so h' = round(x + out - S(x))."""
    shape = MoEShape(64, 12, 3, 32, 48, 8, dtype)
    cfg = orc.make_cfg(shape)
    L = _layers(shape, 1, 5)[0]
    T = 6
    x = _x(shape, T, 6)
    halted = np.zeros(T, np.int32)
    pidx, pprob, conf, h1 = orc.spec_step(cfg, x, 1, 9, 0.5, False, L["wg"], None, L["w13s"], L["w2s"], L["lA"],
                                          L["lB"], halted)
    assert (halted == 0).all()
    xf = synth.as_f32(x, dtype).astype(np.float64)
    for t in range(T):
        out, ys, _ = orc.token_output(cfg, x[t], pidx[t], pprob[t], np.full(3, orc.LORE, np.uint8),
                                      [None] * 12, [None] * 12, L["w13s"], L["w2s"], L["lA"], L["lB"])
        want = np.array([orc.round_to(dtype, v) for v in xf[t] + out - ys])
        got = synth.as_f32(h1[t], dtype).astype(np.float64)
        ulp = np.abs(want) * (2.0 ** -7 if dtype == BF16 else 2.0 ** -23)
        assert np.all(np.abs(got - want) <= ulp), t


def test_halted_tokens_keep_state_and_queue_nothing(orc):
    shape = SMALL
    cfg = orc.make_cfg(shape)
    L = _layers(shape, 1, 7)[0]
    T = 5
    x = _x(shape, T, 8)
    halted = np.array([0, 1, 0, 1, 0], np.int32)
    pidx, pprob, conf, h = orc.spec_step(cfg, x, 2, 1, 0.0, False, L["wg"], None, L["w13s"], L["w2s"], L["lA"],
                                         L["lB"], halted)
    assert (pidx[[1, 3]] == -1).all() and (pprob[[1, 3]] == 0).all() and np.isnan(conf[[1, 3]]).all()
    assert np.array_equal(h[[1, 3]], x[[1, 3]]) and not np.array_equal(h[[0, 2, 4]], x[[0, 2, 4]])
    # the last depth enqueues but does not move the state
    halted = np.zeros(T, np.int32)
    _, _, _, h = orc.spec_step(cfg, x, 2, 1, 0.0, True, L["wg"], None, L["w13s"], L["w2s"], L["lA"], L["lB"],
                               halted)
    assert np.array_equal(h, x) and (halted == 0).all()


def test_prefetch_queue_hand_worked(orc):
    # depth 0: token 0 -> {3: .5, 1: .2}, token 1 -> {1: .4, 5: .3}: masses 3 .5, 1 .6, 5 .3
    # depth 1: token 0 halted (-1), token 1 -> {2: .25, 7: .25}: tie -> lower id first
    idx = np.array([[[3, 1], [1, 5]], [[-1, -1], [7, 2]]], np.int32)
    prob = np.array([[[.5, .2], [.4, .3]], [[0, 0], [.25, .25]]])
    assert orc.prefetch_queue(8, idx, prob, 8) == [[1, 3, 5], [2, 7]]
    assert orc.prefetch_queue(8, idx, prob, 2) == [[1, 3], [2, 7]]
    assert orc.prefetch_queue(8, idx, prob, 0) == [[], []]


def test_lru_prefetch_hand_worked(orc):
    st = orc.LRUState(10, 4, [0, 1, 2, -1])
    st.last_use[:] = [5, 3, 4, -1]
    # step 6, list [9, 1, 8, 7]: 9 takes the empty slot; 1 is resident; 8 evicts expert 2
    # (last use 4; expert 1 is listed so it is no victim); 7 evicts expert 0 (last use 5)
    adm, ev = st.prefetch(6, [9, 1, 8, 7], 5)
    assert adm.tolist() == [9, 8, 7] and ev.tolist() == [-1, 2, 0]
    assert st.slot_expert.tolist() == [7, 1, 8, 9] and st.last_use.tolist() == [6, 3, 6, 6]
    # experts used in this step are never victims; max_prefetch caps the admissions
    st2 = orc.LRUState(10, 4, [0, 1, 2, 3])
    st2.last_use[:] = [6, 6, 2, 1]
    adm, ev = st2.prefetch(6, [4, 5, 6], 2)
    assert adm.tolist() == [4, 5] and ev.tolist() == [3, 2]
    adm, ev = st2.prefetch(6, [7], 3)
    assert adm.tolist() == [] and ev.tolist() == []


def test_halting_is_strict_at_the_threshold(orc):
    """A zero router gives the uniform distribution: with N = 16 and K = 4 the confidence is
    exactly 0.25, so tau = 0.25 keeps going (C < tau is false) and any larger tau halts."""
    shape = MoEShape(64, 16, 4, 32, 48, 8, F32)
    cfg = orc.make_cfg(shape)
    L = _layers(shape, 1, 9)[0]
    x = _x(shape, 3, 10)
    wg0 = np.zeros_like(L["wg"])
    for tau, halts in ((0.25, False), (np.nextafter(0.25, 1.0), True), (0.2, False)):
        halted = np.zeros(3, np.int32)
        _, pprob, conf, _ = orc.spec_step(cfg, x, 1, 1, tau, False, wg0, None, L["w13s"], L["w2s"], L["lA"],
                                          L["lB"], halted)
        assert (conf == 0.25).all() and (pprob == 1 / 16).all()
        assert (halted == int(halts)).all(), tau
