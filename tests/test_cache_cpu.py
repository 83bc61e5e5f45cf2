"""The library's expert cache (moe_cache_*) in bookkeeping-only mode, against the
oracle's LRU step: identical admitted / evicted experts and identical per-slot
state after every layer call, on hand-worked and random traces and on traces
with the stack workload's shapes.  No GPU is needed (no pools, no copies)."""
import numpy as np
import pytest

from paper_2608_21240_amd import spice
from paper_2608_21240_amd.workloads import MoEShape, WORKLOADS

HIT, LORE, EXACT = 0, 1, 2


def _cfg(N, K, C):
    shape = MoEShape(d=64, n_experts=N, top_k=K, inter=32, shared_inter=32, lore_rank=8, dtype=1)
    return spice.make_cfg(shape, C)


def _classes(resident, idx, r, p_lore=0.5):
    return np.where(resident[idx] == 1, HIT, np.where(r.random(idx.shape) < p_lore, LORE, EXACT)).astype(np.uint8)


def test_hand_worked_trace_matches_oracle(orc):
    cfg = _cfg(6, 2, 3)
    lib = spice.ExpertCache(cfg, 1, [[0, 1, 2]])
    ref = orc.LRUState(6, 3)
    trace = [
        (0, [[0, 3], [4, 3]], [[HIT, EXACT], [LORE, EXACT]], 1),
        (1, [[2, 5], [1, 5]], [[HIT, EXACT], [EXACT, EXACT]], 1),
        (2, [[0, 1], [3, 4]], [[EXACT, EXACT], [HIT, EXACT]], 2),
        (3, [[4, 5]], [[EXACT, EXACT]], 4),
        (4, [[3, 4], [5, 0]], [[HIT, HIT], [HIT, EXACT]], 4),
    ]
    for step, idx, cls, ma in trace:
        a, e = lib.step(0, step, np.array(idx), np.array(cls), ma)
        ra, re = ref.step(step, np.array(idx, np.int32), np.array(cls, np.uint8), ma)
        assert (a, e) == (ra.tolist(), re.tolist())
        se, lu = lib.state(0)
        assert se.tolist() == ref.slot_expert.tolist() and lu.tolist() == ref.last_use.tolist()
    lib.close()


@pytest.mark.parametrize("seed", range(6))
def test_random_multilayer_traces_match_oracle(orc, seed):
    r = np.random.default_rng(100 + seed)
    N, K, C, L, T = 16, 3, 5, 3, 7
    init = np.stack([r.permutation(N)[:C] for _ in range(L)]).astype(np.int32)
    if seed % 2:
        init[:, -1] = -1  # an empty slot in every layer
    lib = spice.ExpertCache(_cfg(N, K, C), L, init)
    refs = [orc.LRUState(N, C, init[l]) for l in range(L)]
    for step in range(40):
        for l in range(L):
            res = refs[l].resident_mask()
            idx = np.stack([r.permutation(N)[:K] for _ in range(T)]).astype(np.int32)
            cls = _classes(res, idx, r, p_lore=float(r.random()))
            ma = int(r.integers(0, 5))
            a, e = lib.step(l, step, idx, cls, ma)
            ra, re = refs[l].step(step, idx, cls, ma)
            assert (a, e) == (ra.tolist(), re.tolist()), (step, l)
            se, lu = lib.state(l)
            assert se.tolist() == refs[l].slot_expert.tolist() and lu.tolist() == refs[l].last_use.tolist()
    lib.close()


def test_inconsistent_classes_are_ignored_like_the_oracle(orc):
    # HIT for a non-resident expert and EXACT for a resident one change nothing
    r = np.random.default_rng(7)
    N, K, C = 12, 4, 4
    lib = spice.ExpertCache(_cfg(N, K, C), 1, [list(range(C))])
    ref = orc.LRUState(N, C)
    for step in range(30):
        idx = np.stack([r.permutation(N)[:K] for _ in range(5)]).astype(np.int32)
        cls = r.integers(0, 3, idx.shape).astype(np.uint8)
        a, e = lib.step(0, step, idx, cls, 2)
        ra, re = ref.step(step, idx, cls, 2)
        assert (a, e) == (ra.tolist(), re.tolist())
        assert lib.state(0)[0].tolist() == ref.slot_expert.tolist()
    lib.close()


def test_stack_shaped_trace_matches_oracle(orc):
    """Stack-workload shapes (N=64, K=6, T=64, C=24) with Zipf(1.1)-skewed routing."""
    wl = WORKLOADS["dsv2_stack"]
    s = wl.shape
    r = np.random.default_rng(11)
    N, K, C, T, L = s.n_experts, s.top_k, wl.cache_slots, wl.tokens, 2
    p = np.arange(1, N + 1, dtype=np.float64) ** -1.1
    p /= p.sum()
    init = np.tile(np.arange(C, dtype=np.int32), (L, 1))
    lib = spice.ExpertCache(spice.make_cfg(s, C), L, init)
    refs = [orc.LRUState(N, C) for _ in range(L)]
    for step in range(24):
        for l in range(L):
            idx = np.stack([r.choice(N, K, replace=False, p=p) for _ in range(T)]).astype(np.int32)
            cls = _classes(refs[l].resident_mask(), idx, r)
            a, e = lib.step(l, step, idx, cls, 4)
            ra, re = refs[l].step(step, idx, cls, 4)
            assert (a, e) == (ra.tolist(), re.tolist())
            assert lib.state(l)[1].tolist() == refs[l].last_use.tolist()
    lib.close()


def test_errors_leave_state_unchanged():
    cfg = _cfg(8, 2, 3)
    with pytest.raises(spice.SpiceError):
        spice.ExpertCache(cfg, 1, [[0, 0, 1]])  # an expert twice
    with pytest.raises(spice.SpiceError):
        spice.ExpertCache(cfg, 1, [[0, 1, 8]])  # id out of range
    with pytest.raises(spice.SpiceError):
        spice.ExpertCache(spice.make_cfg(MoEShape(64, 8, 2, 32, 32, 8, 1), 9), 1, [list(range(8)) + [-1]])
    with pytest.raises(spice.SpiceError):
        spice.ExpertCache(cfg, 1, [[0, 1, 2]], load=True)  # load needs pools
    c = spice.ExpertCache(cfg, 2, [[0, 1, 2], [3, 4, -1]])
    before = [c.state(l) for l in range(2)]
    for bad_idx, bad_cls in (([[0, 9]], [[HIT, EXACT]]), ([[0, 5]], [[HIT, 4]])):
        with pytest.raises(spice.SpiceError):
            c.step(0, 0, np.array(bad_idx), np.array(bad_cls), 2)
    with pytest.raises(spice.SpiceError):
        c.step(2, 0, np.array([[0, 5]]), np.array([[HIT, EXACT]]), 1)  # layer out of range
    with pytest.raises(spice.SpiceError):
        c.step(0, 0, np.array([[0, 5]]), np.array([[HIT, EXACT]]), -1)
    after = [c.state(l) for l in range(2)]
    for (s0, l0), (s1, l1) in zip(before, after):
        assert s0.tolist() == s1.tolist() and l0.tolist() == l1.tolist()
    # an empty slot is filled before any resident expert is evicted
    a, e = c.step(1, 0, np.array([[6, 7]]), np.array([[EXACT, EXACT]]), 1)
    assert (a, e) == ([6], [-1])
    c.wait(1)  # bookkeeping only: nothing to wait for
    c.close()
    c.close()
