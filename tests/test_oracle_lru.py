"""Pins for the oracle's LRU expert-cache step (the stack workload).

The paper names LRU only as a cache policy; the rules used here are the
readings recorded in the design notes: hit experts are touched; exact-miss
experts are admitted (most tokens first, then lowest id) into the slot of the
least recently used expert not used in this step (ties -> lowest expert id);
LoRE misses are never admitted (Sec. 4.2: they trigger no host-to-device
transfer); at most max_admit per step (a bounded copy queue, Sec. 4.1).
"""
import numpy as np
import pytest

HIT, LORE, EXACT = 0, 1, 2


def test_hand_worked_trace(orc):
    st = orc.LRUState(n_experts=6, C=3)  # slots hold experts 0,1,2, never used
    # step 0: expert 0 hit; expert 3 exact twice; expert 4 LoRE (never admitted).
    # Victim among slots unused this step: (last_use, id) = (-1,1) < (-1,2) -> evict 1.
    a, e = st.step(0, [[0, 3], [4, 3]], [[HIT, EXACT], [LORE, EXACT]], max_admit=1)
    assert (a.tolist(), e.tolist()) == ([3], [1])
    assert st.slot_expert.tolist() == [0, 3, 2] and st.last_use.tolist() == [0, 0, -1]
    # step 1: 2 hit; 5 exact x2, 1 exact x1 -> candidate 5 first; victims (0,0),(0,3) -> evict 0.
    a, e = st.step(1, [[2, 5], [1, 5]], [[HIT, EXACT], [EXACT, EXACT]], max_admit=1)
    assert (a.tolist(), e.tolist()) == ([5], [0])
    assert st.slot_expert.tolist() == [5, 3, 2] and st.last_use.tolist() == [1, 0, 1]
    # step 2: 3 hit; exact 0,1,4 once each -> order 0,1,4; two admissions:
    # 0 evicts min((1,5),(1,2)) = expert 2; then 1 evicts expert 5.
    a, e = st.step(2, [[0, 1], [3, 4]], [[EXACT, EXACT], [HIT, EXACT]], max_admit=2)
    assert (a.tolist(), e.tolist()) == ([0, 1], [2, 5])
    assert st.slot_expert.tolist() == [1, 3, 0] and st.last_use.tolist() == [2, 2, 2]
    # step 3: no hits; exact 4, 5 -> 4 evicts lowest id among last_use 2 (expert 0), 5 evicts 1.
    a, e = st.step(3, [[4, 5]], [[EXACT, EXACT]], max_admit=4)
    assert (a.tolist(), e.tolist()) == ([4, 5], [0, 1])
    assert st.slot_expert.tolist() == [5, 3, 4] and st.last_use.tolist() == [3, 2, 3]
    # step 4: every slot used this step -> nothing can be evicted.
    a, e = st.step(4, [[3, 4], [5, 0]], [[HIT, HIT], [HIT, EXACT]], max_admit=4)
    assert a.size == 0 and e.size == 0
    assert st.last_use.tolist() == [4, 4, 4]


@pytest.mark.parametrize("seed", range(8))
def test_random_trace_invariants(orc, seed):
    r = np.random.default_rng(seed)
    N, C, K, T = 16, 5, 3, 6
    st = orc.LRUState(N, C)
    for step in range(30):
        res = st.resident_mask()
        idx = np.stack([r.permutation(N)[:K] for _ in range(T)]).astype(np.int32)
        cls = np.where(res[idx] == 1, HIT, np.where(r.random((T, K)) < 0.5, LORE, EXACT)).astype(np.uint8)
        before = st.slot_expert.copy()
        max_admit = int(r.integers(0, 4))
        a, e = st.step(step, idx, cls, max_admit)
        exact_experts = set(idx[cls == EXACT].tolist())
        hit_experts = set(idx[cls == HIT].tolist())
        assert len(a) <= max_admit
        assert set(a.tolist()) <= exact_experts
        assert not (set(e.tolist()) & hit_experts)
        assert len(set(st.slot_expert.tolist())) == C  # no duplicates, size constant
        assert set(st.slot_expert.tolist()) == (set(before.tolist()) - set(e.tolist())) | set(a.tolist())
        # admission order: token count descending, then id ascending
        cnt = {x: int((idx[cls == EXACT] == x).sum()) for x in exact_experts}
        keys = [(-cnt[x], x) for x in a.tolist()]
        assert keys == sorted(keys)
        if len(a) < max_admit:
            # either every exact expert was admitted, or every slot was used this step
            assert set(a.tolist()) == exact_experts or (st.last_use == step).all()
