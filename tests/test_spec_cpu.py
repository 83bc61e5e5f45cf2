"""Host side of speculative prefetching (Sec. 4.1) against the oracle: the minimum
lookahead of Eq. 4, the per-depth issue lists of the prefetch intents (Eq. 3) and the
speculative admissions of the expert cache, interleaved with its demand admissions.
No GPU is needed (the cache runs in bookkeeping-only mode)."""
import numpy as np
import pytest

from paper_2608_21240_amd import spice
from paper_2608_21240_amd.workloads import MoEShape

HIT, LORE, EXACT = 0, 1, 2


def _cfg(N, K, C=1):
    return spice.make_cfg(MoEShape(d=64, n_experts=N, top_k=K, inter=32, shared_inter=32, lore_rank=8, dtype=1), C)


def test_h_min_matches_oracle(orc):
    r = np.random.default_rng(0)
    for _ in range(500):
        P, Me = float(r.integers(0, 12)), float(r.choice([17301504, 55050240, 393216]))
        B = float(r.uniform(5e9, 60e9))
        ta, te, K = float(r.uniform(0, 3e-4)), float(r.uniform(0, 1e-4)), int(r.integers(1, 9))
        assert spice.moe_prefetch_h_min(P, Me, B, ta, K, te) == orc.h_min(P, Me, B, ta, K, te)
    assert spice.moe_prefetch_h_min(1, 1, 1, 0, 3, 0) == -1
    assert spice.moe_prefetch_h_min(1, 1, 0, 1, 3, 1) == -1
    assert spice.moe_prefetch_h_min(-1, 1, 1, 1, 3, 1) == -1


@pytest.mark.parametrize("seed", range(5))
def test_prefetch_queue_matches_oracle(orc, seed):
    r = np.random.default_rng(seed)
    N, K, T, D = 24, 4, 9, 5
    idx = np.stack([[r.permutation(N)[:K] for _ in range(T)] for _ in range(D)]).astype(np.int32)
    prob = r.random((D, T, K)).astype(np.float32)
    prob[:, :, 0] = np.float32(0.25)  # many equal masses: the tie rule decides
    halted = r.random((D, T)) < 0.3
    idx[halted] = -1
    prob[halted] = 0
    for cap in (0, 3, N):
        got = spice.moe_prefetch_queue(_cfg(N, K), idx, prob, cap)
        assert got == orc.prefetch_queue(N, idx, prob.astype(np.float64), cap), cap


def test_prefetch_queue_rejects_bad_ids():
    with pytest.raises(spice.SpiceError):
        spice.moe_prefetch_queue(_cfg(8, 2), np.array([[[0, 8]]], np.int32), np.ones((1, 1, 2), np.float32), 4)
    with pytest.raises(spice.SpiceError):
        spice.moe_prefetch_queue(_cfg(8, 2), np.array([[[0, -2]]], np.int32), np.ones((1, 1, 2), np.float32), 4)


@pytest.mark.parametrize("seed", range(6))
def test_cache_prefetch_interleaved_with_steps_matches_oracle(orc, seed):
    r = np.random.default_rng(200 + seed)
    N, K, C, L, T = 16, 3, 5, 4, 6
    init = np.stack([r.permutation(N)[:C] for _ in range(L)]).astype(np.int32)
    if seed % 2:
        init[:, 0] = -1
    lib = spice.ExpertCache(_cfg(N, K, C), L, init)
    refs = [orc.LRUState(N, C, init[l]) for l in range(L)]
    for step in range(25):
        for l in range(L):
            res = refs[l].resident_mask()
            idx = np.stack([r.permutation(N)[:K] for _ in range(T)]).astype(np.int32)
            cls = np.where(res[idx] == 1, HIT, np.where(r.random(idx.shape) < 0.5, LORE, EXACT)).astype(np.uint8)
            a, e = lib.step(l, step, idx, cls, 2)
            ra, re = refs[l].step(step, idx, cls, 2)
            assert (a, e) == (ra.tolist(), re.tolist())
            # predictions for the next layers of this step, as an anchor at layer l would issue
            for j in range(l + 1, min(l + 3, L)):
                q = r.permutation(N)[: int(r.integers(0, 7))].astype(np.int32)
                cap = int(r.integers(0, 4))
                a, e = lib.prefetch(j, step, q, cap)
                ra, re = refs[j].prefetch(step, q, cap)
                assert (a, e) == (ra.tolist(), re.tolist()), (step, l, j)
            for j in range(L):
                se, lu = lib.state(j)
                assert se.tolist() == refs[j].slot_expert.tolist() and lu.tolist() == refs[j].last_use.tolist()
    lib.close()


def test_cache_prefetch_errors_leave_state_unchanged():
    c = spice.ExpertCache(_cfg(8, 2, 3), 2, [[0, 1, 2], [3, 4, -1]])
    before = [c.state(l) for l in range(2)]
    for args in ((2, 0, [5], 1), (0, -1, [5], 1), (0, 0, [8], 1), (0, 0, [-1], 1), (0, 0, [5], -1)):
        with pytest.raises(spice.SpiceError):
            c.prefetch(*args)
    after = [c.state(l) for l in range(2)]
    for (s0, l0), (s1, l1) in zip(before, after):
        assert s0.tolist() == s1.tolist() and l0.tolist() == l1.tolist()
    assert c.prefetch(1, 0, [], 3) == ([], [])
    assert c.prefetch(1, 0, [5, 6], 0) == ([], [])
    assert c.prefetch(1, 0, [5, 6, 7], 2) == ([5, 6], [-1, 3])
    c.close()
