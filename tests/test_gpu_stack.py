"""The stack workload on the GPU: 26 independent DSV2-Lite-shaped layers, T=64
decode tokens per step, 128 steps, a 24-slot LRU cache per layer kept by the
library (moe_cache_*).

Checked against the oracle at every (step, layer):
  - slot classes computed on the GPU from the library-maintained resident_slot
    equal the oracle's classes from its own LRU state (the same top-K indices);
  - admitted and evicted experts equal the oracle LRU step's.
At sampled (step, layer) pairs: the full oracle routing and the layer output of
sampled tokens (this reads admitted experts out of the pool slots the library
copied them into).  At the end: every pool slot holds the expert the cache
state names, byte for byte.
"""
import numpy as np
import pytest
import torch

from parity import HIT, LORE, EXACT, as_f64, rel_err, tol_for, to_np
from paper_2608_21240_amd import synth
from paper_2608_21240_amd.layer import to_tensor
from paper_2608_21240_amd.stack import StackModel, StackRun
from paper_2608_21240_amd.workloads import WORKLOADS

pytestmark = pytest.mark.gpu


def test_stack_lru_matches_oracle(orc):
    wl = WORKLOADS["dsv2_stack"]
    s = wl.shape
    L, T, N, C, K = wl.layers, wl.tokens, s.n_experts, wl.cache_slots, s.top_k
    print(f"[stack] building {L} layers (T={T}, C={C}, steps={wl.steps})", flush=True)
    m = StackModel(wl)
    sr = StackRun(m, max_admit=4)
    refs = [orc.LRUState(N, C, m.initial[l]) for l in range(L)]
    ocfg = orc.make_cfg(s, tau=wl.tau)
    wg_np = [synth.gen_router(wl, l) for l in range(L)]
    samples = {0: [0, 13], 1: [25], 40: [7], 95: [19], wl.steps - 1: [0, 25]}
    tokens = [0, 31, 63]
    tables = None
    totals = np.zeros(3, np.int64)
    n_adm = 0
    for step in range(wl.steps):
        x_np = synth.gen_x(wl, 0, step, T)
        x = to_tensor(x_np, s.dtype, "cuda")
        conf_np = [synth.gen_conf(wl, l, step, T) for l in range(L)]
        confs = [torch.from_numpy(c).cuda() for c in conf_np]
        outs = {l: torch.empty((T, s.d), dtype=torch.bfloat16, device="cuda") for l in samples.get(step, [])}
        sr.step(step, x, confs, outputs=outs)
        torch.cuda.synchronize()
        for l in range(L):
            tr = sr.trace[step * L + l]
            assert tr["layer"] == l and tr["step"] == step
            mask = refs[l].resident_mask()
            ocls = orc.classify(ocfg, tr["idx"], mask, conf_np[l])
            assert np.array_equal(ocls, tr["cls"]), (step, l)
            if l in outs:
                if tables is None:
                    st = [m.host_storage(e) for e in range(N)]
                    la, lb = zip(*[m.base.lore(e) for e in range(N)])
                    tables = ([a for a, _ in st], [b for _, b in st], list(la), list(lb))
                o = orc.layer(ocfg, x_np, wg_np[l], None, mask, conf_np[l], tables[0], tables[1], m.base.w13s,
                              m.base.w2s, tables[2], tables[3], tokens=tokens)
                assert np.array_equal(o["idx"], tr["idx"]) and np.array_equal(o["cls"], tr["cls"]), (step, l)
                err = rel_err(as_f64(to_np(outs[l])[tokens], s.dtype), o["out"])
                print(f"[stack] step {step} layer {l}: out rel err max {err.max():.2e}", flush=True)
                assert err.max() <= tol_for(s), (step, l, err)
            a, e = refs[l].step(step, tr["idx"], tr["cls"], 4)
            assert tr["admitted"] == a.tolist() and tr["evicted"] == e.tolist(), (step, l)
            totals += np.bincount(tr["cls"].ravel(), minlength=3)
            n_adm += len(a)
        if step % 16 == 0:
            print(f"[stack] step {step}: classes so far {totals.tolist()}, admissions {n_adm}", flush=True)
    torch.cuda.synchronize()
    for l in range(L):
        se, lu = sr.cache.state(l)
        assert se.tolist() == refs[l].slot_expert.tolist() and lu.tolist() == refs[l].last_use.tolist(), l
    sr.close()
    # the pools hold what the cache says, byte for byte
    for l in (0, L // 2, L - 1):
        want = refs[l].slot_expert
        for slot in range(C):
            e = int(want[slot])
            w13, w2 = m.host_storage(e)
            assert np.array_equal(to_np(m.w13_pool[l][slot]), w13), (l, slot, e)
            assert np.array_equal(to_np(m.w2_pool[l][slot]), w2), (l, slot, e)
        dev = m.resident_slot[l].cpu().numpy()
        expect = np.full(N, -1, np.int32)
        expect[want] = np.arange(C, dtype=np.int32)
        assert np.array_equal(dev, expect), l
    hit_rate = totals[HIT] / totals.sum()
    print(f"[stack] slot hit rate {hit_rate:.3f}, LoRE share of misses "
          f"{totals[LORE] / max(totals[LORE] + totals[EXACT], 1):.3f}, admissions {n_adm}", flush=True)
    assert n_adm > 0 and 0.1 < hit_rate < 0.9


def test_stack_with_speculative_prefetch_matches_oracle(orc):
    """The same stack with speculative prefetching (Sec. 4.1): after each layer, the draft
    rollout's issue lists for the next two layers go into their caches (at most 3 per
    layer).  The oracle replays every demand admission and every prefetch batch on its own
    LRU state, and the classes of each call follow from that state.  The stack feeds the
    same x to every layer, so a depth-1 prediction is the next layer's routing itself:
    this checks the bookkeeping and measures the hit rate, not prediction quality."""
    wl = WORKLOADS["dsv2_stack"]
    s = wl.shape
    L, T, N, C = wl.layers, wl.tokens, s.n_experts, wl.cache_slots
    steps = 24
    pf = dict(depth=2, l_min=1, tau=0.0, max_prefetch=3)
    m = StackModel(wl)
    ocfg = orc.make_cfg(s, tau=wl.tau)
    rates = {}
    for use in (False, True):
        sr = StackRun(m, max_admit=4, prefetch=pf if use else None)  # loads the initial experts again
        refs = [orc.LRUState(N, C, m.initial[l]) for l in range(L)]
        totals = np.zeros(3, np.int64)
        n_pre = 0
        for step in range(steps):
            x = to_tensor(synth.gen_x(wl, 0, step, T), s.dtype, "cuda")
            conf_np = [synth.gen_conf(wl, l, step, T) for l in range(L)]
            sr.step(step, x, [torch.from_numpy(c).cuda() for c in conf_np])
            for l in range(L):
                tr = sr.trace[step * L + l]
                ocls = orc.classify(ocfg, tr["idx"], refs[l].resident_mask(), conf_np[l])
                assert np.array_equal(ocls, tr["cls"]), (use, step, l)
                a, e = refs[l].step(step, tr["idx"], tr["cls"], 4)
                assert tr["admitted"] == a.tolist() and tr["evicted"] == e.tolist(), (use, step, l)
                if use:
                    assert len(tr["queue"]) == min(pf["depth"], L - 1 - l)
                    for j, q in enumerate(tr["queue"]):
                        pa, pe = refs[l + 1 + j].prefetch(step, q, pf["max_prefetch"])
                        assert tr["prefetched"][j] == (pa.tolist(), pe.tolist()), (step, l, j)
                        n_pre += len(pa)
                totals += np.bincount(tr["cls"].ravel(), minlength=3)
        torch.cuda.synchronize()
        for l in range(L):
            se, lu = sr.cache.state(l)
            assert se.tolist() == refs[l].slot_expert.tolist() and lu.tolist() == refs[l].last_use.tolist(), l
        # the pools hold what the cache says
        for l in (1, L // 2, L - 1):
            for slot in range(C):
                e = int(refs[l].slot_expert[slot])
                w13, w2 = m.host_storage(e)
                assert np.array_equal(to_np(m.w13_pool[l][slot]), w13), (use, l, slot, e)
            assert sr.spec is None or sr.spec.flags() == 0
        sr.close()
        rates[use] = (totals[HIT] / totals.sum(), totals[EXACT] / totals.sum(), n_pre)
        print(f"[stack] prefetch={use}: slot hit rate {rates[use][0]:.3f}, exact share {rates[use][1]:.3f}, "
              f"prefetched experts {n_pre}", flush=True)
    assert rates[True][2] > 0 and rates[True][0] > rates[False][0]

