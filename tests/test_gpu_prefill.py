"""GPU parity of the prefill path: at T >= 256 tokens (bf16, tile-aligned sizes) the
HIT experts and the shared block run as grouped MFMA GEMMs.

  - a reduced layer (d=256, N=16, K=4, I=256, I_s=384, r=16) at T=300 and 600, every
    token against the oracle, all resident and partly resident (LoRE + exact misses),
    token tiles with ragged tails;
  - the Qwen2-57B-A14B-shaped prefill layer (T=4096, top-8, Zipf(1.1) routing skew),
    all 64 experts resident and half of them absent, routing of every token and the
    outputs of sampled tokens.
"""
import numpy as np
import pytest
import torch

from paper_2608_21240_amd import layer as LY, synth, workloads as W
from parity import EXACT, HIT, LORE, Case, say

pytestmark = pytest.mark.gpu

PF_SMALL = W.MoEShape(d=256, n_experts=16, top_k=4, inter=256, shared_inter=384, lore_rank=16, dtype=W.DTYPE_BF16)


@pytest.mark.parametrize("T,R", [(300, 16), (300, 8), (600, 5)])
def test_prefill_small_every_token(T, R):
    say(f"prefill small T={T} R={R}")
    wl = W.Workload("prefill_small", PF_SMALL, tokens=T, resident=R, skew=True)
    c = Case(wl)
    c.run_gpu()
    c.run_oracle()
    c.check_routing()
    c.check_outputs()
    counts = np.bincount(c.o["cls"].reshape(-1), minlength=3)
    if R < PF_SMALL.n_experts:
        assert (counts > 0).all(), counts
    else:
        assert counts[HIT] == T * PF_SMALL.top_k


@pytest.fixture(scope="module")
def qwen_prefill():
    wl = W.WORKLOADS["qwen2_prefill"]
    say("qwen2 prefill: drawing weights")
    host = LY.HostLayer(wl, 0)
    host.prefetch(range(wl.shape.n_experts), range(wl.shape.n_experts))
    return wl, host


@pytest.mark.parametrize("R", [64, 32])
def test_qwen2_prefill_sampled(qwen_prefill, R):
    wl, host = qwen_prefill
    say(f"qwen2 prefill T={wl.tokens} R={R}")
    wlr = wl.with_(resident=R)
    host.resident = synth.resident_experts(wlr, 0)
    c = Case(wlr, host=host)
    c.run_gpu()
    c.run_oracle(tokens=[0, 1, 777, 2048, 3001, 4095])
    c.check_routing()
    c.check_outputs()
    counts = np.bincount(c.o["cls"].reshape(-1), minlength=3)
    say(f"  classes {counts.tolist()}")
    if R == 64:
        assert counts[HIT] == wl.tokens * wl.shape.top_k
    else:
        assert counts[LORE] > 0 and counts[EXACT] > 0
    del c.dev
    torch.cuda.empty_cache()
