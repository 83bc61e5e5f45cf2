"""GPU parity of the prefill path: at T >= 256 tokens (bf16, tile-aligned sizes) the
HIT experts and the shared block run as grouped MFMA GEMMs.

  - a reduced layer (d=256, N=16, K=4, I=256, I_s=384, r=16) at T=300 and 600, every
    token against the oracle, all resident and partly resident (LoRE + exact misses),
    token tiles with ragged tails;
  - the prefill routing with ragged tiles (fp32 and bf16; partial expert, contraction and
    token tiles), every token;
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


# prefill routing with ragged tiles everywhere: 12 experts (a partial 16-expert MFMA tile),
# d = 196 fp32 (a partial contraction pass), T = 301 (a partial 16-token block), top-3
PF_RAGGED_F32 = W.MoEShape(d=196, n_experts=12, top_k=3, inter=92, shared_inter=100, lore_rank=12,
                           dtype=W.DTYPE_F32)
PF_RAGGED_BF16 = W.MoEShape(d=200, n_experts=20, top_k=5, inter=104, shared_inter=168, lore_rank=24,
                            dtype=W.DTYPE_BF16)


@pytest.mark.parametrize("shape,T,R", [(PF_RAGGED_F32, 301, 5), (PF_RAGGED_BF16, 517, 9)],
                         ids=["f32_T301", "bf16_T517"])
def test_prefill_routing_ragged_every_token(shape, T, R):
    say(f"prefill ragged d={shape.d} N={shape.n_experts} K={shape.top_k} T={T} R={R}")
    wl = W.Workload("prefill_ragged", shape, tokens=T, resident=R, skew=True)
    c = Case(wl)
    c.run_gpu()
    c.run_oracle()
    c.check_routing()
    c.check_outputs()
    assert (np.bincount(c.o["cls"].reshape(-1), minlength=3) > 0).all()


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
