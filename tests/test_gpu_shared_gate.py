"""GPU parity of the gated shared block (the Qwen2-style shared expert, whose output is
scaled by sigmoid(w_sg . x)): moe_expert_ffn_grouped_gated against the oracle's gated
layer, element by element, on the decode kernels (ragged bf16 / fp32 shapes, fused and
separate LoRE) and the prefill GEMM path, and on sampled tokens of the
Qwen2-57B-A14B-shaped decode layer with its shared block gated.
"""
import numpy as np
import pytest
import torch

from paper_2608_21240_amd import layer as LY, synth, workloads as W
from parity import HIT, Case, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_21240_amd import spice
    spice.lib()
    yield
    torch.cuda.synchronize()


RAGGED_BF16 = W.MoEShape(d=200, n_experts=16, top_k=4, inter=104, shared_inter=168, lore_rank=24,
                         dtype=W.DTYPE_BF16)
RAGGED_F32 = W.MoEShape(d=196, n_experts=12, top_k=3, inter=92, shared_inter=100, lore_rank=12, dtype=W.DTYPE_F32)
PF_SMALL = W.MoEShape(d=256, n_experts=16, top_k=4, inter=256, shared_inter=384, lore_rank=16, dtype=W.DTYPE_BF16)


def gated(shape, T, R, skew=False):
    return W.Workload("gated", shape, tokens=T, resident=R, skew=skew, shared_gate=True)


@pytest.mark.parametrize("shape,T,R,fused", [(RAGGED_BF16, 37, 6, True), (RAGGED_BF16, 5, 9, False),
                                             (RAGGED_F32, 41, 4, True), (RAGGED_F32, 3, 4, False)])
def test_gated_ragged_layers(shape, T, R, fused):
    say(f"gated ragged d={shape.d} dtype={shape.dtype} T={T} R={R} fused={fused}")
    c = Case(gated(shape, T, R))
    assert c.host.w_sg is not None
    c.run_gpu(fused=fused)
    c.run_oracle()
    c.check_routing()
    c.check_outputs()
    # the gate is in effect: y_shared differs from the ungated shared block by a per-token factor in (0, 1)
    from oracle import make_cfg, shared_gate
    cfg = make_cfg(shape)
    gs = np.array([shared_gate(cfg, c.x[t], c.host.w_sg) for t in range(T)])
    assert ((gs > 0.05) & (gs < 0.95)).mean() > 0.5, gs


@pytest.mark.parametrize("T,R", [(300, 8), (300, 16)])
def test_gated_prefill_gemm_path(T, R):
    say(f"gated prefill small T={T} R={R}")
    c = Case(gated(PF_SMALL, T, R, skew=True))
    c.run_gpu()
    c.run_oracle()
    c.check_routing()
    c.check_outputs()
    counts = np.bincount(c.o["cls"].reshape(-1), minlength=3)
    if R == PF_SMALL.n_experts:
        assert counts[HIT] == T * PF_SMALL.top_k


def test_qwen2_gated_decode_sampled():
    wl = W.WORKLOADS["qwen2_gated_decode_r32"]
    say(f"qwen2 gated decode T={wl.tokens} R={wl.resident}")
    c = Case(wl)
    c.run_gpu()
    c.run_oracle(tokens=[0, 3, 9, 15])
    c.check_routing()
    c.check_outputs()
    del c.dev
    torch.cuda.empty_cache()
