"""Layer shapes and workload settings of the MoE layers this library is measured on.

Shapes follow the two models the paper evaluates (Sec. 5.1): a DeepSeek-V2-Lite
MoE layer and a Qwen2-57B-A14B MoE layer, plus a tiny fp32 layer for parity.
Nothing here computes any part of the method; it only names sizes.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Optional, Tuple

DTYPE_F32 = 0
DTYPE_BF16 = 1
WFMT_MXFP4 = 2  # routed experts' weights as OCP MXFP4 (E2M1 elements, E8M0 scale per 32)

CONF_INPUT = 0
CONF_GATE = 1
CONF_GATE_RENORM = 2


@dataclass(frozen=True)
class MoEShape:
    """One MoE layer: hidden size d, N routed experts (top-K), routed SwiGLU
    intermediate I, shared-block intermediate I_s (all shared experts of the
    layer concatenated), LoRE rank r (Eq. 9)."""

    d: int
    n_experts: int
    top_k: int
    inter: int
    shared_inter: int
    lore_rank: int
    dtype: int  # DTYPE_F32 or DTYPE_BF16 for activations and weights

    @property
    def wbytes(self) -> int:
        return 4 if self.dtype == DTYPE_F32 else 2

    @property
    def expert_bytes(self) -> int:
        """HBM bytes of one routed expert (gate+up [2I][d] and down [d][I])."""
        return 3 * self.inter * self.d * self.wbytes

    @property
    def shared_bytes(self) -> int:
        return 3 * self.shared_inter * self.d * self.wbytes

    @property
    def lore_bytes(self) -> int:
        """Bytes of one expert's LoRE factors A [r][d] and B [d][r]."""
        return 2 * self.lore_rank * self.d * self.wbytes


@dataclass(frozen=True)
class Workload:
    """A seeded synthetic workload: one layer shape plus token count T,
    residency, routing skew and the confidence rule."""

    name: str
    shape: MoEShape
    tokens: int
    resident: int  # R experts resident in the GPU cache
    skew: bool  # logit bias b_e = ln p_e from the Zipf popularity
    tau: float = 0.5
    conf_mode: int = CONF_INPUT
    norm_topk: int = 0
    shared_gate: bool = False  # sigmoid output gate on the shared block (Qwen2-style shared expert)
    wfmt: int = 0  # routed experts' weight format: 0 = the shape's dtype, WFMT_MXFP4
    zipf_s: float = 1.1
    seed: int = 0
    layers: int = 1
    cache_slots: Optional[int] = None  # LRU-managed cache (stack workload)
    steps: int = 1

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


TINY = MoEShape(d=256, n_experts=8, top_k=2, inter=128, shared_inter=256, lore_rank=8, dtype=DTYPE_F32)
# DeepSeek-V2-Lite: two shared experts of intermediate 1408 form one SwiGLU block of 2816.
DSV2 = MoEShape(d=2048, n_experts=64, top_k=6, inter=1408, shared_inter=2816, lore_rank=32, dtype=DTYPE_BF16)
QWEN2 = MoEShape(d=3584, n_experts=64, top_k=8, inter=2560, shared_inter=20480, lore_rank=64, dtype=DTYPE_BF16)

WORKLOADS = {
    "tiny_f32": Workload("tiny_f32", TINY, tokens=4, resident=4, skew=False),
    "dsv2_decode_t1": Workload("dsv2_decode_t1", DSV2, tokens=1, resident=32, skew=False),
    "dsv2_decode_t8": Workload("dsv2_decode_t8", DSV2, tokens=8, resident=32, skew=False),
    "dsv2_decode_t32": Workload("dsv2_decode_t32", DSV2, tokens=32, resident=32, skew=False),
    # the same layer with MXFP4 routed experts (quantised expert weights)
    "dsv2_decode_mxfp4_t32": Workload("dsv2_decode_mxfp4_t32", DSV2, tokens=32, resident=32, skew=False,
                                      wfmt=WFMT_MXFP4),
    "qwen2_decode_r16": Workload("qwen2_decode_r16", QWEN2, tokens=16, resident=16, skew=True),
    "qwen2_decode_r32": Workload("qwen2_decode_r32", QWEN2, tokens=16, resident=32, skew=True),
    "qwen2_decode_r48": Workload("qwen2_decode_r48", QWEN2, tokens=16, resident=48, skew=True),
    "dsv2_stack": Workload("dsv2_stack", DSV2, tokens=64, resident=24, skew=False, layers=26,
                           cache_slots=24, steps=128),
    "qwen2_prefill": Workload("qwen2_prefill", QWEN2, tokens=4096, resident=64, skew=True),
    # the same layers with the shared block's sigmoid output gate of the released model
    "qwen2_gated_decode_r32": Workload("qwen2_gated_decode_r32", QWEN2, tokens=16, resident=32, skew=True,
                                       shared_gate=True),
}


def small_shape(d: int = 192, n_experts: int = 16, top_k: int = 4, inter: int = 96,
                shared_inter: int = 160, lore_rank: int = 8, dtype: int = DTYPE_BF16) -> MoEShape:
    """A reduced shape for parity at sizes the oracle finishes quickly while
    still spanning several tiles with ragged tails."""
    return MoEShape(d, n_experts, top_k, inter, shared_inter, lore_rank, dtype)
