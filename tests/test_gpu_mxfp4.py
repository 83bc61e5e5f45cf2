"""GPU parity with MXFP4 routed experts (OCP MX: E2M1 codes, one E8M0 scale per 32): the
grouped FFN decodes the pool's blobs with the gfx950 scaled conversion, the host path
decodes the host blobs, and both are checked against the oracle's layer on the same
blobs.  Shapes: reduced layers whose rows end in a partial group of MX blocks (K/32 not a
multiple of 4), a 300-token call (many tokens per expert), and the DeepSeek-V2-Lite-shaped
decode batches, each through the fused decode layer call and through the separate
routing and FFN calls."""
import numpy as np
import pytest
import torch

from paper_2608_21240_amd import layer as LY, workloads as W
from parity import EXACT, HIT, LORE, Case, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_21240_amd import spice
    spice.lib()
    yield
    torch.cuda.synchronize()


MX_A = W.MoEShape(d=192, n_experts=16, top_k=4, inter=96, shared_inter=160, lore_rank=8, dtype=W.DTYPE_BF16)
MX_B = W.MoEShape(d=320, n_experts=12, top_k=3, inter=160, shared_inter=96, lore_rank=16, dtype=W.DTYPE_BF16)


def mx(shape, T, R, **kw):
    return W.Workload("mxfp4", shape, tokens=T, resident=R, skew=kw.pop("skew", False), wfmt=W.WFMT_MXFP4, **kw)


@pytest.mark.parametrize("layer_call", [True, False])
@pytest.mark.parametrize("shape,T,R,fused", [(MX_A, 37, 6, True), (MX_A, 5, 9, False), (MX_B, 23, 5, True),
                                             (MX_B, 300, 8, True)])
def test_mxfp4_layers(shape, T, R, fused, layer_call):
    """layer_call: the fused decode layer call (moe_layer_gpu; at T = 300 it takes the
    separate launches), else the separate routing and FFN calls."""
    say(f"mxfp4 d={shape.d} I={shape.inter} T={T} R={R} fused={fused} layer_call={layer_call}")
    c = Case(mx(shape, T, R))
    c.run_gpu(fused=fused, layer_call=layer_call)
    c.run_oracle()
    c.check_routing()
    c.check_outputs()
    counts = np.bincount(c.o["cls"].reshape(-1), minlength=3)
    assert (counts > 0).all(), counts


# the widest contractions MXFP4 takes (SPICE_MXFP4_MAX_K): 128 scales per row in the up
# pass (d = 4096) and in the down pass (inter = 4096)
MX_WIDE_D = W.MoEShape(d=4096, n_experts=8, top_k=2, inter=1024, shared_inter=256, lore_rank=16, dtype=W.DTYPE_BF16)
MX_WIDE_I = W.MoEShape(d=1024, n_experts=8, top_k=2, inter=4096, shared_inter=256, lore_rank=16, dtype=W.DTYPE_BF16)


@pytest.mark.parametrize("shape", [MX_WIDE_D, MX_WIDE_I], ids=["d4096", "inter4096"])
def test_mxfp4_widest_rows(shape):
    say(f"mxfp4 d={shape.d} I={shape.inter} T=20")
    c = Case(mx(shape, 20, 4))
    c.run_gpu()
    c.run_oracle(tokens=[0, 7, 19])
    c.check_routing()
    c.check_outputs()


def test_mxfp4_gated_shared_block():
    c = Case(mx(MX_B, 19, 6, shared_gate=True))
    c.run_gpu()
    c.run_oracle()
    c.check_routing()
    c.check_outputs()


@pytest.fixture(scope="module")
def dsv2_mx():
    wl = W.WORKLOADS["dsv2_decode_mxfp4_t32"]
    say("dsv2 mxfp4: quantising the experts")
    host = LY.HostLayer(wl, 0)
    dev = LY.DeviceLayer(host)
    return wl, host, dev


@pytest.mark.parametrize("layer_call", [True, False])
@pytest.mark.parametrize("T,tokens", [(1, None), (8, [0, 3, 7]), (32, [0, 9, 20, 31])])
def test_dsv2_mxfp4_decode(dsv2_mx, T, tokens, layer_call):
    wl, host, dev = dsv2_mx
    say(f"dsv2 mxfp4 decode T={T} layer_call={layer_call}")
    c = Case(wl.with_(tokens=T), host=host)
    c.run_gpu(dev=dev, layer_call=layer_call)
    c.run_oracle(tokens=tokens)
    c.check_routing()
    c.check_outputs()
