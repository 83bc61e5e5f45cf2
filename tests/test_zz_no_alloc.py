"""The no-allocation layer call (moe_layer_gpu_noalloc, workspace in a static device array)
against the layer call with a caller's workspace (moe_layer_gpu): the same outputs, on two
calls in a row, the second with fewer tokens, on a DeepSeek-V2-Lite-shaped layer and a
ragged fp32 layer."""
import numpy as np
import pytest
import torch

from paper_2608_21240_amd import layer as LY, spice, synth, workloads as W
from parity import say, to_np, tol_for, rel_err, as_f64

pytestmark = pytest.mark.gpu

RAGGED_F32 = W.MoEShape(d=196, n_experts=12, top_k=3, inter=92, shared_inter=100, lore_rank=12, dtype=W.DTYPE_F32)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    spice.lib()
    yield
    torch.cuda.synchronize()


def _outputs(run, T):
    K = run.shape.top_k
    return dict(idx=to_np(run.topk_idx[:T]), w=to_np(run.topk_w[:T]), cls=to_np(run.slot_class[:T]),
                offsets=to_np(run.offsets), perm=to_np(run.perm[: T * K]), inv_perm=to_np(run.inv_perm[: T * K]),
                y_slots=to_np(run.y_slots[: T * K]), y_shared=to_np(run.y_shared[:T]), out=to_np(run.out[:T]))


@pytest.mark.parametrize("wl,Ts", [(W.WORKLOADS["dsv2_decode_t32"], (32, 8)),
                                   (W.Workload("ragged_f32", RAGGED_F32, tokens=41, resident=4, skew=False), (41, 6))])
def test_noalloc_layer_call_matches_workspace_call(wl, Ts):
    s = wl.shape
    host = LY.HostLayer(wl, 0)
    dev = LY.DeviceLayer(host, host_exact=False)
    ref_run = LY.LayerRun(s, max(Ts), dev.C, tau=wl.tau)
    na_run = LY.LayerRun(s, max(Ts), dev.C, tau=wl.tau)
    for call, T in enumerate(Ts):
        say(f"noalloc {wl.name} call {call} T={T}")
        x = LY.to_tensor(synth.gen_x(wl, 0, call, T), s.dtype, "cuda")
        conf = torch.from_numpy(synth.gen_conf(wl, 0, call, T)).cuda()
        for r in (ref_run, na_run):
            r.y_slots.zero_(); r.y_shared.zero_(); r.out.zero_()
        ref_run.layer_gpu(dev, x, conf, T, to_host=False, resid=None, out=True)
        spice.moe_layer_gpu_noalloc(na_run.cfg, T, x, dev.wg, dev.bias, dev.resident_slot, conf, dev.w13_pool,
                                    dev.w2_pool, dev.w13s, dev.w2s, dev.w_sg, dev.lore_A, dev.lore_B, None,
                                    na_run.topk_idx, na_run.topk_w, na_run.slot_class, na_run.offsets, na_run.perm,
                                    na_run.inv_perm, na_run.y_slots, na_run.y_shared, None, None, na_run.out)
        torch.cuda.synchronize()
        a, b = _outputs(ref_run, T), _outputs(na_run, T)
        for k in ("idx", "cls", "offsets", "perm", "inv_perm"):
            assert np.array_equal(a[k], b[k]), k
        assert np.allclose(a["w"], b["w"], rtol=2e-7, atol=0)
        tol = tol_for(s)
        rows = a["inv_perm"][a["cls"].reshape(-1) <= 1]
        assert rel_err(b["y_slots"][rows], a["y_slots"][rows]).max() <= tol
        assert rel_err(b["y_shared"], a["y_shared"]).max() <= tol
        assert rel_err(as_f64(b["out"], s.dtype), as_f64(a["out"], s.dtype)).max() <= tol
        assert ref_run.flags() == 0


def test_noalloc_rejects_calls_beyond_its_scratch():
    c = spice.make_cfg(W.QWEN2, n_slots=48)
    T = 4096
    assert spice.spice_workspace_bytes(c, T) > spice.SPICE_NOALLOC_SCRATCH_BYTES
    with pytest.raises(spice.SpiceError) as ei:
        spice.moe_layer_gpu_noalloc(c, T, *([0x1000] * 21), None, None, 0x1000)
    assert ei.value.status == spice.SPICE_ERR_UNSUPPORTED
