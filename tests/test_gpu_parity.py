"""GPU parity: the HIP path through the C ABI against the oracle, element by element.

Covers the tiny fp32 layer, reduced bf16/fp32 layers with ragged tails (several
tiles, partial contraction steps, partial row tiles, >32 tokens), the
DeepSeek-V2-Lite-shaped decode batches (T = 1, 8, 32), the Qwen2-57B-A14B-shaped
decode batch at three residencies (outputs sampled per token), and the
degenerate cases of the method.
"""
import numpy as np
import pytest
import torch

from paper_2608_21240_amd import layer as LY, synth, workloads as W
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


RAGGED_BF16 = W.MoEShape(d=200, n_experts=16, top_k=4, inter=104, shared_inter=168, lore_rank=24,
                         dtype=W.DTYPE_BF16)
RAGGED_F32 = W.MoEShape(d=196, n_experts=12, top_k=3, inter=92, shared_inter=100, lore_rank=12, dtype=W.DTYPE_F32)


def small_wl(shape, T, resident, **kw):
    return W.Workload("small", shape, tokens=T, resident=resident, skew=kw.pop("skew", False), **kw)


def check_combine_in_layer_call(c):
    """The same layer call again with the combine inside moe_layer_gpu (out given, the first
    call's host residual as resid): the output equals the first call's (routing and FFN in
    the layer call, then the separate combine) bit for bit."""
    R, s, T = c.run, c.shape, c.T
    xd = LY.to_tensor(c.x, s.dtype, "cuda")
    conf = torch.from_numpy(np.ascontiguousarray(c.conf)).cuda()
    out1 = R.out[:T].clone()
    R.out.zero_()
    R.layer_gpu(c.dev, xd, conf, T, to_host=False, resid=R.resid, out=True)
    torch.cuda.synchronize()
    assert R.flags() == 0
    assert torch.equal(R.out[:T], out1), "the layer call's combine differs from the separate combine"


@pytest.mark.parametrize("fused", [True, False])
def test_tiny_f32_layer(fused):
    say(f"tiny_f32 fused={fused}")
    c = Case(W.WORKLOADS["tiny_f32"])
    c.run_gpu(fused=fused)
    c.run_oracle()
    c.check_routing()
    c.check_outputs()


@pytest.mark.parametrize("layer_call", [True, False])
@pytest.mark.parametrize("shape,T,R", [(RAGGED_BF16, 37, 6), (RAGGED_BF16, 5, 9), (RAGGED_F32, 41, 4),
                                       (W.small_shape(), 70, 5)])
def test_ragged_layers(shape, T, R, layer_call):
    say(f"ragged d={shape.d} N={shape.n_experts} K={shape.top_k} I={shape.inter} Is={shape.shared_inter} "
        f"r={shape.lore_rank} T={T} R={R} layer_call={layer_call}")
    c = Case(small_wl(shape, T, R))
    c.run_gpu(layer_call=layer_call)
    c.run_oracle()
    c.check_routing()
    c.check_outputs()
    counts = np.bincount(c.o["cls"].reshape(-1), minlength=3)
    assert (counts > 0).all(), counts  # all three classes exercised
    if layer_call:
        check_combine_in_layer_call(c)


# A shape the prefill GEMMs never take (d not a multiple of 256), and one they take from
# 256 tokens on.
LIMIT_STREAM = W.MoEShape(d=264, n_experts=16, top_k=8, inter=136, shared_inter=200, lore_rank=8,
                          dtype=W.DTYPE_BF16)
LIMIT_GEMM = W.MoEShape(d=256, n_experts=16, top_k=4, inter=256, shared_inter=384, lore_rank=16,
                        dtype=W.DTYPE_BF16)


@pytest.mark.parametrize("shape,T,R", [
    (LIMIT_STREAM, 128, 6),   # T*K = 1024: the largest call of the three fused launches
    (LIMIT_STREAM, 129, 6),   # 1032 slots: separate routing (decode kernel) and FFN launches
    (LIMIT_GEMM, 255, 7),     # 1020 slots, below the GEMMs' 256 tokens: fused launches
    (LIMIT_GEMM, 256, 7),     # 1024 slots, but the GEMMs apply: decode routing, then the GEMMs
    (LIMIT_GEMM, 257, 7),     # past the decode routing's 256 tokens: prefill routing and GEMMs
], ids=["stream-1024", "stream-1032", "gemm-T255", "gemm-T256", "gemm-T257"])
def test_layer_call_at_its_dispatch_limits(shape, T, R):
    """moe_layer_gpu on either side of each limit that picks its launches (slots of the fused
    launches, tokens of the decode routing, tokens of the prefill GEMMs): every token's
    routing and outputs against the oracle."""
    say(f"layer-call limits d={shape.d} K={shape.top_k} T={T} R={R}")
    c = Case(small_wl(shape, T, R))
    c.run_gpu(layer_call=True)
    c.run_oracle()
    c.check_routing()
    c.check_outputs()
    assert (np.bincount(c.o["cls"].reshape(-1), minlength=3) > 0).all()  # all three classes
    check_combine_in_layer_call(c)


@pytest.fixture(scope="module")
def dsv2():
    wl = W.WORKLOADS["dsv2_decode_t32"]
    host = LY.HostLayer(wl, 0)
    dev = LY.DeviceLayer(host)
    return wl, host, dev


@pytest.mark.parametrize("layer_call", [True, False])
@pytest.mark.parametrize("T", [1, 8, 32])
def test_dsv2_decode(dsv2, T, layer_call):
    wl, host, dev = dsv2
    say(f"dsv2 decode T={T} layer_call={layer_call}")
    c = Case(wl.with_(tokens=T), host=host)
    c.run_gpu(dev=dev, layer_call=layer_call)
    c.run_oracle()
    c.check_routing()
    c.check_outputs()
    if layer_call:
        check_combine_in_layer_call(c)


@pytest.fixture(scope="module")
def qwen2():
    wl = W.WORKLOADS["qwen2_decode_r32"]
    return wl, LY.HostLayer(wl, 0)


@pytest.mark.parametrize("R", [16, 32, 48])
def test_qwen2_decode_sampled(qwen2, R):
    wl, host = qwen2
    say(f"qwen2 decode T=16 R={R}")
    wlr = wl.with_(resident=R)
    host.resident = synth.resident_experts(wlr, 0)
    c = Case(wlr, host=host)
    c.run_gpu()
    c.run_oracle(tokens=[0, 5, 11, 15])
    c.check_routing()
    c.check_outputs()
    del c.dev
    torch.cuda.empty_cache()


def test_zero_input_ties_pick_lowest_ids():
    shape = W.small_shape()
    wl = small_wl(shape, 6, 5)
    x = synth.to_storage(np.zeros((6, shape.d), np.float32), shape.dtype)
    c = Case(wl, x=x)
    c.run_gpu()
    c.run_oracle()
    assert (c.g["idx"] == np.arange(shape.top_k)).all()
    assert (c.g["w"] == np.float32(1.0 / shape.n_experts)).all()
    c.check_routing()
    c.check_outputs()


@pytest.mark.parametrize("mode", ["all_resident", "all_lore", "all_exact", "none_resident"])
def test_residency_extremes(mode):
    shape = RAGGED_BF16
    T = 19
    R = shape.n_experts if mode == "all_resident" else 0
    conf = {"all_lore": 0.0, "all_exact": 1.0}.get(mode)
    wl = small_wl(shape, T, R)
    cf = None if conf is None else np.full((T, shape.top_k), conf, np.float32)
    c = Case(wl, conf=cf, resident=list(range(R)), n_slots=max(R, 1))
    c.run_gpu()
    c.run_oracle()
    c.check_routing()
    c.check_outputs()
    if mode == "all_resident":
        assert (c.g["cls"] == HIT).all()
    if mode == "all_lore":
        assert (c.g["cls"] == LORE).all()
    if mode == "all_exact":
        assert (c.g["cls"] == EXACT).all()
    check_combine_in_layer_call(c)


@pytest.mark.parametrize("conf_mode,norm,tau", [(W.CONF_GATE, 0, 0.1), (W.CONF_GATE_RENORM, 0, 0.3),
                                                (W.CONF_INPUT, 1, 0.5), (W.CONF_GATE, 1, 0.3)])
def test_confidence_modes_and_renormalised_gates(conf_mode, norm, tau):
    shape = RAGGED_BF16
    wl = small_wl(shape, 23, 5, conf_mode=conf_mode, norm_topk=norm, tau=tau)
    c = Case(wl)
    c.run_gpu()
    c.run_oracle()
    # a gate-derived confidence within rounding of tau could legitimately flip
    if conf_mode != W.CONF_INPUT:
        assert np.all(np.abs(c.o["conf"] - tau) > 1e-6)
    c.check_routing()
    c.check_outputs()


def test_nan_confidence_is_exact():
    shape = RAGGED_BF16
    T = 9
    conf = synth.gen_conf(small_wl(shape, T, 0), 0, 0, T)
    conf[::2, 1] = np.nan
    c = Case(small_wl(shape, T, 3), conf=conf)
    c.run_gpu()
    c.run_oracle()
    c.check_routing()
    miss = c.o["cls"][::2, 1] != HIT
    assert (c.g["cls"][::2, 1][miss] == EXACT).all()


def test_workspace_reuse_across_token_counts():
    """Counters in the workspace reset themselves: calls with different T on one
    workspace give the same results as fresh workspaces."""
    shape = RAGGED_BF16
    wl = small_wl(shape, 40, 6)
    host = LY.HostLayer(wl, 0)
    dev = LY.DeviceLayer(host)
    run = LY.LayerRun(shape, 40, dev.C, keep_logits=True)
    outs = {}
    for T in (40, 3, 17, 40):
        c = Case(wl.with_(tokens=T), host=host)
        g = c.run_gpu(dev=dev, run=run)
        fresh = Case(wl.with_(tokens=T), host=host).run_gpu(dev=dev)
        for k in ("idx", "cls", "perm", "offsets", "out"):
            assert np.array_equal(g[k], fresh[k]), (T, k)
        outs.setdefault(T, []).append(g["out"])
    assert np.array_equal(outs[40][0], outs[40][1])


def test_bad_resident_slot_is_flagged_not_faulted():
    shape = RAGGED_BF16
    wl = small_wl(shape, 8, 4)
    host = LY.HostLayer(wl, 0)
    dev = LY.DeviceLayer(host)
    e = host.resident[0]
    slot = dev.resident_slot.clone()
    dev.resident_slot[e] = dev.C + 5  # outside the pool
    run = LY.LayerRun(shape, 8, dev.C)
    x = LY.to_tensor(synth.gen_x(wl, 0, 0, 8), shape.dtype, "cuda")
    conf = torch.from_numpy(synth.gen_conf(wl, 0, 0, 8)).cuda()
    run.forward(dev, x, conf, exact=False)
    torch.cuda.synchronize()
    flags = run.flags(clear=True)
    hit_e = (run.topk_idx == e).any().item()
    if hit_e:
        assert flags & 1
        assert not ((run.topk_idx == e) & (run.slot_class == HIT)).any().item()
    assert run.flags() == 0
    dev.resident_slot.copy_(slot)


def test_repeat_runs_are_bit_identical():
    wl = W.WORKLOADS["tiny_f32"].with_(tokens=13)
    c1 = Case(wl)
    g1 = c1.run_gpu()
    g2 = Case(wl, host=c1.host).run_gpu(dev=c1.dev)
    for k in g1:
        if k != "flags":
            assert np.array_equal(g1[k], g2[k]), k


@pytest.mark.parametrize("layer_call", [True, False])
@pytest.mark.parametrize("shape,T,R", [(RAGGED_BF16, 37, 6), (RAGGED_F32, 41, 4)])
def test_host_copies_match_device_outputs(shape, T, R, layer_call):
    """The bucketing block's pinned-host copies equal the device outputs and the input x;
    the class counts equal the histogram of the classes."""
    say(f"host copies d={shape.d} T={T} layer_call={layer_call}")
    c = Case(small_wl(shape, T, R))
    c.run_gpu(layer_call=layer_call)
    run = c.run
    assert np.array_equal(run.idx_host[:T].numpy(), c.g["idx"])
    assert np.array_equal(run.w_host[:T].numpy(), c.g["w"])
    assert np.array_equal(run.cls_host[:T].numpy(), c.g["cls"])
    assert run.counts_host.tolist() == np.bincount(c.g["cls"].reshape(-1), minlength=3).tolist()
    from parity import to_np
    assert np.array_equal(to_np(run.x_host[:T]), c.x)


# Decode routing of more slots than its bucketing block keeps in LDS (T*K = 2560 > 1024
# at T = 256, the largest decode batch): that block reads the keys the top-K blocks
# published twice, once per pass.
MANY_SLOTS = W.MoEShape(d=200, n_experts=20, top_k=10, inter=104, shared_inter=168, lore_rank=24,
                        dtype=W.DTYPE_BF16)


def test_decode_routing_more_slots_than_the_key_cache():
    T, R = 256, 8
    say(f"decode routing d={MANY_SLOTS.d} N={MANY_SLOTS.n_experts} K={MANY_SLOTS.top_k} T={T} R={R}")
    c = Case(small_wl(MANY_SLOTS, T, R))
    c.run_gpu(layer_call=False)
    c.run_oracle()
    c.check_routing()
    c.check_outputs()
    run = c.run
    assert np.array_equal(run.idx_host[:T].numpy(), c.g["idx"])
    assert np.array_equal(run.w_host[:T].numpy(), c.g["w"])
    assert np.array_equal(run.cls_host[:T].numpy(), c.g["cls"])
    assert run.counts_host.tolist() == np.bincount(c.g["cls"].reshape(-1), minlength=3).tolist()
    assert (np.bincount(c.g["cls"].reshape(-1), minlength=3) > 0).all()


FORCE_FETCH = dict(cpu_bytes_per_s=1e8, cpu_flops_per_s=1e12, pcie_bytes_per_s=1e13, gpu_fixed_s=0.0, margin=0.0)


@pytest.mark.parametrize("shape,T,R,slots", [(W.small_shape(), 24, 5, 3), (RAGGED_BF16, 37, 6, 4),
                                             (RAGGED_F32, 41, 4, 2)])
def test_exact_split_fetched_experts_on_gpu(shape, T, R, slots):
    """Eq. 12's M_fetch: the planner moves some exact misses to the GPU (a cost model that
    makes fetching pay); outputs still match the oracle, whose result does not depend on
    where an exact miss runs."""
    from paper_2608_21240_amd import spice
    say(f"exact split d={shape.d} T={T} R={R} fetch slots={slots}")
    c = Case(small_wl(shape, T, R))
    cost = spice.spice_split_cost_t(**FORCE_FETCH)
    c.run_gpu(split=cost, fetch_slots=slots)
    c.run_oracle()
    fetched = c.run.last_fetch
    assert 0 < len(fetched) <= slots
    o, g = c.o, c.g
    exact_e = set(o["idx"][o["cls"] == EXACT].tolist())
    assert set(fetched) <= exact_e
    on_gpu = np.isin(o["idx"], fetched) & (o["cls"] == EXACT)
    # fetched slots are relabelled on the device and on the host, the rest is the oracle's routing
    assert (g["cls"][on_gpu] == spice.SPICE_CLASS_EXACT_GPU).all()
    assert np.array_equal(g["cls"][~on_gpu], o["cls"][~on_gpu])
    assert np.array_equal(c.run.cls_host[:T].numpy(), g["cls"])
    assert np.array_equal(g["idx"], o["idx"]) and np.array_equal(g["perm"], o["perm"])
    # the layer output covers every exact miss, wherever it ran; fetched slots' expert
    # outputs are the oracle's expert outputs
    from parity import as_f64, rel_err, tol_for
    errs_out = rel_err(as_f64(g["out"], shape.dtype)[o["tokens"]], o["out"])
    assert errs_out.max() <= tol_for(shape), errs_out.max()
    ys = np.array([g["y_slots"][g["inv_perm"][t * shape.top_k + k]] for t, k in np.argwhere(on_gpu)])
    refs = np.array([o["y_slot"][t, k] for t, k in np.argwhere(on_gpu)])
    assert rel_err(ys, refs).max() <= tol_for(shape)
    assert c.run.flags() == 0
