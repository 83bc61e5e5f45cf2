"""MoE-layer decode benchmark: SPICE's per-layer forward under a partial expert cache.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

Workload: a DeepSeek-V2-Lite-shaped MoE layer (hidden 2048, 64 routed experts of
SwiGLU intermediate 1408, shared block 2816, top-6 softmax gating, LoRE rank 32),
bf16 weights/activations with fp32 accumulation, 32 experts resident (Zipf(1.1)
popularity), per-slot confidence U(0,1) with tau = 0.5; decode batch 32 is the
headline, batches 1 and 8 are reported alongside.  Weights and inputs are
seeded synthetic draws.

One step = one whole layer call on one batch: routing + bucketing, grouped FFN of
the resident hits + shared block + LoRE corrections on the GPU (moe_layer_gpu), the
exact-miss residual on the host CPU (overlapped with the GPU work), and the combine.
Steps rotate over several independent layer instances so that the weights
(about 0.6 GB per instance) stream from HBM and not from the 256 MB MALL.

Prints one JSON line.  ``value`` is the end-to-end rate of whole layer calls.
``roofline`` is for the layer's GPU path (one moe_layer_gpu call with the combine, the
host residual precomputed): the average duration of back-to-back calls, from HIP events on
the launch stream around the timed calls (the median of per-call event pairs and graph
replays alongside), against HBM; ``ffn_call`` is the
grouped-FFN call on its own.  ``cpu_baseline`` is the plain fp64 oracle on one host core,
``cpu_baseline_library`` the library's host path on every host core, each on a bounded
sample of the same workload.  ``qwen2`` holds the Qwen2-57B-A14B-shaped decode batch at
three residencies and the 4096-token prefill.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "MoE-layer decode tokens/s + achieved HBM GB/s (% peak), DSV2-Lite-shaped"

# HBM traffic per call of the layer's GPU path and of the grouped-FFN call at the headline batch, from
# two rocprofv3 --pmc passes over this script (FETCH_SIZE, then WRITE_SIZE; KiB per
# dispatch) scaled by what the counters read for a plain 1 GiB device copy
# (FETCH_SIZE x2.0, WRITE_SIZE x1.0).  One record per expert weight format; each is
# reported only while the kernel sources (the files hashed together) are the ones the
# counters were taken on.
TRAFFIC_RECORDS = {
    # the layer's GPU path at T = 32: layer_route + layer_up + layer_down + combine
    "layer_bf16": {
        "kernel_sources": ("paper_2608_21240_amd/csrc/layer_decode.hip",
                           "paper_2608_21240_amd/csrc/route_device.h",
                           "paper_2608_21240_amd/csrc/expert_ffn_tiles.h",
                           "paper_2608_21240_amd/csrc/expert_ffn_mx_tiles.h",
                           "paper_2608_21240_amd/csrc/tile_index.h",
                           "paper_2608_21240_amd/csrc/combine.hip",
                           "paper_2608_21240_amd/csrc/spice_internal.h"),
        "source_sha256_16": "85a4b3319e438b10",
        "fetch_kib_per_call": 12031.4 + 184134.4 + 90267.5 + 905.7,
        "write_kib_per_call": 260.1 + 675.8 + 1195.7 + 128.0,
        "fetch_factor": 2.0,
        "write_factor": 1.0,
        "profile": "profiles/layer_dsv2_decode_kernel_trace_counters.md",
    },
    # the same with the routed experts in MXFP4 (the layer kernels' MX instantiations)
    "layer_mxfp4": {
        "kernel_sources": ("paper_2608_21240_amd/csrc/layer_decode.hip",
                           "paper_2608_21240_amd/csrc/route_device.h",
                           "paper_2608_21240_amd/csrc/expert_ffn_tiles.h",
                           "paper_2608_21240_amd/csrc/expert_ffn_mx_tiles.h",
                           "paper_2608_21240_amd/csrc/tile_index.h",
                           "paper_2608_21240_amd/csrc/combine.hip",
                           "paper_2608_21240_amd/csrc/spice_internal.h"),
        "source_sha256_16": "85a4b3319e438b10",
        "fetch_kib_per_call": 12026.7 + 55328.1 + 26318.2 + 903.1,
        "write_kib_per_call": 260.0 + 675.9 + 1195.9 + 128.0,
        "fetch_factor": 2.0,
        "write_factor": 1.0,
        "profile": "profiles/ffn_dsv2_decode_T32_mxfp4.md",
    },
    # the grouped-FFN call alone at T = 32: ffn_up + ffn_down
    "bf16": {
        "kernel_sources": ("paper_2608_21240_amd/csrc/expert_ffn.hip",
                           "paper_2608_21240_amd/csrc/expert_ffn_tiles.h",
                           "paper_2608_21240_amd/csrc/tile_index.h",
                           "paper_2608_21240_amd/csrc/spice_internal.h"),
        "source_sha256_16": "8ebc4e31dbfbbff5",
        "fetch_kib_per_call": 189111.0 + 96795.7,
        "write_kib_per_call": 462.4 + 1452.0,
        "fetch_factor": 2.0,
        "write_factor": 1.0,
        "profile": "profiles/layer_dsv2_decode_kernel_trace_counters.md",
    },
    "mxfp4": {
        "kernel_sources": ("paper_2608_21240_amd/csrc/expert_ffn_mx.hip",
                           "paper_2608_21240_amd/csrc/expert_ffn_mx_tiles.h",
                           "paper_2608_21240_amd/csrc/expert_ffn_tiles.h",
                           "paper_2608_21240_amd/csrc/tile_index.h",
                           "paper_2608_21240_amd/csrc/spice_internal.h"),
        "source_sha256_16": "562f86020ed6b351",
        "fetch_kib_per_call": 60286.4 + 32786.7,
        "write_kib_per_call": 462.6 + 1452.0,
        "fetch_factor": 2.0,
        "write_factor": 1.0,
        "profile": "profiles/ffn_dsv2_decode_T32_mxfp4.md",
    },
}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=60)
    p.add_argument("--warmup", type=int, default=6)
    p.add_argument("--instances", type=int, default=4, help="independent layer instances to rotate over")
    p.add_argument("--batches", default="1,8,32", help="decode batch sizes; the last is the headline")
    p.add_argument("--threads", type=int, default=0, help="host threads of the exact CPU path (0 = all)")
    p.add_argument("--cpu-baseline-seconds", type=float, default=12.0)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--calib-copy-mib", type=int, default=0,
                   help="finish with a plain device copy of this many MiB (a known-size reference for counters)")
    p.add_argument("--workload", default="dsv2_decode",
                   choices=("dsv2_decode", "qwen2_decode", "qwen2_prefill", "dsv2_stack", "lore_fit"),
                   help="dsv2_decode: the decode layer (default); qwen2_decode: the Qwen2-57B-A14B-shaped "
                        "decode batch (T=16) at 16/32/48 resident experts and the prefill record only; "
                        "qwen2_prefill: the 4096-token "
                        "Qwen2-57B-A14B-shaped layer on the MFMA GEMM path; dsv2_stack: the 26-layer "
                        "LRU-cached decode stack with and without speculative prefetching; lore_fit: "
                        "LoRE calibration fits of DSV2-Lite experts (512 tokens, rank 32)")
    p.add_argument("--spec-depth", type=int, default=2, help="dsv2_stack: lookahead layers of the draft rollout")
    p.add_argument("--spec-tau", type=float, default=0.0, help="dsv2_stack: halting threshold of the rollout")
    p.add_argument("--max-prefetch", type=int, default=3, help="dsv2_stack: prefetched experts per layer and call")
    p.add_argument("--resident", type=int, default=64, help="qwen2_prefill: resident experts")
    p.add_argument("--split", default="auto", choices=("auto", "off"),
                   help="exact-miss split (Eq. 12): auto = calibrate the cost model on this host and let the "
                        "planner fetch experts to the GPU when that beats all-CPU; off = all-CPU")
    p.add_argument("--fetch-slots", type=int, default=8, help="fetch pool slots for the exact-miss split")
    p.add_argument("--gpu-reps", type=int, default=100, help="calls timed for the GPU path (median)")
    p.add_argument("--no-qwen2", action="store_true", help="skip the Qwen2-57B-A14B-shaped decode/prefill records")
    p.add_argument("--weights", default="bf16", choices=("bf16", "mxfp4"),
                   help="dsv2_decode: routed experts' weights in bf16 (default) or MXFP4 (E2M1 + an E8M0 scale "
                        "per 32; the exact-miss split then stays off)")
    return p.parse_args()


def recorded_traffic(weights: str = "bf16"):
    """HBM bytes per grouped-FFN call from the counter record of this weight format, or None
    if there is none or the kernel changed since it was taken."""
    import hashlib

    rec = TRAFFIC_RECORDS.get(weights)
    if rec is None:
        return None
    h = hashlib.sha256()
    for rel in rec["kernel_sources"]:
        h.update(open(os.path.join(ROOT, rel), "rb").read())
    if h.hexdigest()[:16] != rec["source_sha256_16"]:
        return None
    return int(1024 * (rec["fetch_kib_per_call"] * rec["fetch_factor"] + rec["write_kib_per_call"] * rec["write_factor"]))


def expert_bytes(wl) -> int:
    """HBM bytes of one routed expert in the workload's weight format."""
    from paper_2608_21240_amd import synth, workloads as W

    s = wl.shape
    if wl.wfmt == W.WFMT_MXFP4:
        return synth.mxfp4_bytes(2 * s.inter, s.d) + synth.mxfp4_bytes(s.d, s.inter)
    return s.expert_bytes


def algorithmic_bytes(shape, idx, cls, e_bytes=None):
    """Bytes the method must move on the GPU for one layer call, by definition:
    router + shared block + distinct HIT experts x expert bytes + distinct LoRE experts x
    factor bytes + x read + out written.  Skipped non-resident experts and the fp32 scratch
    rows (y_slots, y_shared, H) are not counted.  ffn: the share of the grouped-FFN call
    (shared block, HIT experts, LoRE factors, x)."""
    T, K = idx.shape
    d, wb = shape.d, shape.wbytes
    hit_e = len(set(idx[cls == 0].tolist()))
    lore_e = len(set(idx[cls == 1].tolist()))
    x_b = T * d * wb
    eb = shape.expert_bytes if e_bytes is None else e_bytes
    ffn = hit_e * eb + shape.shared_bytes + lore_e * shape.lore_bytes + x_b
    total = shape.n_experts * d * wb + ffn + T * d * wb
    return dict(ffn=ffn, total=total, hit_experts=hit_e, lore_experts=lore_e,
                slots=np.bincount(cls.ravel(), minlength=3).tolist(), exact_experts=len(set(idx[cls == 2].tolist())))


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def time_gpu_path(devs, xs, confs, runs, T, reps: int = 100, warm: int = 10, graphs: bool = True):
    """The GPU path of a layer call (moe_layer_gpu with the combine; routing, FFN, LoRE and
    combine, the host copies included, the exact residual precomputed in each run's pinned
    buffer), back to back over the layer instances, with plain launches and as replays of
    one captured HIP graph per instance.  Two timings of each on the launch stream: the
    mean per call over one event pair around `reps` back-to-back calls (the average
    duration the roofline uses), and the median of per-call event pairs (a latency figure;
    each pair adds its own markers to the stream).  A spin kernel queued first lets the
    host queue every call before the GPU reaches it, so no span holds host submission
    time.  Returns ((mean, median), (graph mean, graph median) or None, graph_ok)."""
    import torch

    n = len(devs)

    def call(i):
        runs[i].layer_gpu(devs[i], xs[i], confs[i], T, to_host=True, resid=runs[i].resid, out=True, mark=False)

    for w in range(warm):
        call(w % n)
    torch.cuda.synchronize()
    ref_out = []
    for i in range(n):
        call(i)
        torch.cuda.synchronize()
        ref_out.append(runs[i].out[:T].clone())

    def timed(fn):
        spin = int(2e7 + 2e5 * reps)
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        torch.cuda.synchronize()
        torch.cuda._sleep(spin)
        for k in range(reps):
            evs[k][0].record()
            fn(k % n)
            evs[k][1].record()
        torch.cuda.synchronize()
        median = float(np.median([a.elapsed_time(b) for a, b in evs]) * 1e3)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(spin)
        a.record()
        for k in range(reps):
            fn(k % n)
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / reps, median

    plain = timed(call)
    graph, graph_ok = None, None
    if graphs:
        try:
            gs = []
            side = torch.cuda.Stream()
            for i in range(n):
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=side):
                    call(i)
                gs.append(g)
            torch.cuda.synchronize()
            graph = timed(lambda i: gs[i].replay())
            # every replay's output equals the eager call's (eager work and a sync in between)
            graph_ok = True
            for i in range(n):
                call(i)
                torch.cuda.synchronize()
                gs[i].replay()
                torch.cuda.synchronize()
                graph_ok &= bool(torch.equal(runs[i].out[:T], ref_out[i]))
        except Exception as ex:  # capture not available: report plain launches only
            print(f"[bench] graph capture failed: {ex}", file=sys.stderr, flush=True)
            graph, graph_ok = None, None
    if any(r.flags() != 0 for r in runs):
        raise RuntimeError("device flags raised during the GPU-path timing")
    return plain, graph, graph_ok


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the layer path is single-GPU; "
              "expert sharding across GPUs is not built)", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2608_21240_amd import layer as LY, synth, workloads as W

    torch.cuda.set_device(0)
    if args.workload == "qwen2_prefill":
        return prefill_main(args)
    if args.workload == "qwen2_decode":
        rec = qwen2_records(args)
        r32 = rec["decode_T16"]["R32"]
        print(json.dumps({
            "metric": "MoE-layer decode tokens/s + achieved HBM GB/s (% peak), Qwen2-57B-A14B-shaped",
            "value": r32["tokens_per_s"], "unit": "tokens/s", "n_gpus": 1, "steps": None, "warmup": None,
            "ms_per_step": round(r32["avg_call_us"] / 1e3, 4), "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded random-init Qwen2-57B-A14B-shaped layer)",
            "config": {"workload": "qwen2_57b_a14b_moe_layer_decode_T16_R32", "resident": 32, "tokens": 16},
            "roofline": {"bound": "hbm", "kernel": "the layer's GPU path, one moe_layer_gpu call with the combine",
                         "achieved": r32["GBps"], "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": r32["frac"],
                         "traffic": None},
            "qwen2": rec}), flush=True)
        return
    if args.workload == "dsv2_stack":
        return stack_main(args)
    if args.workload == "lore_fit":
        return lore_fit_main(args)
    batches = [int(b) for b in args.batches.split(",")]
    wl = W.WORKLOADS["dsv2_decode_mxfp4_t32" if args.weights == "mxfp4" else "dsv2_decode_t32"]
    if args.weights == "mxfp4":
        args.split = "off"  # the fetched-expert split copies and runs bf16 experts only
    shape = wl.shape
    t_gen = time.time()
    hosts, devs = [], []
    for i in range(args.instances):
        h = LY.HostLayer(wl, layer=i)
        devs.append(LY.DeviceLayer(h))
        hosts.append(h)
    torch.cuda.synchronize()
    print(f"[bench] {args.instances} layer instances ready in {time.time() - t_gen:.1f}s "
          f"({devs[0].hbm_bytes() / 1e9:.2f} GB HBM each)", file=sys.stderr, flush=True)

    results = {}
    split_info = {}
    for T in batches:
        run = LY.LayerRun(shape, T, devs[0].C, tau=wl.tau, fetch_slots=args.fetch_slots if args.split == "auto" else 0,
                          wfmt=wl.wfmt)
        xs = [LY.to_tensor(synth.gen_x(wl, i, 0, T), shape.dtype, "cuda") for i in range(args.instances)]
        confs = [torch.from_numpy(synth.gen_conf(wl, i, 0, T)).cuda() for i in range(args.instances)]
        # per instance: one untimed layer call, for the class counts (fixed inputs per instance)
        # and the exact residual that the GPU-path timing takes as precomputed
        per_inst, gruns = [], []
        for i in range(args.instances):
            r = LY.LayerRun(shape, T, devs[i].C, tau=wl.tau, wfmt=wl.wfmt)
            r.forward(devs[i], xs[i], confs[i], T, n_threads=args.threads)
            torch.cuda.synchronize()
            per_inst.append(algorithmic_bytes(shape, r.idx_host[:T].numpy().copy(), r.cls_host[:T].numpy().copy(),
                                              expert_bytes(wl)))
            gruns.append(r)
        for w in range(args.warmup):
            i = w % args.instances
            run.forward(devs[i], xs[i], confs[i], T, n_threads=args.threads)
        torch.cuda.synchronize()
        if run.flags() != 0:
            raise RuntimeError("device flags raised during warmup")
        split = None
        if args.split == "auto":
            # the calibration reads the routing copies of one call on the instance it passes
            run.forward(devs[0], xs[0], confs[0], T, n_threads=args.threads)
            torch.cuda.synchronize()
            split = calibrate_split(run, devs[0], shape, T, args)
        if split is not None:
            split_info[T] = {f: float(f"{getattr(split, f):.4g}") for f, _ in split._fields_}
            for w in range(args.warmup):
                i = w % args.instances
                run.forward(devs[i], xs[i], confs[i], T, n_threads=args.threads, split=split)
            torch.cuda.synchronize()

        # end to end: whole layer calls, the host's exact residual overlapped with the GPU
        fetched, host_t, host_e = [], [], []
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(args.steps):
            i = k % args.instances
            run.forward(devs[i], xs[i], confs[i], T, n_threads=args.threads, split=split)
            fetched.append(len(run.last_fetch))
            host_t.append(run.last_host_s)
            host_e.append(run.last_host_experts)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        if run.flags() != 0:
            raise RuntimeError("device flags raised during the timed steps")

        # the GPU path alone: routing to combine on the device stream, the host residual precomputed
        (gpu_us, gpu_med), graph, graph_ok = time_gpu_path(devs, xs, confs, gruns, T, reps=args.gpu_reps)
        graph_us, graph_med = graph if graph else (None, None)
        tot_bytes = float(np.mean([p["total"] for p in per_inst]))
        results[T] = dict(
            T=T, wall_s=wall, ms_per_step=1e3 * wall / args.steps, tokens_per_s=T * args.steps / wall,
            gpu_us=gpu_us, gpu_median_us=gpu_med, gpu_tokens_per_s=T / (gpu_us * 1e-6),
            gpu_GBps=tot_bytes / (gpu_us * 1e-6) / 1e9,
            gpu_graph_us=graph_us, gpu_graph_median_us=graph_med, graph_matches_eager=graph_ok,
            gpu_graph_GBps=(tot_bytes / (graph_us * 1e-6) / 1e9) if graph_us else None,
            bytes_per_call=tot_bytes, fetched_experts_per_step=float(np.mean(fetched)),
            host_exact_ms=float(np.mean(host_t) * 1e3), host_exact_experts=float(np.mean(host_e)),
            host_exact_GBps=float(np.sum(host_e) * expert_bytes(wl) / max(np.sum(host_t), 1e-12) / 1e9),
            classes=per_inst[0]["slots"], hit_experts=[p["hit_experts"] for p in per_inst],
            lore_experts=[p["lore_experts"] for p in per_inst], exact_experts=[p["exact_experts"] for p in per_inst],
        )
        # the grouped-FFN call on its own (moe_expert_ffn_grouped, LoRE fused)
        launch_us, launch_bytes = time_ffn_launches(devs, xs, confs, per_inst, shape, wl, T, args)
        results[T].update(ffn_call_us=launch_us, ffn_call_GBps=launch_bytes / (launch_us * 1e-6) / 1e9,
                          ffn_call_bytes=launch_bytes)
        # the routing call on its own (inside the layer call it runs in the first launch)
        results[T].update(route_call_us=time_route_calls(devs, xs, confs, shape, wl, T))
        print(f"[bench] T={T}: {json.dumps(results[T])}", file=sys.stderr, flush=True)
        del run, gruns

    head = results[batches[-1]]
    mx = args.weights == "mxfp4"
    kern = "layer_route_kernel + layer_up_kernel + layer_down_kernel + combine_kernel" + (
        " (MXFP4 HIT tiles)" if mx else "")
    line = {
        "metric": METRIC, "value": round(head["tokens_per_s"], 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(head["ms_per_step"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded random-init DSV2-Lite-shaped layers, Zipf(1.1) residency, conf~U(0,1))",
        "config": {"workload": f"dsv2_lite_moe_layer_decode_T{head['T']}" + ("_mxfp4" if mx else ""),
                   "expert_weights": args.weights, "hidden": shape.d,
                   "experts": shape.n_experts, "top_k": shape.top_k, "inter": shape.inter,
                   "shared_inter": shape.shared_inter, "lore_rank": shape.lore_rank, "resident": wl.resident,
                   "tau": wl.tau, "tokens": head["T"], "layer_instances": args.instances,
                   "host_threads": args.threads or os.cpu_count()},
        "roofline": {"bound": "hbm",
                     "kernel": f"the layer's GPU path, one moe_layer_gpu call with the combine: {kern}",
                     "achieved": round(head["gpu_GBps"], 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(head["gpu_GBps"] / HBM_PEAK_GBS, 4),
                     "traffic": recorded_traffic("layer_" + args.weights),
                     "bytes_per_call": int(head["bytes_per_call"]), "avg_call_us": round(head["gpu_us"], 2),
                     "median_call_us": round(head["gpu_median_us"], 2),
                     "graph_avg_call_us": round(head["gpu_graph_us"], 2) if head["gpu_graph_us"] else None,
                     "graph_frac": round(head["gpu_graph_GBps"] / HBM_PEAK_GBS, 4) if head["gpu_graph_GBps"] else None,
                     "by_batch": {str(T): {"us": round(r["gpu_us"], 2), "frac": round(r["gpu_GBps"] / HBM_PEAK_GBS, 4),
                                           "median_us": round(r["gpu_median_us"], 2),
                                           "graph_us": round(r["gpu_graph_us"], 2) if r["gpu_graph_us"] else None,
                                           "tokens_per_s": round(r["gpu_tokens_per_s"], 1),
                                           "bytes_per_call": int(r["bytes_per_call"])}
                                  for T, r in results.items()}},
        "ffn_call": {"kernel": "grouped expert FFN call alone: " + (
                         "ffn_up_mx_kernel + ffn_down_mx_kernel" if mx else "ffn_up_kernel + ffn_down_kernel") +
                     " (moe_expert_ffn_grouped, LoRE fused)",
                     "achieved": round(head["ffn_call_GBps"], 1), "frac": round(head["ffn_call_GBps"] / HBM_PEAK_GBS, 4),
                     "avg_launch_us": round(head["ffn_call_us"], 2), "bytes_per_call": int(head["ffn_call_bytes"]),
                     "traffic": recorded_traffic(args.weights)},
        "route_call": {"kernel": "route_logits_kernel, one launch with the bucketing in its last block "
                                 "(moe_route_bucket alone, back-to-back calls; the layer call routes inside "
                                 "layer_route_kernel instead)",
                       "us_by_batch": {str(T): round(r["route_call_us"], 2) for T, r in results.items()}},
        "host_path": {"exact_ms": round(head["host_exact_ms"], 3), "experts_per_step": round(head["host_exact_experts"], 2),
                      "GBps": round(head["host_exact_GBps"], 1),
                      "note": "exact-miss residual on the host CPU (Eq. 12 M_cpu): bound by host DRAM reads"},
        "by_batch": {str(T): {k: (round(v, 3) if isinstance(v, float) else v) for k, v in r.items()}
                     for T, r in results.items()},
        "exact_split": {"mode": args.split, "fetch_slots": args.fetch_slots if args.split == "auto" else 0,
                        "cost_model_by_batch": {str(T): c for T, c in split_info.items()}},
    }
    if not args.no_cpu_baseline:
        wl_h = wl.with_(tokens=head["T"])
        line["cpu_baseline"] = cpu_baseline(wl_h, hosts[0], args.cpu_baseline_seconds)
        line["cpu_baseline_library"] = cpu_library_baseline(wl_h, hosts[0], devs[0], args.cpu_baseline_seconds / 3)
    del devs, hosts
    torch.cuda.empty_cache()
    if not args.no_qwen2 and not mx:
        line["qwen2"] = qwen2_records(args)
    if args.calib_copy_mib > 0:
        a = torch.empty(args.calib_copy_mib << 20, dtype=torch.uint8, device="cuda")
        torch.empty_like(a).copy_(a)
        torch.cuda.synchronize()
    print(json.dumps(line), flush=True)


def time_ffn_launches(devs, xs, confs, per_inst, shape, wl, T, args, reps: int = 25):
    """Mean duration (us) and mean algorithmic bytes of one grouped-FFN call, timed with
    HIP events on the launch stream over back-to-back calls that rotate over the layer
    instances (each routed once beforehand into its own buffers)."""
    import torch

    from paper_2608_21240_amd import layer as LY

    runs = []
    for i, dev in enumerate(devs):
        r = LY.LayerRun(shape, T, dev.C, tau=wl.tau, wfmt=wl.wfmt)
        r.route(dev, xs[i], confs[i], T, to_host=False)
        runs.append(r)
    for _ in range(2):
        for i, dev in enumerate(devs):
            runs[i].experts(dev, xs[i], T)
    stream = torch.cuda.current_stream()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(reps * len(devs))]
    torch.cuda.synchronize()
    # a spin kernel ahead of the loop lets the host queue every launch before the GPU
    # reaches the first one, so no event span contains host submission time
    torch.cuda._sleep(int(2e7 + 4e5 * len(evs)))
    j = 0
    for _ in range(reps):
        for i, dev in enumerate(devs):
            evs[j][0].record(stream)
            runs[i].experts(dev, xs[i], T)
            evs[j][1].record(stream)
            j += 1
    torch.cuda.synchronize()
    if any(r.flags() != 0 for r in runs):
        raise RuntimeError("device flags raised during the FFN launch timing")
    us = float(np.mean([a.elapsed_time(b) for a, b in evs]) * 1e3)
    nbytes = float(np.mean([per_inst[i]["ffn"] for i in range(len(devs))]))
    return us, nbytes


def time_route_calls(devs, xs, confs, shape, wl, T, reps: int = 50):
    """Mean duration (us) of one standalone routing call (moe_route_bucket: logits, top-K,
    gates, classes, bucketing and work lists, no host copies): one event pair around
    back-to-back calls that rotate over the layer instances, behind a spin kernel, with no
    event recorded between the calls."""
    import torch

    from paper_2608_21240_amd import layer as LY

    runs = [LY.LayerRun(shape, T, dev.C, tau=wl.tau, wfmt=wl.wfmt) for dev in devs]
    for i, dev in enumerate(devs):
        runs[i].route(dev, xs[i], confs[i], T, to_host=False)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda._sleep(int(2e7))
    a.record()
    for _ in range(reps):
        for i, dev in enumerate(devs):
            runs[i].route(dev, xs[i], confs[i], T, to_host=False, mark=False)
    b.record()
    torch.cuda.synchronize()
    if any(r.flags() != 0 for r in runs):
        raise RuntimeError("device flags raised during the routing timing")
    return a.elapsed_time(b) * 1e3 / (reps * len(devs))


def calibrate_split(run, dev, shape, T, args):
    """Cost model of the exact-miss split measured on this host, from the routing copies
    of the last call on `dev` (restored afterwards).

    CPU arithmetic rate: one exact expert serving every token against the same expert
    serving one token.  CPU rate over expert weights: every exact expert of the call with
    one token each, less that arithmetic.  PCIe: one untimed fetch, then the best of two
    timed fetches into the pool.  Host timings are the best of three calls."""
    import torch

    from paper_2608_21240_amd import spice

    idx0 = run.idx_host[:T].numpy().copy()
    cls0 = run.cls_host[:T].numpy().copy()
    exact = sorted(set(idx0[cls0 == 2].tolist()))
    if not exact:
        return None
    lore = np.full(cls0.shape, 1, np.uint8)  # LoRE slots are not the host's work

    def cpu_time(idx, cls):
        run.idx_host[:T].copy_(torch.from_numpy(idx))
        run.cls_host[:T].copy_(torch.from_numpy(cls))
        best = float("inf")
        for _ in range(3):
            t0 = time.perf_counter()
            spice.moe_exact_residual_host(run.cfg, T, run.x_host, run.idx_host, run.w_host, run.cls_host,
                                          dev.host_w13, dev.host_w2, run.resid, args.threads)
            best = min(best, time.perf_counter() - t0)
        return best

    flops_tok = 6.0 * shape.inter * shape.d
    cpu_flops = 1e18  # one token: the arithmetic cannot be told apart; the byte rate absorbs it
    e0 = exact[0]
    if T >= 4:
        # slot k = 0 of every token goes to e0: no token lists an expert twice, since the
        # other slots of a token are masked to LoRE
        many_i, many_c = idx0.copy(), lore.copy()
        many_i[:, 0] = e0
        many_c[:, 0] = 2
        one_c = lore.copy()
        one_c[0, 0] = 2
        extra = cpu_time(many_i, many_c) - cpu_time(many_i, one_c)
        if extra > 0:
            cpu_flops = (T - 1) * flops_tok / extra
    first = lore.copy()
    seen = set()
    for t, k in zip(*np.nonzero(cls0 == 2)):
        if idx0[t, k] not in seen:
            seen.add(idx0[t, k])
            first[t, k] = 2
    t_first = cpu_time(idx0, first)
    n_exp = len(exact)
    cpu_bytes = n_exp * shape.expert_bytes / max(t_first - n_exp * flops_tok / cpu_flops, 0.2 * t_first)
    run.idx_host[:T].copy_(torch.from_numpy(idx0))
    run.cls_host[:T].copy_(torch.from_numpy(cls0))
    probe = [e for e in range(shape.n_experts) if dev.host_w13[e] is not None][: min(4, run.fetch_slots)]

    def fetch_time():
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        with torch.cuda.stream(run.copy_stream):
            spice.moe_fetch_experts(run.cfg, probe, dev.host_w13, dev.host_w2, run.w13_fetch, run.w2_fetch,
                                    run.fetch_slots, run.fetch_expert, run.fetch_stage)
        run.copy_stream.synchronize()
        return time.perf_counter() - t0

    fetch_time()
    pcie = len(probe) * shape.expert_bytes / min(fetch_time(), fetch_time())
    # the GPU side pays one fetched-FFN call (two launches); a split must save 5 %
    return spice.spice_split_cost_t(cpu_bytes, cpu_flops, pcie, 30e-6, 0.05)


def stack_main(args):
    """26 DSV2-Lite-shaped layers with a 24-slot LRU cache each, T=64 per step (the stack
    workload), run with and without speculative prefetching (Sec. 4.1).  Every step is a
    whole decode step through all layers: per layer route, FFN + LoRE, the host residual of
    the exact misses, combine, the cache's admissions and, with prefetching, the draft
    rollout (overlapped with the host residual) and the speculative admissions.  The
    roofline is for the rollout's own GPU work (route + shared/LoRE FFN + update per depth),
    HBM-bound: router + shared block + distinct predicted experts' LoRE factors per depth."""
    import torch

    from paper_2608_21240_amd import synth, workloads as W
    from paper_2608_21240_amd.layer import to_tensor
    from paper_2608_21240_amd.stack import StackModel, StackRun

    wl = W.WORKLOADS["dsv2_stack"]
    s, T, L = wl.shape, wl.tokens, wl.layers
    t_gen = time.time()
    m = StackModel(wl)
    print(f"[bench] stack of {L} layers ready in {time.time() - t_gen:.1f}s", file=sys.stderr, flush=True)
    pf = dict(depth=args.spec_depth, l_min=1, tau=args.spec_tau, max_prefetch=args.max_prefetch)
    xs = [to_tensor(synth.gen_x(wl, 0, k, T), s.dtype, "cuda") for k in range(args.warmup + args.steps)]
    confs = [[torch.from_numpy(synth.gen_conf(wl, l, k, T)).cuda() for l in range(L)]
             for k in range(args.warmup + args.steps)]
    res = {}
    for use in (False, True):
        sr = StackRun(m, max_admit=4, prefetch=pf if use else None, n_threads=args.threads)
        for k in range(args.warmup):
            sr.step(k, xs[k], confs[k])
        torch.cuda.synchronize()
        n0 = len(sr.trace)
        if use:
            sr.spec_events = []
        t0 = time.perf_counter()
        for k in range(args.warmup, args.warmup + args.steps):
            sr.step(k, xs[k], confs[k])
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        tr = sr.trace[n0:]
        cnt = np.sum([np.bincount(t["cls"].ravel(), minlength=3) for t in tr], axis=0)
        r = dict(tokens_per_s=T * args.steps / wall, ms_per_step=1e3 * wall / args.steps,
                 slot_hit_rate=float(cnt[0] / cnt.sum()), exact_share=float(cnt[2] / cnt.sum()),
                 admissions_per_call=float(np.mean([len(t["admitted"]) for t in tr])))
        if use:
            ms = np.array([a.elapsed_time(b) for a, b, _ in sr.spec_events])
            depths = np.array([n for _, _, n in sr.spec_events])
            # algorithmic bytes of one depth: router, shared block, LoRE factors of the distinct
            # predicted experts (from the issue lists, uncut), x/h rows and the fp32 outputs
            wb = s.wbytes
            nexp = [len(set(np.concatenate([sr.spec.pred_idx_h[j].numpy().ravel()]).tolist()) - {-1})
                    for j in range(sr.spec.n)]
            per_depth = (s.n_experts * s.d * wb + s.shared_bytes + float(np.mean(nexp)) * s.lore_bytes
                         + 2 * T * s.d * wb + (T * s.top_k + T) * s.d * 4)
            r.update(rollout_us=float(ms.mean() * 1e3), rollout_us_per_depth=float((ms / depths).mean() * 1e3),
                     rollout_GBps=float(per_depth * depths.sum() / (ms.sum() * 1e-3) / 1e9),
                     bytes_per_depth=int(per_depth),
                     prefetched_per_call=float(np.mean([sum(len(a) for a, _ in t["prefetched"]) for t in tr])))
        sr.close()
        res["prefetch" if use else "no_prefetch"] = {k: (round(v, 4) if isinstance(v, float) else v)
                                                     for k, v in r.items()}
        print(f"[bench] stack prefetch={use}: {json.dumps(res['prefetch' if use else 'no_prefetch'])}",
              file=sys.stderr, flush=True)
    on = res["prefetch"]
    line = {
        "metric": "MoE stack decode tokens/s, 26 DSV2-Lite-shaped layers, 24-slot LRU cache per layer",
        "value": round(on["tokens_per_s"], 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(on["ms_per_step"], 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded random-init DSV2-Lite-shaped layers, conf~U(0,1); every layer sees the same x)",
        "config": {"workload": "dsv2_stack_T64_L26_C24_prefetch", "layers": L, "tokens": T,
                   "cache_slots": wl.cache_slots, "max_admit": 4, "spec_depth": pf["depth"],
                   "spec_tau": pf["tau"], "max_prefetch": pf["max_prefetch"]},
        "roofline": {"bound": "hbm", "kernel": "draft rollout per depth: route + shared/LoRE FFN + spec update",
                     "achieved": round(on["rollout_GBps"], 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(on["rollout_GBps"] / HBM_PEAK_GBS, 4), "traffic": None,
                     "bytes_per_depth": on["bytes_per_depth"], "avg_depth_us": round(on["rollout_us_per_depth"], 2)},
        "by_mode": res,
    }
    print(json.dumps(line), flush=True)


def lore_fit_main(args):
    """LoRE calibration fits (Eq. 10) of DSV2-Lite-shaped experts from 512 calibration tokens
    at rank 32, one expert per step (rotating over 8 experts).  A step is one whole fit:
    E_e and S on the tokens (MFMA GEMM path), residual, the two fp64 Gram matrices, the host
    eigen-decomposition and solve, and the factor products.  The GPU part is timed with
    events around the whole call less the host's own share, which the call cannot expose;
    the rocprofv3 kernel trace gives the per-kernel split."""
    import torch

    from paper_2608_21240_amd import layer as LY, spice, synth, workloads as W

    s = W.DSV2
    n, r, E = 512, 32, 8
    wl = W.Workload("lore_fit", s, tokens=n, resident=0, skew=False)
    dt = s.dtype
    experts = [tuple(LY.to_tensor(a, dt, "cuda") for a in synth.gen_expert(wl, 0, e)) for e in range(E)]
    w13s, w2s = (LY.to_tensor(a, dt, "cuda") for a in synth.gen_shared(wl, 0))
    X = LY.to_tensor(synth.gen_x(wl, 0, 0, n), dt, "cuda")
    cfg = spice.make_cfg(s, 1)
    A = torch.empty((r, s.d), dtype=torch.float32, device="cuda")
    B = torch.empty((s.d, r), dtype=torch.float32, device="cuda")
    wsb = spice.lib().spice_lore_fit_workspace_bytes(spice.ctypes.byref(cfg), n, r)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    for k in range(args.warmup):
        spice.moe_lore_fit(cfg, n, r, X, *experts[k % E], w13s, w2s, A, B, None, ws, wsb)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    losses = []
    for k in range(args.steps):
        losses.append(spice.moe_lore_fit(cfg, n, r, X, *experts[k % E], w13s, w2s, A, B, None, ws, wsb))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    line = {
        "metric": "LoRE calibration fits per second (DSV2-Lite expert, 512 tokens, rank 32)",
        "value": round(args.steps / wall, 3), "unit": "fits/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(1e3 * wall / args.steps, 2), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16 in, fp32/fp64 fit",
        "data": "synthetic (seeded random-init DSV2-Lite expert and shared block, N(0,1) calibration tokens)",
        "config": {"workload": "lore_fit_dsv2_n512_r32", "tokens": n, "rank": r, "hidden": s.d, "inter": s.inter,
                   "shared_inter": s.shared_inter},
        "mean_loss": float(np.mean(losses)),
    }
    print(json.dumps(line), flush=True)


MFMA_BF16_PEAK_TFLOPS = 2500.0


def prefill_main(args):
    """Qwen2-57B-A14B-shaped layer at 4096 tokens: every step is a whole layer call
    (route, grouped MFMA GEMMs of the HIT experts and the shared block, LoRE and the
    exact CPU path for absent experts, combine); the roofline is MFMA-bound."""
    import torch

    from paper_2608_21240_amd import layer as LY, synth, workloads as W

    wl = W.WORKLOADS["qwen2_prefill"].with_(resident=args.resident)
    s, T = wl.shape, wl.tokens
    t_gen = time.time()
    host = LY.HostLayer(wl, 0)
    dev = LY.DeviceLayer(host, host_exact=args.resident < s.n_experts)
    # separate routing and FFN calls, so that events can bracket the FFN launch
    run = LY.LayerRun(s, T, dev.C, tau=wl.tau, layer_call=False)
    x = LY.to_tensor(synth.gen_x(wl, 0, 0, T), s.dtype, "cuda")
    conf = torch.from_numpy(synth.gen_conf(wl, 0, 0, T)).cuda()
    exact = args.resident < s.n_experts
    run.forward(dev, x, conf, T, exact=exact, n_threads=args.threads)
    torch.cuda.synchronize()
    cls = run.slot_class[:T].cpu().numpy()
    n_hit, n_lore = int((cls == 0).sum()), int((cls == 1).sum())
    # FLOPs of the grouped FFN launch: SwiGLU of every HIT slot and of the shared block for
    # every token (6 d I per token-expert pair), LoRE A and B products (4 d r per slot)
    flops = 6.0 * T * s.d * s.shared_inter + 6.0 * n_hit * s.d * s.inter + 4.0 * n_lore * s.d * s.lore_rank
    print(f"[bench] prefill layer ready in {time.time() - t_gen:.1f}s, classes "
          f"{np.bincount(cls.ravel(), minlength=3).tolist()}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        run.forward(dev, x, conf, T, exact=exact, n_threads=args.threads)
    torch.cuda.synchronize()
    names = ("start", "routed", "experts", "resid", "end")
    evs = [{n: torch.cuda.Event(enable_timing=True) for n in names} for _ in range(args.steps)]
    t0 = time.perf_counter()
    for k in range(args.steps):
        run.forward(dev, x, conf, T, exact=exact, n_threads=args.threads, events=evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    if run.flags() != 0:
        raise RuntimeError("device flags raised")
    ffn_ms = np.array([e["routed"].elapsed_time(e["experts"]) for e in evs])
    route_event_us = float(np.median([e["start"].elapsed_time(e["routed"]) for e in evs]) * 1e3)
    # the routing alone: average over back-to-back calls from one event pair behind a spin
    # kernel and no event between the calls (a per-call event pair also holds the host's
    # submission of the call)
    reps = 30
    ra, rb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda._sleep(int(2e7))
    ra.record()
    for _ in range(reps):
        run.route(dev, x, conf, T, to_host=False, mark=False)
    rb.record()
    torch.cuda.synchronize()
    route_us = ra.elapsed_time(rb) * 1e3 / reps
    achieved = flops / (ffn_ms.mean() * 1e-3) / 1e12
    line = {
        "metric": "MoE-layer prefill tokens/s + grouped-FFN MFMA TFLOP/s (% peak), Qwen2-57B-A14B-shaped",
        "value": round(T * args.steps / wall, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(1e3 * wall / args.steps, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded random-init Qwen2-57B-A14B-shaped layer, Zipf(1.1) routing skew)",
        "config": {"workload": f"qwen2_57b_a14b_moe_layer_prefill_T{T}_R{args.resident}", "hidden": s.d,
                   "experts": s.n_experts, "top_k": s.top_k, "inter": s.inter, "shared_inter": s.shared_inter,
                   "lore_rank": s.lore_rank, "resident": args.resident, "tokens": T},
        "roofline": {"bound": "mfma", "kernel": "grouped expert FFN call: expert_gemm_kernel up + down "
                                                "(moe_expert_ffn_grouped, T >= 256)",
                     "achieved": round(achieved, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": None,
                     "flop_per_launch": flops, "avg_launch_us": round(float(ffn_ms.mean() * 1e3), 1)},
        "route_us": round(route_us, 1), "route_event_us": round(route_event_us, 1),
        "classes": np.bincount(cls.ravel(), minlength=3).tolist(),
    }
    print(json.dumps(line), flush=True)


def cpu_baseline(wl, host, budget_s):
    """The oracle (fp64, one thread) on whole layer calls of the same workload,
    batch after batch, until about budget_s seconds of CPU work are done."""
    import oracle as orc
    from paper_2608_21240_amd import synth

    s = wl.shape
    cfg = orc.make_cfg(s, tau=wl.tau, wfmt=wl.wfmt)
    w13, w2, la, lb = host.tables(range(s.n_experts), range(s.n_experts))
    tokens = 0
    steps = 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < budget_s:
        x = synth.gen_x(wl, 0, 1000 + steps, wl.tokens)
        conf = synth.gen_conf(wl, 0, 1000 + steps, wl.tokens)
        r = orc.route(cfg, x, host.wg, host.bias, host.resident_mask(), conf)
        for t in range(wl.tokens):
            orc.token_output(cfg, x[t], r["idx"][t], r["g"][t], r["cls"][t], w13, w2, host.w13s, host.w2s, la, lb)
            tokens += 1
            if time.perf_counter() - t0 >= budget_s:
                break
        steps += 1
    el = time.perf_counter() - t0
    return {"value": round(tokens / el, 3), "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "cpu_model": cpu_model(), "nproc": os.cpu_count(),
            "sample": f"{tokens} tokens ({steps} batch(es) of {wl.tokens}) of one DSV2-Lite layer: routing for the "
                      f"whole batch + full fp64 layer output per token, {el:.1f}s"}


def cpu_library_baseline(wl, host, dev, budget_s):
    """The library's host path as a whole-layer CPU implementation: every slot of a batch
    treated as an exact miss (moe_exact_residual_host over all routed experts) plus the
    shared block (the same entry with the shared block as a one-expert layer), on all host
    threads.  Routing comes from the oracle, outside the timed calls."""
    import oracle as orc
    from paper_2608_21240_amd import spice, synth, workloads as W

    s, T = wl.shape, wl.tokens
    cfg = spice.make_cfg(s, 0, tau=wl.tau)
    sh = W.MoEShape(s.d, 1, 1, s.shared_inter, 0, 0, s.dtype)
    cfg_sh = spice.make_cfg(sh, 0)
    ocfg = orc.make_cfg(s, tau=wl.tau)
    w13 = [host.expert(e)[0] for e in range(s.n_experts)]
    w2 = [host.expert(e)[1] for e in range(s.n_experts)]
    resid = np.zeros((T, s.d), np.float32)
    resid_s = np.zeros((T, s.d), np.float32)
    zero_idx = np.zeros((T, 1), np.int32)
    one_w = np.ones((T, 1), np.float32)
    exact1 = np.full((T, 1), 2, np.uint8)
    nproc = os.cpu_count() or 1
    spent, tokens, steps = 0.0, 0, 0
    while spent < budget_s or steps < 2:
        x = synth.gen_x(wl, 0, 2000 + steps, T)
        r = orc.route(ocfg, x, host.wg, host.bias, host.resident_mask(), synth.gen_conf(wl, 0, 2000 + steps, T))
        idx = np.ascontiguousarray(r["idx"], np.int32)
        g = np.ascontiguousarray(r["g"], np.float32)
        cls = np.full(idx.shape, 2, np.uint8)
        t0 = time.perf_counter()
        spice.moe_exact_residual_host(cfg, T, x, idx, g, cls, w13, w2, resid, nproc)
        spice.moe_exact_residual_host(cfg_sh, T, x, zero_idx, one_w, exact1, [host.w13s], [host.w2s], resid_s, nproc)
        el = time.perf_counter() - t0
        if steps > 0:  # the first call warms the host caches and the worker pool
            spent += el
            tokens += T
        steps += 1
    wbytes = s.n_experts * s.expert_bytes + s.shared_bytes
    return {"value": round(tokens / spent, 1), "unit": "tokens/s", "cores": nproc, "kind": "library host path",
            "cpu_model": cpu_model(),
            "sample": f"{tokens} tokens ({steps - 1} timed batches of {T}) of one DSV2-Lite layer: every slot exact "
                      f"(moe_exact_residual_host) plus the shared block, {nproc} threads, {spent:.2f}s; "
                      f"{wbytes / 1e9:.2f} GB of host weights per batch at most"}


def qwen2_records(args):
    """The Qwen2-57B-A14B-shaped layer (Sec. 5.1's second model): the 16-token decode batch at
    16, 32 and 48 resident experts (Zipf(1.1) skew, logit bias ln p) timed as the GPU path of
    a layer call (moe_layer_gpu with the combine; a pinned zero residual stands in for the
    host's, which is not computed here), against HBM; and the 4096-token prefill with all 64
    resident, its grouped-FFN call against the bf16 MFMA peak."""
    import torch

    from paper_2608_21240_amd import layer as LY, synth, workloads as W

    wl = W.WORKLOADS["qwen2_prefill"]
    s = wl.shape
    t0 = time.time()
    host = LY.HostLayer(wl, 0)
    dev = LY.DeviceLayer(host, host_exact=False)
    torch.cuda.synchronize()
    print(f"[bench] qwen2 layer ready in {time.time() - t0:.1f}s ({dev.hbm_bytes() / 1e9:.2f} GB HBM)",
          file=sys.stderr, flush=True)
    slot_all = dev.resident_slot.clone()
    out = {"model": "Qwen2-57B-A14B-shaped layer (d 3584, 64 experts, top-8, I 2560, shared I 20480, LoRE rank 64)"}
    dec = {}
    T = 16
    for R in (16, 32, 48):
        wlr = W.WORKLOADS[f"qwen2_decode_r{R}"]
        res = synth.resident_experts(wlr, 0)
        rs = torch.full_like(slot_all, -1)
        rs[res] = slot_all[res]
        dev.resident_slot.copy_(rs)
        run = LY.LayerRun(s, T, dev.C, tau=wlr.tau)
        run.resid.zero_()
        x = LY.to_tensor(synth.gen_x(wlr, 0, 0, T), s.dtype, "cuda")
        conf = torch.from_numpy(synth.gen_conf(wlr, 0, 0, T)).cuda()
        run.layer_gpu(dev, x, conf, T, to_host=False, resid=run.resid, out=True)
        torch.cuda.synchronize()
        idx, cls = run.topk_idx.cpu().numpy(), run.slot_class.cpu().numpy()
        b = algorithmic_bytes(s, idx, cls)
        (us, med), graph, gok = time_gpu_path([dev], [x], [conf], [run], T, reps=max(20, args.gpu_reps // 3))
        gus = graph[0] if graph else None
        dec[f"R{R}"] = {"resident": R, "tokens": T, "avg_call_us": round(us, 2), "median_call_us": round(med, 2),
                        "tokens_per_s": round(T / (us * 1e-6), 1),
                        "bytes_per_call": int(b["total"]), "GBps": round(b["total"] / (us * 1e-6) / 1e9, 1),
                        "frac": round(b["total"] / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                        "graph_us": round(gus, 2) if gus else None, "graph_matches_eager": gok,
                        "slots": b["slots"], "hit_experts": b["hit_experts"], "lore_experts": b["lore_experts"]}
        print(f"[bench] qwen2 decode R={R}: {json.dumps(dec[f'R{R}'])}", file=sys.stderr, flush=True)
        del run
    dev.resident_slot.copy_(slot_all)
    out["decode_T16"] = dec
    # prefill: all 64 resident, every slot a HIT
    T = wl.tokens
    run = LY.LayerRun(s, T, dev.C, tau=wl.tau)
    x = LY.to_tensor(synth.gen_x(wl, 0, 0, T), s.dtype, "cuda")
    conf = torch.from_numpy(synth.gen_conf(wl, 0, 0, T)).cuda()
    run.layer_gpu(dev, x, conf, T, to_host=False, resid=None, out=True)
    torch.cuda.synchronize()
    cls = run.slot_class.cpu().numpy()
    n_hit, n_lore = int((cls == 0).sum()), int((cls == 1).sum())
    flops = 6.0 * T * s.d * s.shared_inter + 6.0 * n_hit * s.d * s.inter + 4.0 * n_lore * s.d * s.lore_rank
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
            torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(6)]
    for a, b, c, d in evs:
        a.record()
        run.route(dev, x, conf, T, to_host=False)
        b.record()
        run.experts(dev, x, T)
        c.record()
        run.combine(None, T)
        d.record()
    torch.cuda.synchronize()
    layer_ms = float(np.median([a.elapsed_time(d) for a, b, c, d in evs]))
    ffn_ms = float(np.median([b.elapsed_time(c) for a, b, c, d in evs]))
    # the routing alone: average over back-to-back calls from one event pair (behind a spin
    # kernel, so that no span holds host submission time)
    reps = 30
    ra, rb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    torch.cuda._sleep(int(2e7))
    ra.record()
    for _ in range(reps):
        run.route(dev, x, conf, T, to_host=False)
    rb.record()
    torch.cuda.synchronize()
    route_ms = ra.elapsed_time(rb) / reps
    out["prefill_T4096"] = {
        "tokens": T, "resident": 64, "layer_ms": round(layer_ms, 3), "tokens_per_s": round(T / (layer_ms * 1e-3), 1),
        "route_us": round(route_ms * 1e3, 1), "ffn_ms": round(ffn_ms, 3), "flop_per_ffn_call": flops,
        "roofline": {"bound": "mfma", "kernel": "grouped expert FFN call: expert_gemm_kernel up + down",
                     "achieved": round(flops / (ffn_ms * 1e-3) / 1e12, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(flops / (ffn_ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)},
        "classes": np.bincount(cls.ravel(), minlength=3).tolist()}
    print(f"[bench] qwen2 prefill: {json.dumps(out['prefill_T4096'])}", file=sys.stderr, flush=True)
    if run.flags() != 0:
        raise RuntimeError("device flags raised in the Qwen2 records")
    return out


if __name__ == "__main__":
    main()
