"""Benchmark: one DiT block forward step on one MI355X.

Default workload: the 480x720x49f video request (13 x 30 x 45 latent grid +
226 text tokens = 17776 tokens), hidden 3072, 48 heads x 64, MLP 12288,
batch 1, under a 2 GiB activation budget (the plan runs it unchunked).
--workload picks another of the five block configurations, --budget or
--chunk another chunking.  Synthetic seeded inputs and random weights,
resident in HBM before timing starts.

Prints one JSON line: whole-step throughput (TFLOP/s of the block's
algorithmic FLOPs), ms per step, the roofline of the dominant kernel
(attention, timed on its own with HIP events on the launch stream) and the
fp64 CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_TFLOPS = 2500.0        # MI355X dense fp16/bf16 MFMA
PEAK_HBM_GBS = 8000.0


def attention_flops(B, H, L, d, q_count=None):
    q_count = L if q_count is None else q_count
    return 4 * B * H * q_count * L * d


# default activation budget per workload (arena bytes)
DEFAULT_BUDGET = {"tiny": 1 << 30, "image": 2 << 30, "image_b4": 2 << 30, "video": 2 << 30,
                  "highres": 32 * 10**9, "long": 8 << 30, "video_dual": 2 << 30}


def bench_gpu(args, shape):
    import numpy as np
    import torch

    import paper_2607_11136_amd as X
    import workloads as W

    dev = "cuda:0"
    torch.cuda.set_device(0)
    inp = W.make_inputs(shape)

    def up(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)

    x, cond = up(inp.x), up(inp.cond)
    w = {k: up(v) for k, v in inp.weights.items()}
    weights_f16 = 0 if args.bf16_weights else 1
    if weights_f16:
        # W_o, W_up, W_down in fp16, converted once per model as a serving
        # process would at load (the block then reads them directly)
        for k in ("o_w", "up_w", "down_w"):
            w[k] = w[k].to(torch.float16)
    weights = X.block_weights(w)
    cfg = X.block_cfg(shape.hidden, shape.heads, shape.head_dim, shape.mlp_hidden, shape.cond_dim,
                      shape.rope_dims, shape.rope_theta, shape.ln_eps, shape.qk_eps,
                      shape.modulation_streams, weights_f16)
    req = X.request(shape.batch, shape.text_len, *shape.grid)
    if args.chunk is not None:
        group = args.batch_group or shape.batch
        plan = X.xema_workspace_layout(cfg, X.request(min(group, shape.batch), shape.text_len, *shape.grid),
                                       args.chunk)
    elif args.batch_group:
        group = args.batch_group
        plan = X.xema_workspace_plan(cfg, X.request(group, shape.text_len, *shape.grid), args.budget)
    else:
        # chunking and temporary serialization, only as much as the budget needs
        group, plan = X.xema_workspace_plan_serial(cfg, req, args.budget)
    ws = torch.empty(plan.workspace_bytes, dtype=torch.uint8, device=dev)
    out = torch.empty((shape.batch, shape.seq_len, shape.hidden), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()

    # a chunked call runs each chunk's attention on a second stream, overlapping
    # the previous chunk's projections (bit-identical to one stream)
    aux = None if args.one_stream else torch.cuda.Stream()

    def step():
        X.xema_dit_block_fwd_pipelined(cfg, req, x, weights, cond, group, plan.chunk_tokens, ws, ws.numel(),
                                       out, stream, aux if aux is not None else stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(args.steps):
        step()
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / args.steps
    print(f"[bench] block step: {ms:.3f} ms over {args.steps} steps", file=sys.stderr, flush=True)

    # dominant kernel: attention over all queries, on the Q/K/V^T the block left in the arena
    # (which holds the sequences of one group when the batch runs in groups)
    B, H, L, d = min(group, shape.batch), shape.heads, shape.seq_len, shape.head_dim
    Lp = X.padded_len(L)
    slots = plan.slots()
    o = torch.empty((B * L, H * d), dtype=torch.float16, device=dev)
    base = ws.data_ptr()
    qp, kp, vp = (base + slots[n][0] for n in ("q", "k", "vt"))
    def attn():
        X.xema_op_attention(qp, kp, vp, B, H, d, L, Lp, 0, L, o, stream)
    for _ in range(2):
        attn()
    a0 = torch.cuda.Event(enable_timing=True)
    a1 = torch.cuda.Event(enable_timing=True)
    n_attn = max(3, args.steps)
    a0.record(stream)
    for _ in range(n_attn):
        attn()
    a1.record(stream)
    torch.cuda.synchronize()
    attn_ms = a0.elapsed_time(a1) / n_attn
    print(f"[bench] attention kernel: {attn_ms:.3f} ms per launch", file=sys.stderr, flush=True)
    if args.copy_bytes > 0:
        # a plain device-to-device copy of known size, so that HBM byte counters
        # read under a profiler can be scaled to bytes
        src = torch.ones(args.copy_bytes, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] copied {args.copy_bytes} bytes x 3", file=sys.stderr, flush=True)
    return {
        "ms": ms,
        "attn_ms": attn_ms,
        "plan": plan,
        "batch_group": group,
        "device_peak_bytes": int(torch.cuda.max_memory_allocated()),
        "weights_f16": weights_f16,
    }


def bench_step(args, shape):
    """N-block step with selective weight offloading: N blocks with distinct
    random weights, the plan's K offloaded blocks kept in pinned host memory
    and prefetched on a copy stream.  Prints one JSON line."""
    import torch

    import paper_2607_11136_amd as X

    dev = "cuda:0"
    torch.cuda.set_device(0)
    n = args.step_blocks
    cfg = X.block_cfg(shape.hidden, shape.heads, shape.head_dim, shape.mlp_hidden, shape.cond_dim,
                      shape.rope_dims, shape.rope_theta, shape.ln_eps, shape.qk_eps,
                      shape.modulation_streams)
    req = X.request(shape.batch, shape.text_len, *shape.grid)
    step_plan = None
    if args.device_budget is not None:
        # offloading, serialization and chunking chosen together under one
        # device budget (resident weights + the step's workspace)
        costs = X.step_costs(args.h2d_gbps, args.block_tflops)
        step_plan = X.xema_step_plan_budget(cfg, req, n, args.staging, args.device_budget, costs)
        plan = step_plan.offload
    elif args.weight_budget is not None:
        plan = X.xema_offload_plan_budget(cfg, n, args.weight_budget, args.staging)
    else:
        plan = X.xema_offload_plan_k(cfg, n, args.offload, args.staging)
    off = set(plan.offloaded_blocks())
    g = torch.Generator(device=dev).manual_seed(2607)
    shapes = shape.weight_shapes()

    def rand(shp, std, mean=0.0):
        return (torch.randn(shp, device=dev, generator=g) * std + mean).to(torch.bfloat16)

    blocks, keep = [], []
    for i in range(n):
        w = {}
        for name, shp in shapes.items():
            if name in ("q_gamma", "k_gamma"):
                t = rand(shp, 0.1, 1.0)
            else:
                t = rand(shp, 1.0 / shape.fan_in(name) ** 0.5)
            if i in off:
                h = torch.empty(t.shape, dtype=torch.bfloat16, pin_memory=True)
                h.copy_(t)
                t = h
            w[name] = t
        keep.append(w)
        blocks.append(X.block_weights(w))
    x = rand((shape.batch, shape.seq_len, shape.hidden), 1.0)
    cond = rand((shape.batch, shape.cond_dim), 1.0)
    nbytes = step_plan.workspace_bytes if step_plan else X.xema_step_workspace_bytes(cfg, req, 0, plan)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    out = torch.empty((shape.batch, shape.seq_len, shape.hidden), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    copy_stream = torch.cuda.Stream()
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()

    def step():
        if step_plan:
            X.xema_dit_step_fwd_planned(cfg, req, x, blocks, step_plan, cond, ws, nbytes, out, stream, copy_stream)
        else:
            X.xema_dit_step_fwd(cfg, req, x, blocks, plan, cond, 0, ws, nbytes, out, stream, copy_stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(args.steps):
        step()
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / args.steps
    # host-to-device rate of one block's weights alone (pinned, copy stream)
    h2d_gbs = None
    if off:
        hw = keep[min(off)]
        dst = {k: torch.empty_like(v, device=dev) for k, v in hw.items()}
        c0 = torch.cuda.Event(enable_timing=True)
        c1 = torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(copy_stream):
            c0.record(copy_stream)
            for k, v in hw.items():
                dst[k].copy_(v, non_blocking=True)
            c1.record(copy_stream)
        torch.cuda.synchronize()
        h2d_gbs = plan.block_weight_bytes / (c0.elapsed_time(c1) * 1e-3) / 1e9
    flops = n * shape.flops()
    result = {
        "metric": "DiT denoising step ms (N blocks, selective weight offloading)",
        "value": round(ms, 3),
        "unit": "ms",
        "higher_is_better": False,
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "tflops": round(flops / (ms * 1e-3) / 1e12, 1),
        "ms_per_block": round(ms / n, 3),
        "dtype": "f16/bf16",
        "data": "synthetic (random N(0,1) tokens and conditioning, N(0,1/fan_in) weights per block)",
        "config": {
            "workload": WORKLOAD_TEXT[args.workload], "n_blocks": n,
            "n_offloaded": plan.n_offloaded, "n_staging": plan.n_staging,
            "offloaded_blocks": sorted(off), "weight_budget_bytes": args.weight_budget,
            "block_weight_bytes": plan.block_weight_bytes,
            "device_weight_bytes": plan.device_weight_bytes,
            "h2d_bytes_per_step": plan.n_offloaded * plan.block_weight_bytes,
            "h2d_block_GBps": None if h2d_gbs is None else round(h2d_gbs, 1),
            "device_peak_bytes": int(torch.cuda.max_memory_allocated()),
            "workspace_bytes": nbytes,
        },
    }
    if step_plan:
        result["config"].update({"device_budget_bytes": args.device_budget, "batch_group": step_plan.batch_group,
                                 "chunk_tokens": step_plan.chunk_tokens, "device_bytes": step_plan.device_bytes,
                                 "est_ms": round(step_plan.est_ms, 3)})
    print(json.dumps(result), flush=True)


def bench_vae(args):
    """The VAE decoder's fused upsampling stage (nearest 2x + 3x3 conv) over a
    whole stage of frames, inputs resident in HBM.  Prints one JSON line."""
    import torch

    import paper_2607_11136_amd as X
    import workloads as W

    dev = "cuda:0"
    torch.cuda.set_device(0)
    s = W.VAE_CONFIGS[args.vae]
    g = torch.Generator(device=dev).manual_seed(2607)
    std = 1.0 / (9 * s.ci) ** 0.5
    x = torch.randn((s.n, s.h, s.w, s.ci), device=dev, generator=g).to(torch.bfloat16)
    w = (torch.randn((s.co, 3, 3, s.ci), device=dev, generator=g) * std).to(torch.bfloat16)
    b = (torch.randn((s.co,), device=dev, generator=g) * std).to(torch.bfloat16)
    wp = torch.empty(X.xema_vae_upconv_weight_bytes(s.ci, s.co) // 2, dtype=torch.bfloat16, device=dev)
    y = torch.empty((s.n, 2 * s.h, 2 * s.w, s.co), dtype=torch.bfloat16, device=dev)
    stream = torch.cuda.current_stream()
    X.xema_vae_upconv_prepare(w, s.ci, s.co, wp, stream)
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()

    def run():
        X.xema_vae_upconv(x, s.n, s.h, s.w, s.ci, wp, b, s.co, 0, s.h, y, stream)

    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(args.steps):
        run()
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / args.steps
    fused_peak = int(torch.cuda.max_memory_allocated())
    context = None
    if args.vae_torch_context:
        # the same stage unfused through PyTorch (nearest interpolate, then a
        # bf16 channels-last Conv2d), for context only
        xt = x.permute(0, 3, 1, 2)                     # NCHW view of the NHWC tensor
        wt = w.permute(0, 3, 1, 2).contiguous(memory_format=torch.channels_last)
        del y
        torch.cuda.synchronize()
        base = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()

        def unfused():
            u = torch.nn.functional.interpolate(xt, scale_factor=2, mode="nearest")
            return torch.nn.functional.conv2d(u, wt, b, padding=1)

        with torch.no_grad():
            for _ in range(2):
                yt = unfused()
            del yt
            torch.cuda.synchronize()
            c0 = torch.cuda.Event(enable_timing=True)
            c1 = torch.cuda.Event(enable_timing=True)
            c0.record(stream)
            for _ in range(3):
                yt = unfused()
                del yt
            c1.record(stream)
            torch.cuda.synchronize()
        context = {"torch_unfused_ms": round(c0.elapsed_time(c1) / 3, 3),
                   "torch_unfused_extra_peak_bytes": int(torch.cuda.max_memory_allocated() - base)}
    flops = s.flops()                      # the definition: 3x3 over the upsampled image
    mfma_flops = flops * 32 // 36          # what the phase form executes (hi and lo weights)
    up_bytes = s.n * 4 * s.h * s.w * s.ci * 2
    result = {
        "metric": "VAE upsampling stage ms (nearest 2x + 3x3 conv, fused)",
        "value": round(ms, 4),
        "unit": "ms",
        "higher_is_better": False,
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "tflops_definition": round(flops / (ms * 1e-3) / 1e12, 1),
        "dtype": "bf16",
        "data": "synthetic (random N(0,1) activations, N(0,1/(9 ci)) weights)",
        "config": {"workload": f"{s.name}: {s.n} frames {s.h}x{s.w} -> {2 * s.h}x{2 * s.w}, "
                               f"{s.ci} -> {s.co} channels",
                   "flops_definition": flops, "mfma_flops": mfma_flops,
                   "input_bytes": s.n * s.h * s.w * s.ci * 2, "output_bytes": s.n * 4 * s.h * s.w * s.co * 2,
                   "upsampled_bytes_not_stored": up_bytes,
                   "device_peak_bytes": fused_peak},
        "roofline": {"kernel": "k_upconv (four 2x2 phase convolutions, implicit GEMM)", "bound": "mfma",
                     "achieved": round(mfma_flops / (ms * 1e-3) / 1e12, 1), "peak": 2500.0, "unit": "TFLOP/s",
                     "frac": round(mfma_flops / (ms * 1e-3) / 1e12 / 2500.0, 4)},
    }
    if context:
        result["context"] = context
    print(json.dumps(result), flush=True)


TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "attention_video_hbm_traffic.md")
# the files the attention kernel is built from
TRAFFIC_SOURCES = ("paper_2607_11136_amd/csrc/k_attention.hip", "paper_2607_11136_amd/csrc/device_common.h",
                   "paper_2607_11136_amd/csrc/attention.h")


def attention_source_digest():
    import hashlib
    h = hashlib.sha256()
    for rel in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per attention launch from the committed counter summary, or
    None when it is missing or was taken on other kernel sources."""
    try:
        with open(TRAFFIC_RECORD) as f:
            line = next(l for l in f if l.startswith("record: "))
        rec = json.loads(line[len("record: "):])
    except (OSError, StopIteration, ValueError):
        return None
    if rec.get("source_sha256") != attention_source_digest():
        return None
    return int(rec["fetch_bytes"] + rec["write_bytes"])


def cpu_baseline(shape, n_rows):
    """The fp64 oracle on a bounded sample: K and V from all tokens (the oracle
    projects every token), outputs for `n_rows` sampled rows.  Rate is the
    algorithmic FLOPs of that sample per second; the per-step figure is
    extrapolated from it."""
    import numpy as np
    import workloads as W
    from oracle import block as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [os.cpu_count()])
    except Exception:  # threadpoolctl missing: numpy's BLAS uses every core
        threads = os.cpu_count()
    inp = W.make_inputs(shape)
    rows = W.sample_rows(shape, n_rows)
    t = time.perf_counter()
    O.block_forward_shape(inp, rows=rows)
    sec = time.perf_counter() - t
    B, L, D, F, Dc = shape.batch, shape.seq_len, shape.hidden, shape.mlp_hidden, shape.cond_dim
    R = len(rows)
    flops = 2 * B * Dc * 6 * D + 6 * B * L * D * D + B * R * (4 * L * D + 2 * D * D + 4 * D * F)
    rate = flops / sec
    return {
        "value": rate / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "kind": "oracle",
        "seconds": round(sec, 2),
        "ms_per_step_extrapolated": round(shape.flops() / rate * 1e3, 1),
        "sample": (f"{shape.name} block, fp64 numpy oracle: QKV of all {L} tokens plus attention, "
                   f"out-projection and MLP for {R} seeded rows ({flops / 1e12:.3f} TFLOP); "
                   f"per-step time extrapolated by FLOP count"),
    }


WORKLOAD_TEXT = {
    "tiny": "tiny DiT block: 32 text + 1x16x16 visual tokens (L=288), D=256, 4x64 heads, MLP 1024, batch 1",
    "image": "image DiT block 1024x1024: 512 text + 1x64x64 visual tokens (L=4608), D=3072, 24x128 heads, "
             "MLP 12288, batch 1",
    "image_b4": "image DiT block 1024x1024: 512 text + 1x64x64 visual tokens (L=4608), D=3072, 24x128 heads, "
                "MLP 12288, batch 4",
    "video": "video DiT block 480x720x49f: 226 text + 13x30x45 visual tokens (L=17776), D=3072, 48x64 heads, "
             "MLP 12288, batch 1",
    "highres": "high-res video DiT block 1080p x49f: 226 text + 13x68x120 visual tokens (L=106306), D=3072, "
               "48x64 heads, MLP 12288, batch 1",
    "long": "long video DiT block: 1024 text + 33x22x38 visual tokens (L=28612), D=4096, 32x128 heads, "
            "MLP 16384, batch 2",
    "video_dual": "video DiT block 480x720x49f with dual-stream modulation (text tokens' own AdaLN map): "
                  "226 text + 13x30x45 visual tokens (L=17776), D=3072, 48x64 heads, MLP 12288, batch 1",
}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="video", help="tiny, image, image_b4, video, highres, long or video_dual")
    ap.add_argument("--budget", type=int, default=None,
                    help="activation budget (arena bytes); default per workload, 2 GiB for video")
    ap.add_argument("--chunk", type=int, default=None, help="chunk_tokens instead of the planned one")
    ap.add_argument("--batch-group", type=int, default=None,
                    help="sequences per group (temporary serialization) instead of the planned one")
    ap.add_argument("--cpu-rows", type=int, default=3072)
    ap.add_argument("--step-blocks", type=int, default=0,
                    help="measure an N-block step with selective weight offloading instead")
    ap.add_argument("--offload", type=int, default=0, help="offloaded blocks K (step mode)")
    ap.add_argument("--weight-budget", type=int, default=None,
                    help="device weight budget in bytes; the plan picks the smallest K (step mode)")
    ap.add_argument("--staging", type=int, default=2, help="device staging slots (step mode)")
    ap.add_argument("--device-budget", type=int, default=None,
                    help="one device budget for resident weights and the step's workspace: the plan picks "
                         "offloading, batch groups and chunking together (step mode)")
    ap.add_argument("--h2d-gbps", type=float, default=56.0, help="copy rate the step plan's model assumes")
    ap.add_argument("--block-tflops", type=float, default=1000.0, help="block rate the step plan's model assumes")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--bf16-weights", action="store_true",
                    help="hand W_o, W_up, W_down over in bf16 (converted into the arena on every call) "
                         "instead of fp16 converted once")
    ap.add_argument("--one-stream", action="store_true",
                    help="run chunked phase B on one stream (no attention/projection overlap)")
    ap.add_argument("--vae", default=None, help="time the VAE upsampling stage vae_video or vae_1080p instead")
    ap.add_argument("--vae-torch-context", action="store_true",
                    help="with --vae, also time the stage unfused through PyTorch (context only)")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="also run a plain device copy of this size (calibrates HBM byte counters)")
    ap.add_argument("--print-digest", action="store_true",
                    help="print the digest of the attention kernel sources and exit")
    args = ap.parse_args()
    if args.print_digest:
        print(attention_source_digest())
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the block forward is measured on a single MI355X; "
              "sharding it across GPUs is not implemented", file=sys.stderr)
        sys.exit(2)

    if args.vae:
        bench_vae(args)
        return
    import workloads as W
    shape = W.CONFIGS[args.workload]
    if args.step_blocks > 0:
        bench_step(args, shape)
        return
    if args.budget is None:
        args.budget = DEFAULT_BUDGET[args.workload]
    g = bench_gpu(args, shape)
    flops = shape.flops()
    tflops = flops / (g["ms"] * 1e-3) / 1e12
    B, H, L, d = shape.batch, shape.heads, shape.seq_len, shape.head_dim
    af = attention_flops(min(g["batch_group"], B), H, L, d)
    attn_tflops = af / (g["attn_ms"] * 1e-3) / 1e12
    plan = g["plan"]
    result = {
        "metric": "DiT block ms/step + TFLOP/s (% bf16 MFMA peak) at fixed activation budget",
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(g["ms"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16/bf16",
        "data": "synthetic (seeded N(0,1) tokens and conditioning, N(0,1/fan_in) random weights)",
        "frac_peak": round(tflops / PEAK_TFLOPS, 4),
        "config": {
            "workload": WORKLOAD_TEXT[args.workload],
            "batch": B, "seq_len": L, "hidden": shape.hidden, "heads": H, "head_dim": d,
            "mlp_hidden": shape.mlp_hidden, "flops_per_step": flops,
            "budget_bytes": args.budget, "chunk_tokens": plan.chunk_tokens, "batch_group": g["batch_group"],
            "phase_b_streams": 1 if args.one_stream or plan.chunk_tokens >= shape.seq_len else 2,
            "arena_bytes": plan.workspace_bytes, "device_peak_bytes": g["device_peak_bytes"],
            "phase_b_weights": ("fp16, converted once per model" if g["weights_f16"]
                                else "bf16, converted to fp16 in every call"),
        },
        "roofline": {
            "kernel": (f"{'k_attention_lazy<64>' if d == 64 else 'k_attention<128>'} (joint attention, "
                       f"all {L} queries x {L} keys x {min(g['batch_group'], B) * H} batch-heads)"),
            "bound": "mfma",
            "achieved": round(attn_tflops, 2),
            "peak": PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(attn_tflops / PEAK_TFLOPS, 4),
            "ms_per_launch": round(g["attn_ms"], 4),
            "flops_per_launch": af,
            "traffic": measured_traffic() if args.workload == "video" else None,
        },
    }
    if not args.no_cpu_baseline and args.workload == "video":
        result["cpu_baseline"] = cpu_baseline(shape, args.cpu_rows)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
