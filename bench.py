"""Benchmark of the VideoMLA latent-attention hot path on one MI355X.

One step = one chunk-step of one Wan2.1-1.3B layer: `videomla_cache_write_prepared` of the
chunk's 4,680 tokens (3 frames of 30x52) into the 21-frame ring (weights packed once, at
setup), then `videomla_attend` of its 4,680 x 12 query rows over the 32,760-token window. Inputs are seeded synthetic tensors already resident
in HBM; the chunk's x cycles through 32 distinct buffers (460 MB) so that the cache write reads
x from HBM rather than from the 256 MB Infinity Cache.

Prints one JSON line: whole-step throughput in TFLOP/s of algorithmic work (write 688,128 FLOP
per token; attend 832 FLOP per query-head-key plus 98,304 per query-head for the two
projections), the per-kernel averages measured with HIP events on the library's stream, the
roofline of the dominant kernel and the CPU oracle's throughput on a bounded sample.
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_BF16_PEAK_TFLOPS = 2500.0   # MI355X published dense bf16 MFMA peak
HBM_PEAK_GBPS = 8000.0           # MI355X published HBM3E bandwidth

# HBM traffic of one latent_attend launch at this workload, from two rocprofv3 --pmc runs
# (FETCH_SIZE, WRITE_SIZE) scaled by the same counters on a plain copy of known size; valid only
# for the kernel source it was measured on (sha256 of the listed files), else reported as null.
ATTEND_TRAFFIC = {"sources": ("paper_2605_30351_amd/csrc/k_attend.hip",
                              "paper_2605_30351_amd/csrc/vmla_device.h",
                              "paper_2605_30351_amd/csrc/vmla_internal.h"),
                  "sha256": "a47ad6e1a56563d990164ba0c5ef2ddd24ccda38ab5361571a63f588d2140e4c",
                  "bytes": 307742817}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def work_model(d, batch=1):
    """Algorithmic FLOPs and bytes of one chunk-step."""
    nq = d.chunk_tokens
    S = d.window_tokens
    rows = batch * nq * d.n_heads
    per_score = 2 * (d.d_c + d.d_rope) + 2 * d.d_c             # QK over 224, PV over 192
    attend_core = rows * S * per_score
    attend_proj = rows * 2 * (d.d_nope * d.d_c + d.d_c * d.d_v)  # absorption + W_UV
    write_flop = batch * nq * 2 * d.d_model * (d.d_c + d.d_rope)
    write_bytes = (batch * nq * (2 * d.d_model + 2 * (d.d_c + d.d_rope))
                   + 2 * d.d_model * (d.d_c + d.d_rope))
    return {"attend_core": attend_core, "attend": attend_core + attend_proj,
            "write": write_flop, "write_bytes": write_bytes}


def cpu_baseline(d, n_rows=4680):
    """The fp64 oracle on the host: window latents from x, then reconstructed-K/V attention for
    a sample of query tokens (all heads). Credited with the algorithmic FLOPs of that sample."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import videomla_oracle as O
    from workloads import make_layer_inputs

    inp = make_layer_inputs(d, seed=1, n_frames=24)
    rows = np.linspace(0, d.chunk_tokens - 1, n_rows).astype(np.int64)
    t0 = time.perf_counter()
    O.chunk_attention(inp, 0, 21, rows=rows)
    dt = time.perf_counter() - t0
    per_score = 2 * (d.d_c + d.d_rope) + 2 * d.d_c
    flop = (n_rows * d.n_heads * (d.window_tokens * per_score + 2 * (d.d_nope * d.d_c + d.d_c * d.d_v))
            + d.chunk_tokens * 2 * d.d_model * (d.d_c + d.d_rope))
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {"value": flop / dt / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "seconds": dt,
            "sample": (f"fp64 numpy oracle: latents of the 32,760-token window from x, then "
                       f"explicit per-head K/V attention for {n_rows} of the 4,680 query tokens x 12 heads; "
                       f"credited with the method's algorithmic FLOPs of that sample plus the chunk's "
                       f"cache write; host has {len(os.sched_getaffinity(0))} usable cores")}


def extrapolated_oracle(d, flop):
    """The oracle's time for `flop` algorithmic FLOPs, extrapolated from one measured Wan
    chunk-step at the rate it sustains there (the oracle is dominated by fp64 matrix products,
    so its rate is about the same for every call of the workload)."""
    cb = cpu_baseline(d)
    return {"seconds": round(flop / (cb["value"] * 1e12), 1), "kind": "oracle",
            "cores": cb["cores"], "measured_chunk_step_s": round(cb["seconds"], 3),
            "note": ("extrapolated: the whole workload's algorithmic FLOPs divided by the rate "
                     "the fp64 oracle reaches on one measured Wan chunk-step (cache write + "
                     "attend of all 4,680 query tokens), not run end to end")}


def source_digest(paths):
    import hashlib
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def attend_traffic():
    """Measured HBM bytes per attend launch if the kernel is unchanged since the measurement."""
    if ATTEND_TRAFFIC["sha256"] is None:
        return None
    if source_digest(ATTEND_TRAFFIC["sources"]) != ATTEND_TRAFFIC["sha256"]:
        return None
    return ATTEND_TRAFFIC["bytes"]


def copy_probe(torch, dev, nbytes=1 << 28, reps=3):
    """A plain device copy of known size, whose FETCH_SIZE / WRITE_SIZE counters calibrate the
    counters of the library's kernels (each launch reads and writes nbytes)."""
    a = torch.ones(nbytes // 2, dtype=torch.bfloat16, device=dev)
    b = torch.empty_like(a)
    for _ in range(reps):
        b.copy_(a)
    torch.cuda.synchronize()
    del a, b


def timed_steps(vm, torch, step, n, names):
    """Milliseconds per step from n steps that carry no timing events, their per-step times,
    then per-kernel HIP-event averages ({name: {"launches", "avg_us"}}) from a second pass of n
    steps with every kernel bracketed (each event pair adds a few microseconds).

    step(i, timer) runs one step; the attention call passes `timer` (a videomla Timer or None)
    in its options, and the cache write is bracketed by the same timer's begin / end."""
    import numpy as np
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    marks[0].record()
    for i in range(n):
        step(i, None)
        marks[i + 1].record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    step_ms = np.array([marks[i].elapsed_time(marks[i + 1]) for i in range(n)])
    timer = vm.Timer()
    for i in range(n):
        step(i, timer)
    torch.cuda.synchronize()
    kernels = {}
    for k in names:
        c, tot = timer.read(k)
        kernels[k] = {"launches": c, "avg_us": round(1e3 * tot / max(c, 1), 3)}
    timer.close()
    return 1e3 * elapsed / n, step_ms, kernels


def bracket(timer, name, launch):
    """Run `launch` between timer.begin(name) and timer.end(name) on the current stream, or
    plainly when `timer` is None."""
    if timer is None:
        return launch()
    timer.begin(name)
    r = launch()
    timer.end(name)
    return r


def calibrate(vm, torch, call, n=3):
    """A few adaptive calls on the workspace the timed calls use: they set the per-XCD weights
    of the partition, which the timed (frozen) calls then reuse unchanged."""
    for _ in range(n):
        call(vm.AttendOpts(partition="adaptive"))
    torch.cuda.synchronize()


def thirty_layer_chunk(args, vm, torch, d, n_layers=30, n_steps=4):
    """One chunk through the whole network's attention layers: for each of 4 denoising steps,
    every one of the 30 layers (own weights, own ring, filled with frames 0..20) writes the
    chunk's latents and attends over its window; then the window advances. Activations and
    weights are seeded synthetic bf16 drawn on the GPU (N(0,1) activations, N(0, 1/fan_in)
    weights); `steps` counts chunks."""
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(3)

    def normal(shape, std=1.0):
        return (torch.randn(shape, generator=g, device=dev) * std).to(torch.bfloat16)

    hw, nq = d.hw, d.chunk_tokens
    log(f"building {n_layers} layers")
    layers = []
    for _ in range(n_layers):
        L = {
            "w_dkv": normal((d.d_c, d.d_model), d.d_model ** -0.5),
            "w_kr": normal((d.d_rope, d.d_model), d.d_model ** -0.5),
            "w_uk": normal((d.n_heads * d.d_nope, d.d_c), d.d_c ** -0.5),
            "w_uv": normal((d.n_heads * d.d_v, d.d_c), d.d_c ** -0.5),
            "gamma": torch.ones(d.d_c, dtype=torch.bfloat16, device=dev),
            "x": normal((1, nq, d.d_model)),
            "q_nope": normal((1, nq, d.n_heads, d.d_nope)),
            "q_r": normal((1, nq, d.n_heads, d.d_rope)),
            "c_kv": torch.zeros((1, d.window_tokens, d.d_c), dtype=torch.bfloat16, device=dev),
            "k_r": torch.zeros((1, d.window_tokens, d.d_rope), dtype=torch.bfloat16, device=dev),
        }
        L["w_packed"] = torch.empty(vm.write_weights_bytes(d), dtype=torch.uint8, device=dev)
        vm.prepare_write_weights(d, L["w_dkv"], L["w_kr"], L["w_packed"])
        for fe in range(0, d.window_frames, d.chunk_frames):  # frames 0..20 in the ring
            vm.cache_write_prepared(d, fe, 1, normal((1, nq, d.d_model)), L["w_packed"],
                                    L["gamma"], L["c_kv"], L["k_r"])
        layers.append(L)
    out = torch.empty((1, nq, d.n_heads, d.d_v), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(vm.attend_workspace_bytes(d, 1), dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()

    frame = [d.window_frames]  # the chunk being generated: frames 21..23, then 24..26, ...
    opts = vm.AttendOpts(partition=args.partition)

    def chunk():
        fe = frame[0]
        for _ in range(n_steps):
            for L in layers:
                vm.cache_write_prepared(d, fe, 1, L["x"], L["w_packed"], L["gamma"], L["c_kv"],
                                        L["k_r"])
                vm.attend(d, fe, 1, L["q_nope"], L["q_r"], L["w_uk"], L["w_uv"], L["c_kv"],
                          L["k_r"], out, ws, opts=opts)
        frame[0] = vm.window_advance(d, fe)

    if args.partition == "frozen":
        L = layers[0]
        calibrate(vm, torch, lambda o: vm.attend(d, frame[0], 1, L["q_nope"], L["q_r"], L["w_uk"],
                                                 L["w_uv"], L["c_kv"], L["k_r"], out, ws, opts=o))

    n_warm, n_time = max(1, min(args.warmup, 3)), max(1, min(args.steps, 10))
    log(f"warmup {n_warm} chunks, timing {n_time}")
    for _ in range(n_warm):
        chunk()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n_time + 1)]
    ev[0].record()
    for i in range(n_time):
        chunk()
        ev[i + 1].record()
    torch.cuda.synchronize()
    ms = [ev[i].elapsed_time(ev[i + 1]) for i in range(n_time)]
    W = work_model(d)
    flop = n_layers * n_steps * (W["attend"] + W["write"])
    latent = n_layers * d.window_tokens * vm.cache_bytes_per_token(d)
    # the dense per-head cache the latent one replaces: K and V of 12 heads x 128 per token
    dense = n_layers * d.window_tokens * d.n_heads * 2 * d.d_v * 2
    mean = sum(ms) / len(ms)
    extra = {}
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle, one chunk-step)")
        extra["cpu_baseline_extrapolated"] = extrapolated_oracle(d, flop)
    print(json.dumps({
        "metric": "ms per chunk: 30 layers x 4 denoising steps of cache write + latent attend",
        **extra,
        "value": round(mean, 3), "unit": "ms", "n_gpus": 1, "steps": n_time, "warmup": n_warm,
        "higher_is_better": False, "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "ms_per_chunk_min_max": [round(min(ms), 3), round(max(ms), 3)],
        "tflops": round(flop / (mean / 1e3) / 1e12, 2),
        "latent_cache_bytes": latent, "dense_cache_bytes_same_window": dense,
        "config": {"workload": ("Wan2.1-1.3B, one 3-frame chunk (4,680 tokens x 12 heads) "
                                "through 30 attention layers x 4 denoising steps over a "
                                "32,760-token 21-frame window each, then the window advance"),
                   "layers": n_layers, "denoising_steps": n_steps, "seed": 3,
                   "attend_partition": args.partition},
    }), flush=True)


def sink_chunk_step(args, vm, torch, d, fe=237):
    """One chunk-step with the paper's long-rollout context: one sink frame and the six most
    recent frames (10,920 keys), late in a rollout (the chunk of frames 237..239, context frames
    0 and 234..239), batch 1. The ring holds unrotated keys; the step is the cache write of the
    chunk, then the attend call, which also rotates the context's keys at window-local time.
    Seeded synthetic bf16 drawn on the GPU; the chunk's x cycles through 32 buffers (460 MB)."""
    import numpy as np
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(9)

    def normal(shape, std=1.0):
        return (torch.randn(shape, generator=g, device=dev) * std).to(torch.bfloat16)

    nq = d.chunk_tokens
    w_dkv = normal((d.d_c, d.d_model), d.d_model ** -0.5)
    w_kr = normal((d.d_rope, d.d_model), d.d_model ** -0.5)
    w_uk = normal((d.n_heads * d.d_nope, d.d_c), d.d_c ** -0.5)
    w_uv = normal((d.n_heads * d.d_v, d.d_c), d.d_c ** -0.5)
    gamma = torch.ones(d.d_c, dtype=torch.bfloat16, device=dev)
    q_nope, q_r = normal((1, nq, d.n_heads, d.d_nope)), normal((1, nq, d.n_heads, d.d_rope))
    c_kv = torch.zeros((1, d.window_tokens, d.d_c), dtype=torch.bfloat16, device=dev)
    k_r = torch.zeros((1, d.window_tokens, d.d_rope), dtype=torch.bfloat16, device=dev)
    out = torch.empty((1, nq, d.n_heads, d.d_v), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(vm.attend_workspace_bytes(d, 1), dtype=torch.uint8, device=dev)
    w_packed = torch.empty(vm.write_weights_bytes(d), dtype=torch.uint8, device=dev)
    vm.prepare_write_weights(d, w_dkv, w_kr, w_packed)
    for f in (0, fe - 6, fe - 3):  # the sink (first chunk) and the recent frames before fe
        vm.cache_write_prepared(d, f, 1, normal((1, nq, d.d_model)), w_packed, gamma, c_kv, k_r)
    xs = [normal((1, nq, d.d_model)) for _ in range(args.x_buffers)]
    torch.cuda.synchronize()

    def attend(o):
        vm.attend(d, fe, 1, q_nope, q_r, w_uk, w_uv, c_kv, k_r, out, ws, opts=o)

    def step(i, timer=None):
        bracket(timer, "cache_write", lambda: vm.cache_write_prepared(d, fe, 1, xs[i % len(xs)], w_packed,
                                                            gamma, c_kv, k_r))
        attend(vm.AttendOpts(partition=args.partition, timer=timer))

    for i in range(args.warmup):
        step(i)
    if args.partition == "frozen":
        calibrate(vm, torch, attend)
    torch.cuda.synchronize()
    names = ("cache_write", "q_absorb", "rope_window", "latent_attend", "latent_merge", "out_proj")
    ms, step_ms, kernels = timed_steps(vm, torch, step, args.steps, names)
    S = vm.valid_tokens(d, fe)
    rows = nq * d.n_heads
    attend_core = rows * S * (2 * (d.d_c + d.d_rope) + 2 * d.d_c)
    attend_flop = attend_core + rows * 2 * (d.d_nope * d.d_c + d.d_c * d.d_v)
    write_flop = nq * 2 * d.d_model * (d.d_c + d.d_rope)
    k3 = kernels["latent_attend"]["avg_us"] / 1e6
    print(json.dumps({
        "metric": "ms/chunk-step & TFLOP/s, sink frame + 6-frame local window (window-local RoPE)",
        "value": round((attend_flop + write_flop) / (ms / 1e3) / 1e12, 2), "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "step_ms_p10_p50_p90": [round(float(np.percentile(step_ms, q)), 4) for q in (10, 50, 90)],
        "higher_is_better": True, "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "kernels": kernels,
        "latent_attend_tflops": round(attend_core / k3 / 1e12, 2),
        "latent_attend_mfma_frac": round(attend_core / k3 / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
        "config": {"workload": (f"Wan2.1-1.3B layer chunk-step late in a rollout (frames "
                                f"{fe}..{fe + 2}): cache write of 4,680 tokens + latent attend "
                                f"of 4,680 x 12 query rows over {S:,} keys (1 sink frame + 6 "
                                "recent frames), batch 1"),
                   "sink_frames": d.sink_frames, "window_frames": d.window_frames,
                   "window_tokens": S, "seed": 9, "attend_partition": args.partition},
    }), flush=True)


def full_layer_chunk_step(args, vm, torch, d, d_q=768, fe=21):
    """One chunk-step of the whole attention layer in latent form: the cache write of the chunk
    (frames 21..23, evicting 0..2), then videomla_attend_layer from the chunk's attention input x
    to the output of W_O (query latent, absorbed queries, latent attention over the 32,760-key
    window, value/output absorption), batch 1, d_q = 768. Weights are packed once before the
    timed region. Seeded synthetic bf16 drawn on the GPU; x cycles through 32 buffers."""
    import numpy as np
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(12)

    def normal(shape, std=1.0):
        return (torch.randn(shape, generator=g, device=dev) * std).to(torch.bfloat16)

    nq, H = d.chunk_tokens, d.n_heads
    w_dkv = normal((d.d_c, d.d_model), d.d_model ** -0.5)
    w_kr = normal((d.d_rope, d.d_model), d.d_model ** -0.5)
    gamma = torch.ones(d.d_c, dtype=torch.bfloat16, device=dev)
    weights = torch.empty(vm.layer_weights_bytes(d, d_q), dtype=torch.uint8, device=dev)
    vm.prepare_layer_weights(
        d, d_q, normal((d_q, d.d_model), d.d_model ** -0.5),
        torch.ones(d_q, dtype=torch.bfloat16, device=dev),
        normal((H * d.d_nope, d_q), d_q ** -0.5), normal((H * d.d_rope, d_q), d_q ** -0.5),
        normal((H * d.d_nope, d.d_c), d.d_c ** -0.5), normal((H * d.d_v, d.d_c), d.d_c ** -0.5),
        normal((d.d_model, H * d.d_v), (H * d.d_v) ** -0.5), weights)
    c_kv = torch.zeros((1, d.window_tokens, d.d_c), dtype=torch.bfloat16, device=dev)
    k_r = torch.zeros((1, d.window_tokens, d.d_rope), dtype=torch.bfloat16, device=dev)
    y = torch.empty((1, nq, d.d_model), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(vm.attend_layer_workspace_bytes(d, d_q, 1), dtype=torch.uint8, device=dev)
    w_packed = torch.empty(vm.write_weights_bytes(d), dtype=torch.uint8, device=dev)
    vm.prepare_write_weights(d, w_dkv, w_kr, w_packed)
    for f in range(0, fe, d.chunk_frames):
        vm.cache_write_prepared(d, f, 1, normal((1, nq, d.d_model)), w_packed, gamma, c_kv, k_r)
    xs = [normal((1, nq, d.d_model)) for _ in range(args.x_buffers)]
    torch.cuda.synchronize()

    def layer(o, x=None):
        vm.attend_layer(d, fe, 1, d_q, xs[0] if x is None else x, weights, c_kv, k_r, y, ws,
                        opts=o)

    def step(i, timer=None):
        x = xs[i % len(xs)]
        bracket(timer, "cache_write", lambda: vm.cache_write_prepared(d, fe, 1, x, w_packed, gamma, c_kv,
                                                            k_r))
        layer(vm.AttendOpts(partition=args.partition, timer=timer), x)

    for i in range(args.warmup):
        step(i)
    if args.partition == "frozen":
        calibrate(vm, torch, layer)
    torch.cuda.synchronize()
    names = ("cache_write", "q_down", "q_up", "latent_attend", "latent_merge", "out_mix")
    ms, step_ms, kernels = timed_steps(vm, torch, step, args.steps, names)
    S = d.window_tokens
    rows = nq * H
    flop = {"cache_write": nq * 2 * d.d_model * (d.d_c + d.d_rope),
            "q_down": nq * 2 * d.d_model * d_q,
            "q_up": nq * 2 * d_q * H * (d.d_c + d.d_rope),
            "latent_attend": rows * S * (2 * (d.d_c + d.d_rope) + 2 * d.d_c),
            "out_mix": nq * 2 * H * d.d_c * d.d_model}
    for k, f in flop.items():
        kernels[k]["tflops"] = round(f / (kernels[k]["avg_us"] / 1e6) / 1e12, 1)
    print(json.dumps({
        "metric": "ms/chunk-step & TFLOP/s, whole attention layer in latent form (x -> W_O output)",
        "value": round(sum(flop.values()) / (ms / 1e3) / 1e12, 2), "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "step_ms_p10_p50_p90": [round(float(np.percentile(step_ms, q)), 4) for q in (10, 50, 90)],
        "higher_is_better": True, "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "kernels": kernels,
        "config": {"workload": ("Wan2.1-1.3B attention layer chunk-step, latent form: cache write "
                                "of 4,680 tokens, then c^Q = RMSNorm(W_DQ x) (d_q = 768), "
                                "absorbed queries, latent attend over 32,760 keys x 12 heads, "
                                "y = sum_h B_h o_lat_h; batch 1"),
                   "d_q": d_q, "seed": 12, "attend_partition": args.partition},
    }), flush=True)


def rollout_comparison(args, vm, torch, d, batch=4, n_layers=30, n_steps=4):
    """Minute-scale rollout at batch 4: `--chunks` consecutive 3-frame chunks (80 = frames
    0..239, temporal RoPE index up to 239, the ring wrapping eleven times) through 30 attention
    layers x 4 denoising steps, each layer with its own weights, queries and ring; the window
    advances after every chunk. Run once with the latent path (cache write + latent attend) and
    once with the dense per-head comparator (per-head K/V cache write + standard attention) on
    the same schedule, shapes and activations. Seeded synthetic bf16 drawn on the GPU; chunk
    activations cycle through 8 distinct buffers (460 MB) so that each call reads them from
    HBM. Per-kernel averages are taken with HIP events over the last chunk (full window)."""
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(4)

    def normal(shape, std=1.0):
        return (torch.randn(shape, generator=g, device=dev) * std).to(torch.bfloat16)

    nq, B = d.chunk_tokens, batch
    n_chunks = args.chunks
    xs = [normal((B, nq, d.d_model)) for _ in range(8)]

    def x_of(c, s, li):
        return xs[(c * n_steps * n_layers + s * n_layers + li) % len(xs)]

    def run(path):
        log(f"{path}: building {n_layers} layers at batch {B}")
        layers = []
        for _ in range(n_layers):
            if path == "latent":
                L = {"w_dkv": normal((d.d_c, d.d_model), d.d_model ** -0.5),
                     "w_kr": normal((d.d_rope, d.d_model), d.d_model ** -0.5),
                     "w_uk": normal((d.n_heads * d.d_nope, d.d_c), d.d_c ** -0.5),
                     "w_uv": normal((d.n_heads * d.d_v, d.d_c), d.d_c ** -0.5),
                     "gamma": torch.ones(d.d_c, dtype=torch.bfloat16, device=dev),
                     "q_nope": normal((B, nq, d.n_heads, d.d_nope)),
                     "q_r": normal((B, nq, d.n_heads, d.d_rope)),
                     "c_kv": torch.zeros((B, d.window_tokens, d.d_c), dtype=torch.bfloat16,
                                         device=dev),
                     "k_r": torch.zeros((B, d.window_tokens, d.d_rope), dtype=torch.bfloat16,
                                        device=dev)}
                L["w_packed"] = torch.empty(vm.write_weights_bytes(d), dtype=torch.uint8,
                                            device=dev)
                vm.prepare_write_weights(d, L["w_dkv"], L["w_kr"], L["w_packed"])
            else:
                L = {"w_k": normal((d.n_heads * d.d_v, d.d_model), d.d_model ** -0.5),
                     "w_v": normal((d.n_heads * d.d_v, d.d_model), d.d_model ** -0.5),
                     "q": normal((B, nq, d.n_heads, d.d_v)),
                     "kv": torch.zeros((B, d.window_tokens, d.n_heads, 2 * d.d_v),
                                       dtype=torch.bfloat16, device=dev)}
            layers.append(L)
        out = torch.empty((B, nq, d.n_heads, d.d_v), dtype=torch.bfloat16, device=dev)
        if path == "latent":
            ws = torch.empty(vm.attend_workspace_bytes(d, B), dtype=torch.uint8, device=dev)
            names = ("cache_write", "q_absorb", "latent_attend", "latent_merge", "out_proj")
        else:
            ws = torch.empty(vm.dense_attend_workspace_bytes(d, B), dtype=torch.uint8, device=dev)
            names = ("dense_cache_write", "dense_q_prep", "dense_attend", "dense_merge")

        def call(L, fe, x, part, timer=None):
            o = vm.AttendOpts(partition=part, timer=timer)
            if path == "latent":
                bracket(timer, "cache_write", lambda: vm.cache_write_prepared(
                    d, fe, B, x, L["w_packed"], L["gamma"], L["c_kv"], L["k_r"]))
                vm.attend(d, fe, B, L["q_nope"], L["q_r"], L["w_uk"], L["w_uv"], L["c_kv"],
                          L["k_r"], out, ws, opts=o)
            else:
                bracket(timer, "dense_cache_write", lambda: vm.dense_cache_write(
                    d, fe, B, x, L["w_k"], L["w_v"], L["kv"]))
                vm.dense_attend(d, fe, B, L["q"], L["kv"], out, ws, opts=o)

        # warm-up: one chunk-step of every layer at frame 0 (rewritten by chunk 0 below); with
        # the frozen partition, adaptive calls at the full window first set its weights
        if args.partition == "frozen":
            for li in range(3):
                call(layers[li], d.window_frames, x_of(0, 0, li), "adaptive")
        for li, L in enumerate(layers):
            call(L, 0, x_of(0, 0, li), args.partition)
        torch.cuda.synchronize()
        log(f"{path}: timing {n_chunks} chunks")
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(n_chunks + 1)]
        fe = 0
        t0 = time.perf_counter()
        ev[0].record()
        timer = None
        for c in range(n_chunks):
            if c == n_chunks - 1:
                torch.cuda.synchronize()
                timer = vm.Timer()
            for s in range(n_steps):
                for li, L in enumerate(layers):
                    call(L, fe, x_of(c, s, li), args.partition, timer)
            ev[c + 1].record()
            fe = vm.window_advance(d, fe)
            if c % 10 == 9:
                log(f"{path}: chunk {c + 1}/{n_chunks}")
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        kern = {}
        for k in names:
            n, tot = timer.read(k)
            kern[k] = {"launches": n, "avg_us": round(1e3 * tot / max(n, 1), 2)}
        timer.close()
        ms = [ev[i].elapsed_time(ev[i + 1]) for i in range(n_chunks)]
        full = ms[(d.window_frames - 1) // d.chunk_frames:] or ms
        del layers, out, ws
        torch.cuda.empty_cache()
        return {"seconds": round(wall, 3), "ms_per_chunk": round(sum(ms) / len(ms), 3),
                "ms_per_chunk_full_window": round(sum(full) / len(full), 3),
                "ms_first_chunk": round(ms[0], 3), "kernels_last_chunk": kern}

    lat = run("latent")
    den = run("dense")
    # the vendor GEMM library (torch.matmul) on each path's bare cache projection at this batch,
    # x [B Nq, d_model] @ [W_DKV; W_KR]^T or [W_K; W_V]^T: the dense comparator's cache write at
    # the library's rate, for the comparison below
    filler_a, filler_b = normal((8192, 8192)), normal((8192, 8192))
    x2 = [xs[i].view(B * nq, d.d_model) for i in range(len(xs))]
    lib_proj = {}
    for name, n_out in (("latent", d.d_c + d.d_rope), ("dense", 2 * d.n_heads * d.d_v)):
        w_t = normal((d.d_model, n_out), d.d_model ** -0.5)
        y = torch.empty((B * nq, n_out), dtype=torch.bfloat16, device=dev)
        avg, _ = event_timed(torch, lambda i: torch.matmul(x2[i % len(x2)], w_t, out=y),
                             lambda: torch.matmul(filler_a, filler_b))
        lib_proj[name] = round(avg, 2)
        del w_t, y
    del filler_a, filler_b
    if args.copy_probe:
        log("copy probe")
        copy_probe(torch, dev)
    # algorithmic work of the whole rollout (valid window per chunk)
    lat_flop = den_flop = 0
    fe = 0
    for c in range(n_chunks):
        S = vm.valid_tokens(d, fe)
        rows = B * nq * d.n_heads
        lat_flop += n_layers * n_steps * (
            rows * S * (2 * (d.d_c + d.d_rope) + 2 * d.d_c)
            + rows * 2 * (d.d_nope * d.d_c + d.d_c * d.d_v)
            + B * nq * 2 * d.d_model * (d.d_c + d.d_rope))
        den_flop += n_layers * n_steps * (rows * S * 4 * d.d_v
                                          + B * nq * 2 * d.d_model * 2 * d.n_heads * d.d_v)
        fe = vm.window_advance(d, fe)
    lat["tflops"] = round(lat_flop / lat["seconds"] / 1e12, 2)
    den["tflops"] = round(den_flop / den["seconds"] / 1e12, 2)
    lat_bytes = n_layers * B * d.window_tokens * vm.cache_bytes_per_token(d)
    den_bytes = n_layers * B * d.window_tokens * vm.dense_cache_bytes_per_token(d)
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle, one chunk-step)")
        lat["cpu_baseline_extrapolated"] = extrapolated_oracle(d, lat_flop)
    la, da = lat["kernels_last_chunk"], den["kernels_last_chunk"]
    lat_call = sum(v["avg_us"] for v in la.values())
    den_call = sum(v["avg_us"] for v in da.values())
    # the attention kernels at the full window: their MFMA fractions, and the latent/dense time
    # ratio they would have at equal MFMA efficiency (the ratio of their algorithmic FLOPs)
    S_full = d.window_tokens
    rows_full = B * nq * d.n_heads
    lat_att_flop = rows_full * S_full * (2 * (d.d_c + d.d_rope) + 2 * d.d_c)
    den_att_flop = rows_full * S_full * 4 * d.d_v
    eff = {"latent_attend_mfma_frac": round(lat_att_flop / (la["latent_attend"]["avg_us"] / 1e6)
                                            / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
           "dense_attend_mfma_frac": round(den_att_flop / (da["dense_attend"]["avg_us"] / 1e6)
                                           / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
           "attention_time_ratio_at_equal_mfma_efficiency": round(lat_att_flop / den_att_flop, 4),
           "attention_time_ratio_measured": round(la["latent_attend"]["avg_us"]
                                                  / da["dense_attend"]["avg_us"], 4)}
    print(json.dumps({
        "metric": "ms per chunk: 30 layers x 4 denoising steps, latent vs dense per-head cache",
        "value": lat["ms_per_chunk"], "unit": "ms", "n_gpus": 1, "steps": n_chunks, "warmup": 1,
        "higher_is_better": False, "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "latent": lat, "dense": den,
        "latent_over_dense_time": round(lat["seconds"] / den["seconds"], 3),
        "latent_over_dense_time_per_call_full_window": round(lat_call / den_call, 3),
        "attention_kernels_full_window": eff,
        "library_projection_us": lib_proj,
        "latent_over_dense_per_call_full_window_dense_write_at_library_rate": round(
            lat_call / (den_call - da["dense_cache_write"]["avg_us"] + lib_proj["dense"]), 3),
        "cache_bytes": {"latent": lat_bytes, "dense": den_bytes,
                        "dense_over_latent": round(den_bytes / lat_bytes, 3)},
        "config": {"workload": (f"Wan2.1-1.3B rollout, batch 4: {n_chunks} chunks of 3 frames "
                                f"(frames 0..{3 * n_chunks - 1}) x 30 layers x 4 denoising "
                                "steps, 21-frame window; latent path and dense per-head "
                                "comparator on the same schedule"),
                   "batch": B, "layers": n_layers, "denoising_steps": n_steps,
                   "chunks": n_chunks, "seed": 4, "attend_partition": args.partition},
    }), flush=True)


def chunk_step_kernels(vm, torch, d, batch, steps, warmup, seed, x_buffers=8,
                       materialized=False, partition="frozen"):
    """Per-kernel HIP-event averages of `steps` chunk-steps (packed cache write + attend) of
    one layer with dims d at the wrapped full window (chunk at frame window_frames), batch
    `batch`; the attend is the latent form, or the materialized-K/V form when `materialized`.
    Seeded synthetic bf16 drawn on the GPU; x cycles through `x_buffers` buffers."""
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(seed)

    def normal(shape, std=1.0):
        return (torch.randn(shape, generator=g, device=dev) * std).to(torch.bfloat16)

    nq, B = d.chunk_tokens, batch
    w_dkv = normal((d.d_c, d.d_model), d.d_model ** -0.5)
    w_kr = normal((d.d_rope, d.d_model), d.d_model ** -0.5)
    w_uk = normal((d.n_heads * d.d_nope, d.d_c), d.d_c ** -0.5)
    w_uv = normal((d.n_heads * d.d_v, d.d_c), d.d_c ** -0.5)
    gamma = torch.ones(d.d_c, dtype=torch.bfloat16, device=dev)
    q_nope, q_r = normal((B, nq, d.n_heads, d.d_nope)), normal((B, nq, d.n_heads, d.d_rope))
    c_kv = torch.zeros((B, d.window_tokens, d.d_c), dtype=torch.bfloat16, device=dev)
    k_r = torch.zeros((B, d.window_tokens, d.d_rope), dtype=torch.bfloat16, device=dev)
    out = torch.empty((B, nq, d.n_heads, d.d_v), dtype=torch.bfloat16, device=dev)
    form = "materialized" if materialized else "latent"
    ws = torch.empty(vm.attend_workspace_bytes(d, B, vm.AttendOpts(form=form)), dtype=torch.uint8,
                     device=dev)
    w_packed = torch.empty(vm.write_weights_bytes(d), dtype=torch.uint8, device=dev)
    vm.prepare_write_weights(d, w_dkv, w_kr, w_packed)
    for f in range(0, d.window_frames, d.chunk_frames):
        vm.cache_write_prepared(d, f, B, normal((B, nq, d.d_model)), w_packed, gamma, c_kv, k_r)
    fe = d.window_frames
    xs = [normal((B, nq, d.d_model)) for _ in range(x_buffers)]
    torch.cuda.synchronize()

    def attend(o):
        vm.attend(d, fe, B, q_nope, q_r, w_uk, w_uv, c_kv, k_r, out, ws, opts=o)

    def step(i, timer=None):
        bracket(timer, "cache_write", lambda: vm.cache_write_prepared(d, fe, B, xs[i % len(xs)], w_packed,
                                                            gamma, c_kv, k_r))
        attend(vm.AttendOpts(partition=partition, form=form, timer=timer))

    for i in range(warmup):
        step(i)
    if partition == "frozen":
        calibrate(vm, torch, lambda o: attend(dataclasses.replace(o, form=form)))
    torch.cuda.synchronize()
    names = (("cache_write", "mat_kv", "mat_q_prep", "mat_attend", "mat_merge") if materialized
             else ("cache_write", "q_absorb", "latent_attend", "latent_merge", "out_proj"))
    ms, _, kernels = timed_steps(vm, torch, step, steps, names)
    return ms, {k: v["avg_us"] for k, v in kernels.items()}


def latent_vs_materialized(args, vm, torch):
    """The two exact forms of the attention at Wan geometry (3-frame chunk of 4,680 x 12 query
    rows over the wrapped 32,760-key window, batch 1, d_c 192), for both head splits: the
    paper's d_nope 96 + d_rope 32 and the measured configuration's 128 + 32. Latent form:
    absorbed queries, 2 d_c + d_rope = 416 multiply-adds per score. Materialized form: per-head
    K_h, V_h reconstructed for the window each call, then d_nope + d_rope + d_v = 256 or 288
    per score. Each step also writes the chunk's latents (packed cache write)."""
    from workloads import WAN, WAN_PAPER
    steps = max(10, args.steps // 2)
    out = {}
    for label, d in (("d_nope 96 (paper)", WAN_PAPER), ("d_nope 128", WAN)):
        res = {}
        for name, mat in (("latent", False), ("materialized", True)):
            log(f"{label}: {name}")
            ms, k = chunk_step_kernels(vm, torch, d, 1, steps, args.warmup, seed=52, materialized=mat,
                                       partition=args.partition)
            res[name] = {"ms_per_step": round(ms, 4), "kernels_us": k}
        rows = d.chunk_tokens * d.n_heads
        flop_lat = rows * d.window_tokens * 2 * (2 * d.d_c + d.d_rope)
        flop_mat = rows * d.window_tokens * 2 * (d.d_nope + d.d_rope + d.d_v)
        res["latent"]["attention_kernel_tflops"] = round(flop_lat / (res["latent"]["kernels_us"]["latent_attend"] / 1e6) / 1e12, 1)
        res["materialized"]["attention_kernel_tflops"] = round(flop_mat / (res["materialized"]["kernels_us"]["mat_attend"] / 1e6) / 1e12, 1)
        att = {n: round(sum(v for k2, v in res[n]["kernels_us"].items() if k2 != "cache_write"), 2)
               for n in res}
        out[label] = {**res, "attend_us": att, "materialized_over_latent": round(att["materialized"] / att["latent"], 4)}
    print(json.dumps({
        "metric": "attend us per call: latent form vs materialized per-head K/V",
        "value": out["d_nope 128"]["materialized_over_latent"], "unit": "materialized / latent attend time (d_nope 128)",
        "n_gpus": 1, "higher_is_better": False, "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic", "results": out,
        "config": {"workload": ("Wan2.1-1.3B geometry, d_c 192, d_rope 32, d_nope 96 and 128: "
                                "chunk of 3 frames (4,680 x 12 query rows) over the wrapped "
                                "32,760-key window, batch 1")},
    }), flush=True)


def dc_sweep(args, vm, torch, d0):
    """The paper's latent-width sweep (Table 5) at Wan geometry: one chunk-step (packed cache
    write + attend of 4,680 x 12 query rows over the 32,760-key window) per d_c, batch 1, and
    the few-query regime (1-frame chunks: 1,560 x 12 rows) at d_c = 192."""
    from workloads import DC_SWEEP, WAN_1F
    rows = []
    for dc in DC_SWEEP:
        d = d0.replace(d_c=dc)
        entry = {"d_c": dc, "cache_bytes_per_token": 2 * (dc + d.d_rope),
                 "vs_dense_cache": round(2 * d.n_heads * d.d_v / (dc + d.d_rope), 2)}
        if vm.attend_workspace_bytes(d, 1) == 0:
            entry["status"] = ("not built: 32 query rows x 512 fp32 latent accumulators per "
                               "wave exceed the register file")
            rows.append(entry)
            continue
        log(f"d_c {dc}")
        ms, k = chunk_step_kernels(vm, torch, d, 1, max(10, args.steps // 2), args.warmup, seed=50,
                                   partition=args.partition)
        W = work_model(d)
        entry.update({"ms_per_step": round(ms, 4), "kernels_us": k,
                      "latent_attend_tflops": round(W["attend_core"] / (k["latent_attend"] / 1e6) / 1e12, 1),
                      "latent_attend_mfma_frac": round(W["attend_core"] / (k["latent_attend"] / 1e6) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
                      "cache_write_hbm_frac": round(W["write_bytes"] / (k["cache_write"] / 1e6) / 1e9 / HBM_PEAK_GBPS, 4)})
        rows.append(entry)
    log("1-frame chunks")
    d = WAN_1F
    ms, k = chunk_step_kernels(vm, torch, d, 1, max(10, args.steps // 2), args.warmup, seed=51,
                               partition=args.partition)
    W = work_model(d)
    few = {"chunk_tokens": d.chunk_tokens, "ms_per_step": round(ms, 4), "kernels_us": k,
           "latent_attend_tflops": round(W["attend_core"] / (k["latent_attend"] / 1e6) / 1e12, 1),
           "latent_attend_mfma_frac": round(W["attend_core"] / (k["latent_attend"] / 1e6) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)}
    print(json.dumps({
        "metric": "latent attend TFLOP/s and % MFMA peak per latent width d_c (Table 5 sweep)",
        "value": next(r["latent_attend_tflops"] for r in rows if r["d_c"] == d0.d_c),
        "unit": "TFLOP/s", "n_gpus": 1, "higher_is_better": True, "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic", "sweep": rows, "one_frame_chunks": few,
        "config": {"workload": ("Wan2.1-1.3B layer chunk-step (3-frame chunk, 21-frame window, "
                                "batch 1) at d_c in {64, 128, 192, 256, 512}, d_rope 32; plus "
                                "1-frame chunks at d_c 192")},
    }), flush=True)


def few_query(args, vm, torch, d, batch=8):
    """The few-query regime: blocks of n_q query tokens (x 12 heads) per batch element of a
    batch of 8 videos, each attending over its wrapped 32,760-key Wan window (frames 3..23), in
    the latent path and in the dense per-head comparator at identical shapes. Per call the
    latent path reads 448 B per cached token, the dense one 6,144 B. Rings are filled by the
    library's own cache writes of seeded synthetic activations (frames 0..23); queries and
    weights are seeded synthetic bf16 drawn on the GPU. Per n_q: the per-kernel HIP-event
    averages of `steps` calls (frozen partition after adaptive calibration), the algorithmic
    bytes and HBM fraction of both attention kernels, and the floor any dense kernel faces from
    reading its cache once at the 8 TB/s peak."""
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(13)

    def normal(shape, std=1.0):
        return (torch.randn(shape, generator=g, device=dev) * std).to(torch.bfloat16)

    B, H, fe = batch, d.n_heads, d.window_frames
    S = vm.valid_tokens(d, fe)
    log("filling the latent and dense rings")
    w_dkv = normal((d.d_c, d.d_model), d.d_model ** -0.5)
    w_kr = normal((d.d_rope, d.d_model), d.d_model ** -0.5)
    w_uk = normal((H * d.d_nope, d.d_c), d.d_c ** -0.5)
    w_uv = normal((H * d.d_v, d.d_c), d.d_c ** -0.5)
    gamma = torch.ones(d.d_c, dtype=torch.bfloat16, device=dev)
    w_k = normal((H * d.d_v, d.d_model), d.d_model ** -0.5)
    w_v = normal((H * d.d_v, d.d_model), d.d_model ** -0.5)
    c_kv = torch.zeros((B, d.window_tokens, d.d_c), dtype=torch.bfloat16, device=dev)
    k_r = torch.zeros((B, d.window_tokens, d.d_rope), dtype=torch.bfloat16, device=dev)
    kv = torch.zeros((B, d.window_tokens, H, 2 * d.d_v), dtype=torch.bfloat16, device=dev)
    w_packed = torch.empty(vm.write_weights_bytes(d), dtype=torch.uint8, device=dev)
    vm.prepare_write_weights(d, w_dkv, w_kr, w_packed)
    for f in range(0, fe + 1, d.chunk_frames):
        x = normal((B, d.chunk_tokens, d.d_model))
        vm.cache_write_prepared(d, f, B, x, w_packed, gamma, c_kv, k_r)
        vm.dense_cache_write(d, f, B, x, w_k, w_v, kv)
    del x
    torch.cuda.synchronize()
    steps = max(10, args.steps // 2) if args.steps >= 10 else args.steps
    n_qs = tuple(int(v) for v in args.n_q.split(","))
    rows_out = []
    for n_q in n_qs:
        log(f"n_q {n_q}")
        q_nope, q_r = normal((B, n_q, H, d.d_nope)), normal((B, n_q, H, d.d_rope))
        q = normal((B, n_q, H, d.d_v))
        out = torch.empty((B, n_q, H, d.d_v), dtype=torch.bfloat16, device=dev)
        base = vm.AttendOpts(query_count=n_q)
        ws_l = torch.zeros(vm.attend_workspace_bytes(d, B, base), dtype=torch.uint8, device=dev)
        ws_d = torch.zeros(vm.dense_attend_workspace_bytes(d, B, base), dtype=torch.uint8,
                           device=dev)

        def lat(o):
            vm.attend(d, fe, B, q_nope, q_r, w_uk, w_uv, c_kv, k_r, out, ws_l, opts=o)

        def den(o):
            vm.dense_attend(d, fe, B, q, kv, out, ws_d, opts=o)

        res = {}
        for name, call, kern in (("latent", lat, ("q_absorb", "latent_attend", "latent_merge", "out_proj")),
                                 ("dense", den, ("dense_q_prep", "dense_attend", "dense_merge"))):
            part = args.partition
            for _ in range(args.warmup):
                call(dataclasses.replace(base, partition="adaptive" if part == "frozen" else part))
            torch.cuda.synchronize()
            timer = vm.Timer()
            for _ in range(steps):
                call(dataclasses.replace(base, partition=part, timer=timer))
            torch.cuda.synchronize()
            k_us = {}
            for k in kern:
                c, tot = timer.read(k)
                k_us[k] = round(1e3 * tot / max(c, 1), 2)
            timer.close()
            res[name] = {"kernels_us": k_us, "attend_us": round(sum(k_us.values()), 2)}
        rows = B * n_q * H
        # algorithmic bytes of the attention kernels: the cache read once, the query rows in
        lat_bytes = B * S * 2 * (d.d_c + d.d_rope) + rows * 2 * (d.d_c + d.d_rope)
        den_bytes = B * S * H * 2 * d.d_v * 2 + rows * 2 * d.d_v
        t_l = res["latent"]["kernels_us"]["latent_attend"] / 1e6
        t_d = res["dense"]["kernels_us"]["dense_attend"] / 1e6
        res["latent"].update({"attention_kernel_bytes": lat_bytes,
                              "attention_kernel_hbm_frac": round(lat_bytes / t_l / 8e12, 4),
                              "attention_kernel_tflops": round(rows * S * 832 / t_l / 1e12, 1)})
        res["dense"].update({"attention_kernel_bytes": den_bytes,
                             "attention_kernel_hbm_frac": round(den_bytes / t_d / 8e12, 4),
                             "attention_kernel_tflops": round(rows * S * 512 / t_d / 1e12, 1),
                             "hbm_floor_us": round(den_bytes / 8e12 * 1e6, 2)})
        res["latent_over_dense_attend"] = round(res["latent"]["attend_us"] / res["dense"]["attend_us"], 4)
        rows_out.append({"n_q": n_q, "query_rows": rows, **res})
        del ws_l, ws_d
        torch.cuda.empty_cache()
    if args.copy_probe:
        log("copy probe")
        copy_probe(torch, dev)
    faster = [r["n_q"] for r in rows_out if r["latent_over_dense_attend"] < 1.0]
    print(json.dumps({
        "metric": "attend us per call, few-query regime: latent vs dense per-head cache",
        "value": rows_out[0]["latent_over_dense_attend"],
        "unit": f"latent / dense attend time at n_q = {rows_out[0]['n_q']}",
        "n_gpus": 1, "higher_is_better": False, "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic", "results": rows_out,
        "latent_faster_at_n_q": faster,
        "cache_bytes_per_token": {"latent": vm.cache_bytes_per_token(d),
                                  "dense": vm.dense_cache_bytes_per_token(d)},
        "config": {"workload": ("Wan2.1-1.3B geometry, batch 8: blocks of n_q query tokens x 12 "
                                "heads per video over its wrapped 32,760-key 21-frame window, "
                                "latent path vs dense per-head comparator"),
                   "batch": B, "n_q": list(n_qs), "window_tokens": S, "seed": 13,
                   "attend_partition": args.partition},
    }), flush=True)


def form_crossover(args, vm, torch, n_qs=(208, 1560, 4680)):
    """Latent against materialized form per shape, and the form VIDEOMLA_FORM_AUTO picks: Wan
    geometry, batch 1, a 3-frame chunk over its wrapped 32,760-key window, with the queries of
    the first n_q chunk tokens (208 tokens, 1 frame, 3 frames), d_nope 96 (the paper's split,
    pairs (6,5,5)) and 128, d_c 128 and 192. Per point: the attend time of each form (sum of its
    kernels' HIP-event averages over `steps` calls, frozen partition after adaptive calibration)
    and whether the automatic choice took the faster one. Seeded synthetic bf16 drawn on the
    GPU; the ring is filled by the library's cache writes."""
    from workloads import WAN, WAN_PAPER
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(14)

    def normal(shape, std=1.0):
        return (torch.randn(shape, generator=g, device=dev) * std).to(torch.bfloat16)

    steps = max(10, args.steps // 4)
    points = []
    for base_dims, split in ((WAN_PAPER, "d_nope 96"), (WAN, "d_nope 128")):
        for d_c in (128, 192):
            d = base_dims.replace(d_c=d_c)
            H, fe = d.n_heads, d.window_frames
            log(f"{split}, d_c {d_c}")
            w_dkv = normal((d.d_c, d.d_model), d.d_model ** -0.5)
            w_kr = normal((d.d_rope, d.d_model), d.d_model ** -0.5)
            w_uk = normal((H * d.d_nope, d.d_c), d.d_c ** -0.5)
            w_uv = normal((H * d.d_v, d.d_c), d.d_c ** -0.5)
            gamma = torch.ones(d.d_c, dtype=torch.bfloat16, device=dev)
            c_kv = torch.zeros((1, d.window_tokens, d.d_c), dtype=torch.bfloat16, device=dev)
            k_r = torch.zeros((1, d.window_tokens, d.d_rope), dtype=torch.bfloat16, device=dev)
            w_packed = torch.empty(vm.write_weights_bytes(d), dtype=torch.uint8, device=dev)
            vm.prepare_write_weights(d, w_dkv, w_kr, w_packed)
            for f in range(0, fe + 1, d.chunk_frames):
                vm.cache_write_prepared(d, f, 1, normal((1, d.chunk_tokens, d.d_model)), w_packed,
                                        gamma, c_kv, k_r)
            for n_q in n_qs:
                q_nope, q_r = normal((1, n_q, H, d.d_nope)), normal((1, n_q, H, d.d_rope))
                out = torch.empty((1, n_q, H, d.d_v), dtype=torch.bfloat16, device=dev)
                res = {}
                for form, kern in (("latent", ("q_absorb", "latent_attend", "latent_merge", "out_proj")),
                                   ("materialized", ("mat_kv", "mat_q_prep", "mat_attend",
                                                     "mat_merge"))):
                    base = vm.AttendOpts(form=form, query_count=n_q)
                    ws = torch.zeros(vm.attend_workspace_bytes(d, 1, base), dtype=torch.uint8,
                                     device=dev)

                    def call(o):
                        vm.attend(d, fe, 1, q_nope, q_r, w_uk, w_uv, c_kv, k_r, out, ws, opts=o)
                    for _ in range(args.warmup):
                        call(dataclasses.replace(base, partition="adaptive"))
                    timer = vm.Timer()
                    for _ in range(steps):
                        call(dataclasses.replace(base, partition="frozen", timer=timer))
                    torch.cuda.synchronize()
                    us = {k: round(1e3 * v[1] / max(v[0], 1), 2)
                          for k, v in ((k, timer.read(k)) for k in kern)}
                    timer.close()
                    res[form] = {"attend_us": round(sum(us.values()), 2), "kernels_us": us}
                    del ws
                auto = vm.AttendOpts(form="auto", query_count=n_q)
                auto_mat = (vm.attend_workspace_bytes(d, 1, auto)
                            == vm.attend_workspace_bytes(d, 1, vm.AttendOpts(form="materialized",
                                                                             query_count=n_q)))
                faster = ("materialized" if res["materialized"]["attend_us"]
                          < res["latent"]["attend_us"] else "latent")
                points.append({"head_split": split, "d_c": d_c, "n_q": n_q, **res,
                               "materialized_over_latent": round(res["materialized"]["attend_us"]
                                                                 / res["latent"]["attend_us"], 4),
                               "faster": faster,
                               "auto_picks": "materialized" if auto_mat else "latent",
                               "auto_right": (auto_mat and faster == "materialized")
                               or (not auto_mat and faster == "latent")})
                torch.cuda.empty_cache()
    print(json.dumps({
        "metric": "attend us per call: latent vs materialized form per shape, and the automatic choice",
        "value": sum(p["auto_right"] for p in points), "unit": f"points of {len(points)} where auto "
        "picked the faster form", "n_gpus": 1, "higher_is_better": True, "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic", "points": points,
        "config": {"workload": ("Wan2.1-1.3B geometry, batch 1: the first n_q tokens of a 3-frame "
                                "chunk (208, 1,560, 4,680) x 12 heads over the wrapped 32,760-key "
                                "window; d_nope 96 / 128, d_c 128 / 192"), "seed": 14},
    }), flush=True)


def xcd_balance(args, vm, torch, d, n_calls=12):
    """The per-XCD imbalance the weighted partition corrects, read from the library's own
    record: the partition state at the end of the attention workspace holds the weights a call
    used and each workgroup's duration (100 MHz ticks). The first adaptive call on a fresh
    workspace splits evenly (no record yet), so its durations are the even split's; each later
    adaptive call re-weights the XCDs from the previous one's. Wan chunk-step shape, batch 1,
    wrapped window; latent_attend timed by HIP events."""
    import numpy as np
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(15)

    def normal(shape, std=1.0):
        return (torch.randn(shape, generator=g, device=dev) * std).to(torch.bfloat16)

    nq, H = d.chunk_tokens, d.n_heads
    c_kv, k_r = normal((1, d.window_tokens, d.d_c)), normal((1, d.window_tokens, d.d_rope))
    q_nope, q_r = normal((1, nq, H, d.d_nope)), normal((1, nq, H, d.d_rope))
    w_uk = normal((H * d.d_nope, d.d_c), d.d_c ** -0.5)
    w_uv = normal((H * d.d_v, d.d_c), d.d_c ** -0.5)
    out = torch.empty((1, nq, H, d.d_v), dtype=torch.bfloat16, device=dev)
    ws = torch.zeros(vm.attend_workspace_bytes(d, 1), dtype=torch.uint8, device=dev)
    state_words, state_bytes = 16 + 4096, ((16 + 4096) * 4 + 255) // 256 * 256
    fe = d.window_frames
    for _ in range(args.warmup):  # clock ramp, on another workspace
        vm.attend(d, fe, 1, q_nope, q_r, w_uk, w_uv, c_kv, k_r, out,
                  torch.empty_like(ws))
    torch.cuda.synchronize()
    timer = vm.Timer()
    rows = []
    for call in range(n_calls):
        vm.attend(d, fe, 1, q_nope, q_r, w_uk, w_uv, c_kv, k_r, out, ws,
                  opts=vm.AttendOpts(partition="adaptive", timer=timer))
        torch.cuda.synchronize()
        _, t_ms = timer.read("latent_attend")
        st = ws[-state_bytes:][:state_words * 4].cpu().numpy().view(np.uint32)
        G = int(st[8])
        dur = st[16:16 + G].astype(np.float64) / 100.0  # us
        per_xcd = [float(dur[x::8].max()) for x in range(8)]
        spread = [float(dur[x::8].max() - dur[x::8].min()) for x in range(8)]
        rows.append({"call": call, "weights": [int(v) for v in st[:8]],
                     "xcd_slowest_workgroup_us": [round(v, 1) for v in per_xcd],
                     "slowest_over_fastest_xcd": round(max(per_xcd) / min(per_xcd), 4),
                     "within_xcd_spread_us_max": round(max(spread), 1),
                     "latent_attend_us": round(1e3 * t_ms, 1)})
    timer.close()
    print(json.dumps({
        "metric": "per-XCD workgroup times of latent_attend under the even and the weighted split",
        "value": rows[0]["slowest_over_fastest_xcd"], "unit": "slowest / fastest XCD, even split",
        "n_gpus": 1, "higher_is_better": False, "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic", "calls": rows,
        "config": {"workload": ("Wan2.1-1.3B layer attend (4,680 x 12 query rows over 32,760 keys), "
                                "batch 1; call 0 splits evenly (no record), later calls re-weight"),
                   "seed": 15},
    }), flush=True)


STAMP_POINTS = {
    "cache_write_packed": {0: "start", 1: "x first half landed", 2: "x second half landed",
                           3: "last MFMA issued", 4: "sums of squares exchanged",
                           5: "output tile complete", 6: "stores complete"},
    "cache_write_wide": {0: "start", 1: "tables done",
                         **{2 + p: f"phase {p} landed" for p in range(10)},
                         12: "last MFMA issued", 13: "sums of squares exchanged",
                         14: "output tile complete", 15: "stores complete"},
    "q_absorb": {0: "start", 1: "W_UK_h staged", 2: "last MFMA issued", 3: "latent part written",
                 4: "RoPE part written", 5: "rows staged", 6: "stores complete"},
    "latent_attend": {0: "start", 1: "first two tiles landed", 10: "last step done",
                      11: "partial results stored"},
    "out_proj": {0: "start", 1: "coefficients and W_UV_h in LDS", 2: "o_lat merged",
                 3: "last MFMA issued", 4: "output rows staged", 5: "stores complete"},
}


def stamp_summary(rec, points):
    """Per point: the median over workgroups of the time (us) at which the last wave of the
    workgroup reached it, after the workgroup's start (its first wave's point 0); plus the
    workgroups' own durations and the span from the first start to the last point."""
    import numpy as np
    live = rec[:, :, 0].max(axis=1) > 0
    r = rec[live].astype(np.float64)             # [wg][wave][point], 100 MHz ticks
    r[r == 0] = np.nan
    start = np.nanmin(r[:, :, 0], axis=1)        # [wg]
    last = np.nanmax(r, axis=(1, 2))
    out = {"workgroups": int(live.sum()),
           "span_us": round(float(np.nanmax(last) - np.nanmin(start)) / 100, 2),
           "workgroup_us_median": round(float(np.median(last - start)) / 100, 2),
           "workgroup_us_max": round(float(np.max(last - start)) / 100, 2),
           "start_spread_us": round(float(np.nanmax(start) - np.nanmin(start)) / 100, 2),
           "points_us": {}}
    for p, name in points.items():
        if p == 0 or np.isnan(r[:, :, p]).all():  # the start, or a point no wave reached
            continue
        col = np.nanmax(r[:, :, p], axis=1) - start
        col = col[~np.isnan(col)]
        if len(col):
            out["points_us"][name] = round(float(np.median(col)) / 100, 2)
    return out


def attend_step_waves(rec):
    """latent_attend, steps 200..203 of every workgroup: the step time (barrier release to
    barrier release); per SIMD (waves w and w + 4) how long each wave waits at the barrier after
    its instruction stream ends, the older wave (w) and the younger (w + 4) apart; the time from
    the last wave's stream end to the release; and how far apart the four SIMDs end."""
    import numpy as np
    live = rec[:, :, 0].max(axis=1) > 0
    r = rec[live].astype(np.float64)
    steps, older, younger, alone, last_gap, simd_spread = [], [], [], [], [], []
    for i in range(4):
        end, rel = r[:, :, 2 + 2 * i], r[:, :, 3 + 2 * i]    # [wg][wave]
        ok = (end > 0).all(axis=1) & (rel > 0).all(axis=1)
        release = rel[ok].min(axis=1)
        older.append((release[:, None] - end[ok][:, 0:4]).ravel())
        younger.append((release[:, None] - end[ok][:, 4:8]).ravel())
        alone.append(np.abs(end[ok][:, 4:8] - end[ok][:, 0:4]).ravel())
        # the barrier's own delay: from the last wave's stream end to the release (this includes
        # the wait for the next tile's loads), and how far apart the SIMDs end
        last_gap.append(release - end[ok].max(axis=1))
        simd_end = np.maximum(end[ok][:, 0:4], end[ok][:, 4:8])
        simd_spread.append(simd_end.max(axis=1) - simd_end.min(axis=1))
        if i > 0:
            prev = r[:, :, 1 + 2 * i]
            ok2 = ok & (prev > 0).all(axis=1)
            steps.append(rel[ok2].min(axis=1) - prev[ok2].min(axis=1))
    cat = lambda xs: np.concatenate(xs) / 100.0  # noqa: E731
    s, o, y, a = cat(steps), cat(older), cat(younger), cat(alone)
    return {"step_us_median": round(float(np.median(s)), 3),
            "older_wave_barrier_wait_us_median": round(float(np.median(o)), 3),
            "younger_wave_barrier_wait_us_median": round(float(np.median(y)), 3),
            "older_wave_ends_first_fraction": round(float(np.mean(o >= y)), 3),
            "one_wave_alone_us_median": round(float(np.median(a)), 3),
            "last_stream_end_to_release_us_median": round(float(np.median(cat(last_gap))), 3),
            "simd_end_spread_us_median": round(float(np.median(cat(simd_spread))), 3),
            "samples": int(len(o))}


def attend_segments(rec):
    """latent_attend: the switch between a workgroup's two segments (first segment's last step
    to the second's first two tiles landed, split at the partial results' issue), the tail from
    the last step to the partial results stored, and the workgroup durations of one- and
    two-segment workgroups."""
    import numpy as np
    live = rec[:, :, 0].max(axis=1) > 0
    r = rec[live].astype(np.float64)
    r[r == 0] = np.nan
    start = np.nanmin(r[:, :, 0], axis=1)
    end = np.nanmax(r[:, :, 11], axis=1)
    def row_max(p):  # the last wave's stamp per workgroup; NaN where no wave recorded it
        m = np.where(np.isnan(r[:, :, p]), -np.inf, r[:, :, p]).max(axis=1)
        return np.where(np.isinf(m), np.nan, m)
    last, p12, p13, p14 = (row_max(p) for p in (10, 12, 13, 14))
    two = ~np.isnan(p14)
    us = lambda x: round(float(np.median(x)) / 100, 2) if len(x) else None  # noqa: E731
    return {"two_segment_workgroups": int(two.sum()),
            "switch_us_median": us(p14[two] - p12[two]),
            "switch_stores_issued_us_median": us(p13[two] - p12[two]),
            "switch_to_tiles_landed_us_median": us(p14[two] - p13[two]),
            "end_tail_us_median": us(end - last),
            "one_segment_workgroup_us_median": us((end - start)[~two]),
            "two_segment_workgroup_us_median": us((end - start)[two])}


def phase_timelines(args, vm, torch, d, reps=5):
    """Phase timelines of the stamped kernels (the diagnostic build, loaded because this
    workload sets VIDEOMLA_LIBRARY=stamps): the Wan chunk-step at batch 1 (packed cache write,
    q_absorb, latent_attend on the frozen partition, out_proj) and the batch-4 cache write
    (wide kernel), each recorded `reps` times after warm-up. Every figure is the median of the
    per-record figures of stamp_summary / attend_step_waves. The stamped kernels' own HIP-event
    times are reported beside them: the stamps' stores and waits make them a little slower
    than the product build's."""
    import numpy as np
    if not vm.STAMPS:
        raise RuntimeError("wan-phase-timelines needs the diagnostic build (VIDEOMLA_LIBRARY=stamps)")
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(21)

    def normal(shape, std=1.0):
        return (torch.randn(shape, generator=g, device=dev) * std).to(torch.bfloat16)

    nq, H = d.chunk_tokens, d.n_heads
    w_dkv = normal((d.d_c, d.d_model), d.d_model ** -0.5)
    w_kr = normal((d.d_rope, d.d_model), d.d_model ** -0.5)
    w_uk = normal((H * d.d_nope, d.d_c), d.d_c ** -0.5)
    w_uv = normal((H * d.d_v, d.d_c), d.d_c ** -0.5)
    gamma = torch.ones(d.d_c, dtype=torch.bfloat16, device=dev)
    w_packed = torch.empty(vm.write_weights_bytes(d), dtype=torch.uint8, device=dev)
    vm.prepare_write_weights(d, w_dkv, w_kr, w_packed)
    rings = {}
    for B in (1, 4):
        c_kv = torch.zeros((B, d.window_tokens, d.d_c), dtype=torch.bfloat16, device=dev)
        k_r = torch.zeros((B, d.window_tokens, d.d_rope), dtype=torch.bfloat16, device=dev)
        for f in range(0, d.window_frames, d.chunk_frames):
            vm.cache_write_prepared(d, f, B, normal((B, nq, d.d_model)), w_packed, gamma, c_kv, k_r)
        rings[B] = (c_kv, k_r, normal((B, nq, d.d_model)))
    q_nope, q_r = normal((1, nq, H, d.d_nope)), normal((1, nq, H, d.d_rope))
    out = torch.empty((1, nq, H, d.d_v), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(vm.attend_workspace_bytes(d, 1), dtype=torch.uint8, device=dev)
    fe = d.window_frames

    def write(B):
        c_kv, k_r, x = rings[B]
        vm.cache_write_prepared(d, fe, B, x, w_packed, gamma, c_kv, k_r)

    def attend(o):
        c_kv, k_r, _ = rings[1]
        vm.attend(d, fe, 1, q_nope, q_r, w_uk, w_uv, c_kv, k_r, out, ws, opts=o)

    def step(i, timer=None):
        bracket(timer, "cache_write", lambda: write(1))
        attend(vm.AttendOpts(partition="frozen", timer=timer))

    for i in range(args.warmup):
        step(i)
        write(4)
    calibrate(vm, torch, attend)
    # the stamped kernels' own times, before any stamp buffer is attached
    _, _, kernels = timed_steps(vm, torch, step, 10, ("cache_write", "q_absorb", "latent_attend",
                                                      "out_proj"))
    buf = torch.zeros(vm.stamps_buffer_bytes() // 8, dtype=torch.int64, device=dev)
    vm.stamps_attach(buf)
    shape = (vm.STAMP_KERNELS, vm.STAMP_WORKGROUPS, vm.STAMP_WAVES, vm.STAMP_POINTS)
    per = {k: [] for k in STAMP_POINTS}
    steps, segs = [], []
    try:
        for _ in range(reps):
            buf.zero_()
            step(0)
            write(4)
            torch.cuda.synchronize()
            rec = buf.cpu().numpy().view(np.uint64).reshape(shape)
            for k, pts in STAMP_POINTS.items():
                per[k].append(stamp_summary(rec[vm.STAMP_KERNEL[k]], pts))
            steps.append(attend_step_waves(rec[vm.STAMP_KERNEL["latent_attend"]]))
            segs.append(attend_segments(rec[vm.STAMP_KERNEL["latent_attend"]]))
    finally:
        vm.stamps_attach(None)
        torch.cuda.synchronize()

    def med(rows):
        keys = rows[0].keys()
        res = {}
        for key in keys:
            if isinstance(rows[0][key], dict):
                res[key] = med([r[key] for r in rows])
            elif any(r[key] is None for r in rows):
                res[key] = None
            else:
                res[key] = round(float(np.median([r[key] for r in rows])), 3)
        return res

    print(json.dumps({
        "metric": "phase timelines of the stamped kernels (median over workgroups, then over records)",
        "value": med(per["latent_attend"])["span_us"], "unit": "us (latent_attend span)",
        "n_gpus": 1, "higher_is_better": False, "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic", "records": reps,
        "stamped_build_event_us": {k: v["avg_us"] for k, v in kernels.items()},
        "kernels": {k: med(v) for k, v in per.items()},
        "latent_attend_steps_200_203": med(steps),
        "latent_attend_segments": med(segs),
        "config": {"workload": ("Wan2.1-1.3B chunk-step at batch 1 (cache write of 4,680 tokens, "
                                "attend of 4,680 x 12 query rows over 32,760 keys, frozen "
                                "partition) and the batch-4 cache write, diagnostic build"),
                   "seed": 21},
    }), flush=True)


def event_timed(torch, fn, filler, n=60, warm=10):
    """Mean and median microseconds of fn(i), each call bracketed by HIP events on the current
    stream, with filler() (a long kernel) queued ahead of every ten calls so that the events time
    the kernels rather than host launch gaps."""
    for i in range(warm):
        fn(i)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(n)]
    for i in range(n):
        if i % 10 == 0:
            filler()
        ev[i][0].record()
        fn(i)
        ev[i][1].record()
    torch.cuda.synchronize()
    t = sorted(a.elapsed_time(b) * 1e3 for a, b in ev)
    return sum(t) / len(t), t[len(t) // 2]


def library_references(args, vm, torch, d):
    """Reference rates of the vendor GEMM library (hipBLASLt, through torch.matmul) on this machine:
    large square bf16 products (a practical dense MFMA ceiling, against the published 2.5 PF)
    and the cache write's bare projection x [B*Nq, d_model] @ [W_DKV; W_KR]^T at the Wan shape,
    next to the library's fused cache write of the same tokens (projection + RMSNorm + RoPE +
    ring scatter). Every call is bracketed by HIP events on the current stream, with a long
    product queued ahead of every ten calls so that the events time kernels, not host launch
    gaps. Seeded synthetic bf16 drawn on the GPU; x cycles through 8 buffers."""
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(7)

    def normal(shape, std=1.0):
        return (torch.randn(shape, generator=g, device=dev) * std).to(torch.bfloat16)

    filler_a, filler_b = normal((8192, 8192)), normal((8192, 8192))

    def timed(fn, n=60, warm=10):
        return event_timed(torch, fn, lambda: torch.matmul(filler_a, filler_b), n, warm)

    gemms = []
    for (m, n, k) in ((8192, 8192, 8192), (16384, 16384, 4096)):
        a, b = normal((m, k)), normal((k, n))
        avg, med = timed(lambda i: torch.matmul(a, b), n=20, warm=5)
        gemms.append({"m": m, "n": n, "k": k, "avg_us": round(avg, 2),
                      "tflops": round(2 * m * n * k / (avg * 1e-6) / 1e12, 1),
                      "frac_of_2.5pf": round(2 * m * n * k / (avg * 1e-6) / 1e12
                                             / MFMA_BF16_PEAK_TFLOPS, 4)})
        del a, b
    log(f"square GEMMs: {gemms}")

    no = d.d_c + d.d_rope
    w_dkv = normal((d.d_c, d.d_model), d.d_model ** -0.5)
    w_kr = normal((d.d_rope, d.d_model), d.d_model ** -0.5)
    w_t = torch.cat([w_dkv, w_kr], 0).t().contiguous()          # [d_model, d_c + d_rope]
    gamma = torch.ones(d.d_c, dtype=torch.bfloat16, device=dev)
    w_packed = torch.empty(vm.write_weights_bytes(d), dtype=torch.uint8, device=dev)
    vm.prepare_write_weights(d, w_dkv, w_kr, w_packed)
    proj = []
    for B in (1, 2, 4, 8):
        M = B * d.chunk_tokens
        xs = [normal((B, d.chunk_tokens, d.d_model)) for _ in range(8)]
        y = torch.empty((M, no), dtype=torch.bfloat16, device=dev)
        c_kv = torch.zeros((B, d.window_tokens, d.d_c), dtype=torch.bfloat16, device=dev)
        k_r = torch.zeros((B, d.window_tokens, d.d_rope), dtype=torch.bfloat16, device=dev)
        lib, _ = timed(lambda i: torch.matmul(xs[i % 8].view(M, d.d_model), w_t, out=y))
        fused, _ = timed(lambda i: vm.cache_write_prepared(d, 21, B, xs[i % 8], w_packed, gamma,
                                                           c_kv, k_r))
        byts = M * (2 * d.d_model + 2 * no) + 2 * d.d_model * no
        proj.append({"batch": B, "tokens": M, "library_gemm_us": round(lib, 2),
                     "fused_cache_write_us": round(fused, 2),
                     "fused_over_library": round(fused / lib, 3),
                     "algorithmic_bytes": byts,
                     "fused_hbm_frac": round(byts / (fused * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                     "library_hbm_frac": round(byts / (lib * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)})
        log(f"projection batch {B}: {proj[-1]}")
        del xs, y, c_kv, k_r
        torch.cuda.empty_cache()
    print(json.dumps({
        "metric": "vendor GEMM library references: square bf16 products and the cache write's "
                  "bare projection vs the fused cache write",
        "value": proj[0]["fused_over_library"], "unit": "fused cache write / library GEMM time, batch 1",
        "n_gpus": 1, "higher_is_better": False, "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic", "square_gemms": gemms, "cache_write_projection": proj,
        "config": {"workload": ("torch.matmul (hipBLASLt) bf16: square products, and "
                                "x[B*4680, 1536] @ [W_DKV; W_KR]^T (1536 x 224) at batch 1-8 "
                                "against videomla_cache_write_prepared on the same tokens"),
                   "seed": 7},
    }), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--x-buffers", type=int, default=32)
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a 256 MiB device copy (counter calibration)")
    ap.add_argument("--workload", default="wan-layer-chunk-step",
                    choices=("wan-layer-chunk-step", "wan-30-layer-chunk", "wan-rollout-b4",
                             "wan-sink-chunk-step", "wan-full-layer-chunk-step", "wan-dc-sweep",
                             "wan-latent-vs-materialized", "wan-few-query",
                             "wan-form-crossover", "wan-xcd-balance", "library-references",
                             "wan-phase-timelines"),
                    help="wan-layer-chunk-step: the headline (one layer's write + attend); "
                         "wan-30-layer-chunk: one chunk through 30 layers x 4 denoising steps "
                         "plus the window advance; wan-rollout-b4: batch-4 rollout of --chunks "
                         "chunks through 30 layers, latent path and dense comparator; "
                         "wan-sink-chunk-step: one chunk-step with a sink frame + 6 recent "
                         "frames late in a rollout; wan-full-layer-chunk-step: the whole "
                         "attention layer in latent form (query path and W_O absorbed); "
                         "wan-dc-sweep: chunk-steps at the latent widths of the paper's d_c "
                         "sweep and with 1-frame chunks; wan-latent-vs-materialized: the "
                         "latent and the materialized-K/V attention at both head splits; "
                         "wan-few-query: blocks of 16..1560 query tokens at batch 8, latent vs "
                         "dense; wan-form-crossover: latent vs materialized per (n_q, d_nope, "
                         "d_c) and the automatic choice; wan-xcd-balance: per-XCD workgroup "
                         "times from the partition's own record; library-references: the "
                         "vendor GEMM library's rate on square products and on the cache "
                         "write's bare projection, next to the fused cache write; "
                         "wan-phase-timelines: per-phase times of the kernels from the "
                         "diagnostic build's stamps (libvideomla_stamps.so)")
    ap.add_argument("--chunks", type=int, default=80, help="chunks of the wan-rollout-b4 run")
    ap.add_argument("--n-q", default="16,52,208,1560",
                    help="query tokens per video of the wan-few-query run (comma-separated)")
    ap.add_argument("--partition", choices=("frozen", "even", "adaptive"), default="frozen",
                    help="work partition of the attention calls: frozen (default; per-XCD "
                         "weights calibrated by a few adaptive calls before the timed region, "
                         "then fixed: bitwise reproducible), even, or adaptive (re-weighted "
                         "every call)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    if args.workload == "wan-phase-timelines":
        os.environ["VIDEOMLA_LIBRARY"] = "stamps"  # read by the binding at import
    import paper_2605_30351_amd as vm
    from workloads import WAN, make_layer_inputs

    if args.workload == "wan-phase-timelines":
        phase_timelines(args, vm, torch, WAN)
        return

    if args.workload == "wan-30-layer-chunk":
        thirty_layer_chunk(args, vm, torch, WAN)
        return
    if args.workload == "wan-rollout-b4":
        rollout_comparison(args, vm, torch, WAN)
        return
    if args.workload == "wan-full-layer-chunk-step":
        full_layer_chunk_step(args, vm, torch, WAN)
        return
    if args.workload == "wan-latent-vs-materialized":
        latent_vs_materialized(args, vm, torch)
        return
    if args.workload == "wan-xcd-balance":
        xcd_balance(args, vm, torch, WAN)
        return
    if args.workload == "library-references":
        library_references(args, vm, torch, WAN)
        return
    if args.workload == "wan-form-crossover":
        form_crossover(args, vm, torch)
        return
    if args.workload == "wan-few-query":
        few_query(args, vm, torch, WAN)
        return
    if args.workload == "wan-dc-sweep":
        dc_sweep(args, vm, torch, WAN)
        return
    if args.workload == "wan-sink-chunk-step":
        from workloads import WAN_SINK
        sink_chunk_step(args, vm, torch, WAN_SINK)
        return

    d = WAN
    dev = torch.device("cuda:0")
    log("generating inputs")
    inp = make_layer_inputs(d, seed=1, n_frames=24)

    def t(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)

    w_dkv, w_kr, w_uk, w_uv, gamma = (t(inp.w_dkv), t(inp.w_kr), t(inp.w_uk), t(inp.w_uv),
                                      t(inp.gamma))
    q_nope, q_r = t(inp.q_nope), t(inp.q_r)
    x_all = t(inp.x)
    c_kv = torch.zeros((1, d.window_tokens, d.d_c), dtype=torch.bfloat16, device=dev)
    k_r = torch.zeros((1, d.window_tokens, d.d_rope), dtype=torch.bfloat16, device=dev)
    out = torch.empty((1, d.chunk_tokens, d.n_heads, d.d_v), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(vm.attend_workspace_bytes(d, 1), dtype=torch.uint8, device=dev)
    # the layer's compression weights, packed once (model-load time, outside the timed region)
    w_packed = torch.empty(vm.write_weights_bytes(d), dtype=torch.uint8, device=dev)
    vm.prepare_write_weights(d, w_dkv, w_kr, w_packed)

    # fill the ring with frames 0..20, then the step writes frames 21..23 (evicting 0..2)
    for fe in range(0, 21, d.chunk_frames):
        vm.cache_write(d, fe, 1, x_all[:, fe * d.hw:(fe + 3) * d.hw].contiguous(), w_dkv, w_kr,
                       gamma, c_kv, k_r)
    fe = 21
    x_chunk = x_all[:, fe * d.hw:(fe + 3) * d.hw].contiguous()
    xs = [x_chunk.clone() for _ in range(args.x_buffers)]
    del x_all
    torch.cuda.synchronize()

    def attend(o):
        vm.attend(d, fe, 1, q_nope, q_r, w_uk, w_uv, c_kv, k_r, out, ws, opts=o)

    def step(i, timer=None, partition=args.partition):
        bracket(timer, "cache_write", lambda: vm.cache_write_prepared(d, fe, 1, xs[i % len(xs)], w_packed,
                                                            gamma, c_kv, k_r))
        attend(vm.AttendOpts(partition=partition, timer=timer))

    log(f"warmup {args.warmup}")
    for i in range(args.warmup):
        step(i)
    if args.partition == "frozen":
        calibrate(vm, torch, attend)  # per-XCD weights for the frozen calls below
    torch.cuda.synchronize()

    if args.copy_probe:
        log("copy probe")
        copy_probe(torch, dev)

    # The timed region carries HIP events around the roofline kernel (latent_attend) only: every
    # event pair adds a few microseconds to the step. The per-kernel breakdown comes from a
    # second pass of the same steps with every kernel bracketed.
    log(f"timing {args.steps} steps")
    k3_timer = vm.Timer()
    k3_timer.only("latent_attend")
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    marks[0].record()
    for i in range(args.steps):
        step(i, k3_timer)
        marks[i + 1].record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    step_ms = np.array([marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps)])
    n_k3, t_k3 = k3_timer.read("latent_attend")
    log("timed region done")
    frozen_out = out.clone() if args.partition == "frozen" else None

    names = ("cache_write", "q_absorb", "latent_attend", "latent_merge", "out_proj")
    kernels = {}
    all_timer = vm.Timer()
    for i in range(args.steps):
        step(i, all_timer)
    torch.cuda.synchronize()
    for k in names:
        n, tot = all_timer.read(k)
        kernels[k] = {"launches": n, "avg_us": 1e3 * tot / max(n, 1)}
    # the same steps with the even split, for comparison with the measured partition
    for i in range(args.steps):
        step(i, all_timer, "even")
    torch.cuda.synchronize()
    n_even, t_even = all_timer.read("latent_attend")
    if frozen_out is not None:  # frozen calls repeat bitwise
        attend(vm.AttendOpts(partition="frozen"))
        torch.cuda.synchronize()
        repeat_ok = bool(torch.equal(out.view(torch.int16), frozen_out.view(torch.int16)))
    all_timer.read("cache_write")
    # The writes below run back to back, each shorter than its host-side launch; an attention
    # call queued ahead of every ten keeps the stream busy, so that the events bracket the
    # kernels rather than the host's launch gaps. First the cache write alone with one x
    # buffer, which then stays in the 256 MB Infinity Cache:
    for i in range(20):
        if i % 10 == 0:
            attend(vm.AttendOpts(partition=args.partition))
        bracket(all_timer, "cache_write", lambda: vm.cache_write_prepared(
            d, fe, 1, xs[0], w_packed, gamma, c_kv, k_r))
    torch.cuda.synchronize()
    n_w, t_w = all_timer.read("cache_write")
    warm_mall_us = 1e3 * t_w / max(n_w, 1)
    # the same write from the plain row-major weights (videomla_cache_write), rotating x buffers
    for i in range(50):
        if i % 10 == 0:
            attend(vm.AttendOpts(partition=args.partition))
        x = xs[i % len(xs)]
        bracket(all_timer, "cache_write", lambda: vm.cache_write(d, fe, 1, x, w_dkv, w_kr, gamma,
                                                                 c_kv, k_r))
    torch.cuda.synchronize()
    n_p, t_p = all_timer.read("cache_write")
    plain_us = 1e3 * t_p / max(n_p, 1)
    all_timer.close()

    ms = 1e3 * elapsed / args.steps
    W = work_model(d)
    att_ms = (kernels["q_absorb"]["avg_us"] + kernels["latent_attend"]["avg_us"]
              + kernels["latent_merge"]["avg_us"] + kernels["out_proj"]["avg_us"]) / 1e3
    k3_s = t_k3 / max(n_k3, 1) / 1e3  # from the timed region
    k3_tflops = W["attend_core"] / k3_s / 1e12
    wr_s = kernels["cache_write"]["avg_us"] / 1e6
    even_s = t_even / max(n_even, 1) / 1e3

    result = {
        "metric": "ms/chunk-step & TFLOP/s for latent-MLA attend (Wan-1.3B shape); % MFMA peak",
        "value": round((W["attend"] + W["write"]) / (ms / 1e3) / 1e12, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "step_ms_p10_p50_p90": [round(float(np.percentile(step_ms, q)), 4) for q in (10, 50, 90)],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": ("Wan2.1-1.3B layer chunk-step: cache write of 4,680 tokens (3 frames of "
                         "30x52) + latent attend of 4,680 tokens x 12 heads over a 32,760-token "
                         "21-frame window, batch 1"),
            "d_model": d.d_model, "heads": d.n_heads, "d_nope": d.d_nope, "d_rope": d.d_rope,
            "d_c": d.d_c, "d_v": d.d_v, "chunk_tokens": d.chunk_tokens,
            "window_tokens": d.window_tokens, "rope_pairs": list(d.rope_pairs), "seed": 1,
            "attend_partition": args.partition,
        },
        "attend": {
            "ms": round(att_ms, 4),
            "tflops": round(W["attend"] / (att_ms / 1e3) / 1e12, 2),
            "mfma_frac": round(W["attend"] / (att_ms / 1e3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
        },
        "cache_write": {
            "us": round(wr_s * 1e6, 3),
            "gbps": round(W["write_bytes"] / wr_s / 1e9, 1),
            "hbm_frac": round(W["write_bytes"] / wr_s / 1e9 / HBM_PEAK_GBPS, 4),
            "warm_infinity_cache_us": round(warm_mall_us, 3),
            "weights": "packed once (videomla_prepare_write_weights)",
            "plain_weights_us": round(plain_us, 3),
        },
        "kernels": {k: {"launches": v["launches"], "avg_us": round(v["avg_us"], 3)}
                    for k, v in kernels.items()},
        "kernels_pass": "a second pass of the same steps with every kernel bracketed by events; "
                        "the timed region brackets latent_attend only",
        "latent_attend_even_split": {"avg_us": round(even_s * 1e6, 3),
                                     "frac": round(W["attend_core"] / even_s / 1e12
                                                   / MFMA_BF16_PEAK_TFLOPS, 4)},
        "roofline": {
            "kernel": "latent_attend",
            "bound": "mfma",
            "achieved": round(k3_tflops, 2),
            "avg_us": round(k3_s * 1e6, 3),
            "launches": n_k3,
            "peak": round(MFMA_BF16_PEAK_TFLOPS, 1),
            "unit": "TFLOP/s",
            "frac": round(k3_tflops / MFMA_BF16_PEAK_TFLOPS, 4),
            "traffic": attend_traffic(),
        },
    }
    if frozen_out is not None:
        result["frozen_repeat_bitwise_equal"] = repeat_ok
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        del xs
        result["cpu_baseline"] = cpu_baseline(d)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
