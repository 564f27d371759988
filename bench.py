"""Benchmark of the MI355X fused W4A16 routed-expert layer on one GPU.

    python bench.py [--steps K] [--warmup W]
                    [--workload decode|prefill|multiwave|stack|frontier|copy] [--no-cpu-baseline]

A step is one full layer call (route, group, grouped gate/up+SwiGLU, grouped
down, combine) on OLMoE-shaped synthetic inputs (d_model 2048, d_ff 1024,
64 experts, top-8; weights ~N(0, 0.02) as bf16, quantized once to int4
group-128 before timing; activations ~N(0, 1)).  Prints one JSON line.

decode  : 1 token, all 64 experts resident; 16 distinct expert banks are
          rotated step by step so the 26 MB working set cannot sit in the
          256 MB last-level cache across steps.  value = algorithmic HBM GB/s.
prefill : 2048 tokens (16,384 token-expert pairs), all experts resident.
          value = expert TFLOP/s.
multiwave: 16 tokens through a 16-slot cache backed by a pinned host bank of
          the 64 packed experts; routing logits select 40/48/56/64 distinct
          experts (3-4 waves).  Fused and per-expert sequential paths, cold
          (empty slots) and warm (experts 0-15 resident), end to end (fills
          included) and kernels only.  value = fused warm tokens/s at 56
          experts.
stack   : 16 layers x 64 experts (1024 packed records in one pinned host
          bank), a 16-slot cache per layer, 64 tokens per step, Zipf(1.1)
          expert popularity per layer (Gumbel top-8).  value = tokens/s over
          32 steps of 16 layer calls; H2D bytes and hit rates reported.
frontier: the stack's capacity and batch frontier: C in {8, 16, 32, 64} slots
          per layer and T in {1, 2, 4, 8} tokens per step (C = 64: every
          expert resident).  Tokens/s, hit rate and H2D bytes per token for
          each point; value = tokens/s at C = 16, T = 1.
decoder : synthetic OLMoE-shaped decoder (16 layers of attention + this layer,
          random weights): time to first token for a 128-token prompt and greedy
          decode tokens/s over 128 generated tokens, at 64 and 16 slots per
          layer.  value = decode tokens/s at 64 slots.
copy    : calibration only (not a layer): a plain 1 GiB device-to-device copy of
          known size, so hardware byte counters (FETCH_SIZE, WRITE_SIZE) read on
          the layer kernels can be scaled to bytes.  value = copy GB/s.
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

METRIC = "fused W4A16 MoE layer: HBM GB/s + tokens/s (decode), TFLOP/s (prefill)"
D_MODEL, D_FF, N_EXPERTS, TOP_K = 2048, 1024, 64, 8
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_olmoe.md")
# Source files each measured kernel is built from: a traffic figure read with
# the hardware counters is reported only while these files are unchanged.
KERNEL_SOURCES = {
    "decode_fused": ["common.h", "decode.h", "decode.hip", "device_gemv.h", "device_route.h"],
    "decode_fused_t4": ["common.h", "decode.h", "decode.hip", "device_gemv.h", "device_route.h"],
    "gateup_mfma": ["common.h", "gemm.hip"],
    "down_mfma": ["common.h", "gemm.hip"],
}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=None)
    p.add_argument("--warmup", type=int, default=None)
    p.add_argument("--workload", default="decode",
                   choices=["decode", "decode_t4", "prefill", "multiwave", "stack", "frontier",
                            "decoder", "copy"])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-prefill", action="store_true",
                   help="decode only: skip the prefill sub-record")
    p.add_argument("--no-t4", action="store_true",
                   help="decode only: skip the 4-token decode sub-record")
    return p.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def record_bytes():
    return 3 * D_MODEL * D_FF // 2 + 3 * D_MODEL * D_FF // 64


def w13_bytes():
    return D_FF * D_MODEL + D_FF * D_MODEL // 32


def w2_bytes():
    return D_MODEL * D_FF // 2 + D_MODEL * D_FF // 64


def source_digest(kernel):
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2608_15383_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the FETCH_SIZE / WRITE_SIZE
    passes recorded in profiles/hbm_traffic_olmoe.md (scaled by the copy
    calibration there), or None when the kernel has no record or its sources
    changed since the counters were read."""
    if kernel not in KERNEL_SOURCES or not os.path.exists(TRAFFIC_FILE):
        return None
    with open(TRAFFIC_FILE) as f:
        for line in f:
            parts = line.split()
            if len(parts) == 4 and parts[0] == "traffic" and parts[1] == kernel:
                return int(parts[2]) if parts[3] == source_digest(kernel) else None
    return None


def make_bank(api, dm, torch, seed):
    """Random bf16 weights on the GPU, quantized into a resident 64-expert bank."""
    g = torch.Generator(device="cuda").manual_seed(seed)
    kw = dict(dtype=torch.bfloat16, device="cuda", generator=g)
    wg = torch.randn((N_EXPERTS, D_FF, D_MODEL), **kw) * 0.02
    wu = torch.randn((N_EXPERTS, D_FF, D_MODEL), **kw) * 0.02
    wd = torch.randn((N_EXPERTS, D_MODEL, D_FF), **kw) * 0.02
    bank = torch.empty(N_EXPERTS * api.expert_record_bytes(dm), dtype=torch.uint8, device="cuda")
    api.quantize_experts(dm, wg, wu, wd, bank)
    cache = api.Cache(dm, N_EXPERTS, slot_bank=bank)
    cache.preload_all()
    return bank, cache, (wg, wu, wd)


def oracle_baseline(weights, wr, h, k, alg_bytes, flops, unit, budget_s=12.0):
    """Time the CPU oracle (as it stands) on a bounded sample of the same workload."""
    import oracle as O
    from paper_2608_15383_amd.inputs import bf16_bits_to_f32
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        threads = 1
    wg, wu, wd = weights
    hf = bf16_bits_to_f32(h)
    wrf = bf16_bits_to_f32(wr)
    r = O.route(hf, wrf, k)
    needed = sorted(set(r.ids.reshape(-1).tolist()))
    experts = {e: O.quantize_expert(bf16_bits_to_f32(wg[e]), bf16_bits_to_f32(wu[e]),
                                    bf16_bits_to_f32(wd[e])) for e in needed}
    out = {}

    def call():
        for ex in experts.values():
            ex._hat.clear()          # dequantize again each call, as the GPU path does
        out["y"] = O.moe_forward(hf, experts, O.route(hf, wrf, k))

    calls, el = timed_calls(call, budget_s)
    per_call = el / calls
    value = alg_bytes / per_call / 1e9 if unit == "GB/s" else flops / per_call / 1e12
    res = dict(value=value, unit=unit, cores=int(threads), kind="oracle",
               sample=f"{calls} full layer calls of this workload ({hf.shape[0]} token(s)), "
                      f"{el:.1f} s, numpy fp64 with dequantization each call",
               seconds_per_call=per_call)
    one = single_thread_rate(call, budget_s / 2)
    if one is not None:
        c1, e1 = one
        per1 = e1 / c1
        res["single_thread"] = dict(
            value=alg_bytes / per1 / 1e9 if unit == "GB/s" else flops / per1 / 1e12,
            cores=1, sample=f"{c1} calls, {e1:.1f} s, BLAS and OpenMP pools limited to 1 thread")
    return out["y"], res


def timed_calls(call, budget_s):
    """Run call() until budget_s has passed (at most 1000 calls); (calls, seconds)."""
    calls, t0 = 0, time.perf_counter()
    while True:
        call()
        calls += 1
        el = time.perf_counter() - t0
        if el >= budget_s or calls >= 1000:
            return calls, el


def single_thread_rate(call, budget_s):
    """The same oracle calls with every thread pool held to one thread, or None."""
    try:
        from threadpoolctl import threadpool_limits
    except Exception:
        return None
    with threadpool_limits(limits=1):
        return timed_calls(call, budget_s)


def measure_resident(api, torch, dm, T, steps, warmup, n_banks, keep_first_weights=False,
                     prebuilt=None):
    """Time T-token layer calls over n_banks fully resident expert banks
    (rotated call by call) and the dominant kernel of a separate profiled
    pass.  Returns a dict (and bank-0 weights when asked, for the oracle).
    prebuilt: (banks, caches) of an earlier call, reused instead of new banks."""
    gen = torch.Generator(device="cuda").manual_seed(7)
    wr = (torch.randn((N_EXPERTS, D_MODEL), dtype=torch.bfloat16, device="cuda", generator=gen) * 0.02)
    h = torch.randn((T, D_MODEL), dtype=torch.bfloat16, device="cuda", generator=gen)
    y = torch.empty_like(h)
    ws = torch.empty(api.workspace_bytes(dm, T), dtype=torch.uint8, device="cuda")
    banks, caches, keep_weights = [], [], None
    if prebuilt is not None:
        banks, caches = prebuilt
        n_banks = len(caches)
    for b in range(n_banks if prebuilt is None else 0):
        bank, cache, weights = make_bank(api, dm, torch, 1000 + b)
        banks.append(bank)
        caches.append(cache)
        if b == 0 and keep_first_weights:
            keep_weights = tuple(w.view(torch.int16).cpu().numpy().view(np.uint16) for w in weights)
        del weights
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    log(f"T={T}: {n_banks} banks ready")

    # routing of this workload (identical across banks: same h and router)
    api.moe_forward(caches[0], h, wr, y, ws)
    torch.cuda.synchronize()
    L = api.workspace_layout(dm, T)
    counts = ws[L.counts:L.counts + 4 * N_EXPERTS].cpu().numpy().view(np.int32)
    n_distinct = int((counts > 0).sum())
    P = T * TOP_K
    alg_bytes = (n_distinct * record_bytes() + N_EXPERTS * D_MODEL * 2 + 2 * T * D_MODEL * 2)
    flops = P * (2 * D_MODEL * 2 * D_FF + 2 * D_FF * D_MODEL)

    def run(n):
        for i in range(n):
            api.moe_forward(caches[i % n_banks], h, wr, y, ws)

    run(warmup)
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    run(steps)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    log(f"T={T}: timed {steps} steps: {ms * 1e3:.2f} us/step")

    # per-kernel durations with HIP events on the launch stream (separate pass)
    api.profile_begin(8 * steps)
    run(steps)
    prof = api.profile_end(8 * steps)
    per_kernel = {}
    for name, t in prof:
        per_kernel.setdefault(name, []).append(t)
    kern = {n: dict(avg_us=1e3 * float(np.mean(v)), launches=len(v)) for n, v in per_kernel.items()}
    dominant = max(kern, key=lambda n: kern[n]["avg_us"] * kern[n]["launches"])
    dur_s = kern[dominant]["avg_us"] * 1e-6
    if dominant.startswith("gateup"):
        k_bytes = n_distinct * w13_bytes() + T * D_MODEL * 2 + P * D_FF * 2
        k_flops = P * 2 * D_MODEL * 2 * D_FF
    elif dominant.startswith("down"):
        out_bytes = 2 if dominant.endswith("mfma") else 4  # bf16 / fp32 pair outputs
        k_bytes = n_distinct * w2_bytes() + P * D_FF * 2 + P * D_MODEL * out_bytes
        k_flops = P * 2 * D_FF * D_MODEL
    else:
        k_bytes, k_flops = alg_bytes, flops
    # the fused decode kernel's counters are recorded per token count
    tkey = f"{dominant}_t{T}" if dominant == "decode_fused" and T != 1 else dominant
    if T <= 4 or "gemv" in dominant:
        ach = k_bytes / dur_s / 1e9
        roof = dict(bound="hbm", achieved=ach, peak=HBM_PEAK_GBS, unit="GB/s", frac=ach / HBM_PEAK_GBS,
                    traffic=measured_traffic(tkey), kernel=dominant,
                    alg_bytes_per_launch=k_bytes)
    else:
        ach = k_flops / dur_s / 1e12
        roof = dict(bound="mfma", achieved=ach, peak=BF16_PEAK_TFLOPS, unit="TFLOP/s",
                    frac=ach / BF16_PEAK_TFLOPS, traffic=measured_traffic(dominant), kernel=dominant,
                    alg_flops_per_launch=k_flops, alg_bytes_per_launch=k_bytes)
    return dict(ms=ms, kern=kern, roofline=roof, n_distinct=n_distinct, alg_bytes=alg_bytes,
                flops=flops, caches=caches, banks=banks, h=h, wr=wr, y=y, ws=ws,
                keep_weights=keep_weights, run=run)


def timeouts_of(caches):
    """Bounded device waits of the fused decode launch that gave up (must be 0)."""
    return int(sum(c.sync_timeouts() for c in caches))


def bench_layer(args):
    import torch
    from paper_2608_15383_amd import api

    torch.cuda.init()
    dm = api.dims(D_MODEL, D_FF, N_EXPERTS, TOP_K)
    decode = args.workload in ("decode", "decode_t4")
    T = 4 if args.workload == "decode_t4" else 1 if decode else 2048
    steps = args.steps or (400 if decode else 50)
    warmup = args.warmup if args.warmup is not None else (40 if decode else 5)
    n_banks = 16 if decode else 2
    log(f"workload={args.workload} T={T} banks={n_banks} steps={steps} warmup={warmup}")
    m = measure_resident(api, torch, dm, T, steps, warmup, n_banks,
                         keep_first_weights=not args.no_cpu_baseline)
    ms, kern, roof = m["ms"], m["kern"], m["roofline"]
    caches, h, wr, y, ws = m["caches"], m["h"], m["wr"], m["y"], m["ws"]
    alg_bytes, flops, n_distinct = m["alg_bytes"], m["flops"], m["n_distinct"]
    P = T * TOP_K

    sec = ms * 1e-3
    if decode:
        value, unit = alg_bytes / sec / 1e9, "GB/s"
    else:
        value, unit = flops / sec / 1e12, "TFLOP/s"
    out = dict(metric=METRIC, value=value, unit=unit, n_gpus=1, steps=steps, warmup=warmup,
               ms_per_step=ms, higher_is_better=True, scaling="weak", vs_baseline=None,
               dtype="bf16", data="synthetic",
               config=dict(workload=f"olmoe_{args.workload}", tokens=T, d_model=D_MODEL, d_ff=D_FF,
                           n_experts=N_EXPERTS, top_k=TOP_K, slots=N_EXPERTS, group=128,
                           weights="int4 group-128, fp16 scales", distinct_experts=n_distinct,
                           rotated_banks=n_banks),
               tokens_per_s=T / sec, alg_bytes_per_step=alg_bytes, flops_per_step=flops,
               roofline=roof, kernels=kern)
    if decode:
        # The same bytes against what a plain device copy achieves on this GPU.
        cp = device_copy_gbs(torch)
        out["device_copy"] = dict(gbs=cp, layer_frac=value / cp, kernel_frac=roof["achieved"] / cp)
        # One call per bank captured into a HIP graph and replayed.
        us, same = graph_replay(torch, lambda i: api.moe_forward(caches[i], h, wr, y, ws),
                                n_banks, max(steps // n_banks, 1), y)
        out["graph_replay"] = dict(us_per_call=us, gbs=alg_bytes / (us * 1e-6) / 1e9,
                                   calls_per_graph=n_banks, equals_eager=same)
        log(f"graph replay: {us:.2f} us per call, equal to eager: {same}")
        if T == 1 and not args.no_t4:
            out["decode_t4"] = decode_t4_record(api, torch, dm, m["banks"], caches)
    # Every bounded wait of the fused decode launch must have been met: a
    # timeout would mean some call's output is invalid (it is written as NaN).
    out["sync_timeouts"] = timeouts_of(caches)

    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        api.moe_forward(caches[0], h, wr, y, ws)
        torch.cuda.synchronize()
        y0 = y.view(torch.int16).cpu().numpy().view(np.uint16)
        h_np = h.view(torch.int16).cpu().numpy().view(np.uint16)
        wr_np = wr.view(torch.int16).cpu().numpy().view(np.uint16)
        if not decode:
            h_np = h_np[:8]            # bounded sample: 8 of the 2048 tokens
        yref, cpu = oracle_baseline(m["keep_weights"], wr_np, h_np, TOP_K,
                                    alg_bytes if decode else None,
                                    8 * TOP_K * (flops // P), unit)
        from paper_2608_15383_amd.inputs import bf16_bits_to_f32
        yg = bf16_bits_to_f32(y0[:h_np.shape[0]]).astype(np.float64)
        out["parity_max_rel_err"] = float(np.abs(yg - yref).max() / np.abs(yref).max())
        if not decode:
            cpu["sample"] += "; 8 tokens of the 2048-token batch"
        out["cpu_baseline"] = cpu
    del m, caches
    if T == 1 and not args.no_prefill:
        out["prefill"] = prefill_record(api, torch, dm)
    if out["sync_timeouts"]:
        print(json.dumps(out), file=sys.stderr, flush=True)
        sys.exit(f"{out['sync_timeouts']} bounded device waits gave up: results invalid")
    print(json.dumps(out), flush=True)


def decode_t4_record(api, torch, dm, banks, caches, steps=200, warmup=20):
    """Decode with four tokens per call (every expert resident, the same
    rotated banks): per-call time, tokens/s and the fused kernel's roofline."""
    m = measure_resident(api, torch, dm, 4, steps, warmup, len(caches), prebuilt=(banks, caches))
    sec = m["ms"] * 1e-3
    rec = dict(workload="olmoe_decode_t4", tokens=4, steps=steps, warmup=warmup,
               us_per_call=m["ms"] * 1e3, distinct_experts=m["n_distinct"],
               alg_bytes_per_call=m["alg_bytes"], gbs=m["alg_bytes"] / sec / 1e9,
               tokens_per_s=4 / sec, roofline=m["roofline"], kernels=m["kern"])
    log(f"decode T=4: {rec['us_per_call']:.2f} us per call, {rec['gbs']:.0f} GB/s")
    del m
    return rec


def prefill_record(api, torch, dm, steps=20, warmup=3):
    """The prefill half of the metric (2048 tokens, every expert resident):
    per-call time, expert TFLOP/s and the dominant MFMA kernel's roofline."""
    torch.cuda.empty_cache()
    m = measure_resident(api, torch, dm, 2048, steps, warmup, 2)
    sec = m["ms"] * 1e-3
    rec = dict(workload="olmoe_prefill", tokens=2048, steps=steps, warmup=warmup,
               us_per_call=m["ms"] * 1e3, tflops=m["flops"] / sec / 1e12,
               frac_of_bf16_peak=m["flops"] / sec / 1e12 / BF16_PEAK_TFLOPS,
               tokens_per_s=2048 / sec, flops_per_call=m["flops"], roofline=m["roofline"],
               kernels=m["kern"])
    log(f"prefill: {rec['us_per_call']:.1f} us per call, {rec['tflops']:.0f} TFLOP/s")
    del m
    torch.cuda.empty_cache()
    return rec


def quantized_host_bank(api, dm, torch, seeds):
    """Packed records of len(seeds) 64-expert layers in one pinned host bank."""
    rec = api.expert_record_bytes(dm)
    host = torch.empty(len(seeds) * N_EXPERTS * rec, dtype=torch.uint8, pin_memory=True)
    raw = []
    for li, seed in enumerate(seeds):
        bank, cache, weights = make_bank(api, dm, torch, seed)
        host[li * N_EXPERTS * rec:(li + 1) * N_EXPERTS * rec].copy_(bank)
        if li == 0:
            raw = weights
        cache.close()
        del bank, cache, weights
    torch.cuda.synchronize()
    return host, raw


def device_copy_gbs(torch, n_bytes=1 << 30, steps=5):
    """Bytes moved (read + written) per second by a plain device-to-device copy."""
    src = torch.ones(n_bytes // 2, dtype=torch.bfloat16, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        dst.copy_(src)
    torch.cuda.synchronize()
    gbs = 2 * n_bytes * steps / (time.perf_counter() - t0) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return gbs


def graph_replay(torch, call, n_calls, reps, y):
    """Capture call(0 .. n_calls-1) into one HIP graph and replay it `reps`
    times: (us per call, whether the last replay's y equals an eager call's)."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for i in range(n_calls):
            call(i)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    eager = y.clone()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(n_calls):
            call(i)
    graph.replay()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(reps):
        graph.replay()
    t1.record()
    torch.cuda.synchronize()
    same = bool(torch.equal(y, eager))
    del graph
    return t0.elapsed_time(t1) * 1e3 / (reps * n_calls), same


def pinned_h2d_gbs(torch, host):
    """Measured pinned host -> device copy bandwidth (hipMemcpyAsync)."""
    n = min(host.numel(), 256 << 20)
    dst = torch.empty(n, dtype=torch.uint8, device="cuda")
    dst.copy_(host[:n], non_blocking=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(4):
        dst.copy_(host[:n], non_blocking=True)
    torch.cuda.synchronize()
    return 4 * n / (time.perf_counter() - t0) / 1e9


def bench_multiwave(args):
    """16 tokens, 16 slots, 40-64 distinct experts: fused vs sequential waves."""
    import torch
    from paper_2608_15383_amd import api
    from paper_2608_15383_amd.inputs import spread_logits

    torch.cuda.init()
    dm = api.dims(D_MODEL, D_FF, N_EXPERTS, TOP_K)
    T, C = 16, 16
    reps = args.steps or 5
    rec = api.expert_record_bytes(dm)
    host, weights = quantized_host_bank(api, dm, torch, [1000])
    keep_weights = None
    if not args.no_cpu_baseline:
        keep_weights = tuple(w.view(torch.int16).cpu().numpy().view(np.uint16) for w in weights)
    del weights
    torch.cuda.empty_cache()
    h2d_gbs = pinned_h2d_gbs(torch, host)
    slots = torch.zeros(C * rec, dtype=torch.uint8, device="cuda")
    gen = torch.Generator(device="cuda").manual_seed(7)
    h = torch.randn((T, D_MODEL), dtype=torch.bfloat16, device="cuda", generator=gen)
    y = torch.empty_like(h)
    ws = torch.empty(api.workspace_bytes(dm, T), dtype=torch.uint8, device="cuda")
    log(f"multiwave: host bank ready, pinned H2D {h2d_gbs:.1f} GB/s")

    def one_call(z, state, sequential, profiled, overlap=False):
        """One call from a fresh cache in `state`: end-to-end seconds (host
        clock, fills included) of an unprofiled call, or the summed kernel
        seconds of a profiled one (dispatch-level events around each launch
        would otherwise inflate the many-launch sequential path's wall time)."""
        cache = api.Cache(dm, C, slot_bank=slots, host_bank=host)
        if state == "warm":
            _, fills = cache.build_slot_map(list(range(C)))
            cache.fill_slots(fills)
        cache.set_wave_overlap(overlap)
        torch.cuda.synchronize()
        st = api.Stats()
        if profiled:
            api.profile_begin(4096)
        t0 = time.perf_counter()
        api.moe_forward(cache, h, None, y, ws, logits_override=z, stats=st, sequential=sequential)
        torch.cuda.synchronize()
        sec = time.perf_counter() - t0
        if profiled:
            sec = sum(t for _, t in api.profile_end(4096)) * 1e-3
        cache.close()
        return sec, st, y.clone()

    cases, outs = [], {}
    for D in (40, 48, 56, 64):
        z = torch.from_numpy(spread_logits(T, N_EXPERTS, TOP_K, D, seed=2)).to("cuda")
        for state in ("cold", "warm"):
            row = dict(distinct_experts=D, state=state)
            for name, seq, ov in (("fused", False, False), ("fused_overlap", False, True),
                                  ("sequential", True, False)):
                one_call(z, state, seq, False, ov)           # warm-up of this case
                e2e, kern, k_sum = [], [], None
                for _ in range(reps):
                    a, st, yy = one_call(z, state, seq, False, ov)
                    e2e.append(a)
                    k_sum = st
                for _ in range(reps):
                    kern.append(one_call(z, state, seq, True, ov)[0])
                outs[(D, state, name)] = yy
                row[name] = dict(e2e_ms=1e3 * float(np.median(e2e)), kernel_ms=1e3 * float(np.median(kern)),
                                 waves=int(k_sum.waves), hits=int(k_sum.hits), misses=int(k_sum.misses),
                                 h2d_bytes=int(k_sum.h2d_bytes), kernel_launches=int(k_sum.kernel_launches))
            row["speedup_e2e"] = row["sequential"]["e2e_ms"] / row["fused"]["e2e_ms"]
            row["speedup_kernels"] = row["sequential"]["kernel_ms"] / row["fused"]["kernel_ms"]
            row["fused_equals_sequential"] = bool(torch.equal(outs[(D, state, "fused")],
                                                              outs[(D, state, "sequential")]))
            row["overlap_equals_fused"] = bool(torch.equal(outs[(D, state, "fused")],
                                                           outs[(D, state, "fused_overlap")]))
            row["overlap_speedup_e2e"] = row["fused"]["e2e_ms"] / row["fused_overlap"]["e2e_ms"]
            cases.append(row)
            log(f"D={D} {state}: fused {row['fused']['e2e_ms']:.2f} ms e2e / "
                f"{row['fused']['kernel_ms']:.3f} ms kernels, overlap "
                f"{row['fused_overlap']['e2e_ms']:.2f} ms e2e, sequential "
                f"{row['sequential']['e2e_ms']:.2f} / {row['sequential']['kernel_ms']:.3f} ms")
    head = next(c for c in cases if c["distinct_experts"] == 56 and c["state"] == "warm")
    sec = head["fused"]["e2e_ms"] * 1e-3
    kern_s = head["fused"]["kernel_ms"] * 1e-3
    alg = 56 * rec + 2 * T * D_MODEL * 2
    ach = alg / kern_s / 1e9
    out = dict(metric=METRIC, value=T / sec, unit="tokens/s", n_gpus=1, steps=reps, warmup=1,
               ms_per_step=1e3 * sec, higher_is_better=True, scaling="weak", vs_baseline=None,
               dtype="bf16", data="synthetic",
               config=dict(workload="olmoe_16tok_16slots_waves", tokens=T, d_model=D_MODEL, d_ff=D_FF,
                           n_experts=N_EXPERTS, top_k=TOP_K, slots=C, group=128,
                           weights="int4 group-128, fp16 scales", headline="56 experts, warm, fused"),
               roofline=dict(bound="hbm", achieved=ach, peak=HBM_PEAK_GBS, unit="GB/s",
                             frac=ach / HBM_PEAK_GBS, traffic=None,
                             kernel="all kernels of the fused call (fills excluded)",
                             alg_bytes_per_launch=alg),
               host_link=dict(pinned_h2d_gbs=h2d_gbs), cases=cases)
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        out["cpu_baseline"] = oracle_multiwave(keep_weights, T, head)
    print(json.dumps(out), flush=True)


def oracle_multiwave(weights, T, head, budget_s=12.0):
    """The CPU oracle on the 56-expert 16-token batch (single and multi-wave)."""
    import oracle as O
    from paper_2608_15383_amd.inputs import bf16_bits_to_f32, spread_logits
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        threads = 1
    wg, wu, wd = weights
    rng = np.random.default_rng(7)
    h = rng.standard_normal((T, D_MODEL)).astype(np.float32)
    z = spread_logits(T, N_EXPERTS, TOP_K, 56, seed=2)
    r = O.route(h, None, TOP_K, logits_override=z)
    needed = sorted(set(r.ids.reshape(-1).tolist()))
    experts = {e: O.quantize_expert(bf16_bits_to_f32(wg[e]), bf16_bits_to_f32(wu[e]),
                                    bf16_bits_to_f32(wd[e])) for e in needed}
    def call():
        for ex in experts.values():
            ex._hat.clear()
        O.moe_forward(h, experts, O.route(h, None, TOP_K, logits_override=z))

    calls, el = timed_calls(call, budget_s)
    res = dict(value=T * calls / el, unit="tokens/s", cores=int(threads), kind="oracle",
               sample=f"{calls} calls of the 16-token, 56-expert batch, {el:.1f} s, numpy fp64 "
                      f"with dequantization each call")
    one = single_thread_rate(call, budget_s / 2)
    if one is not None:
        res["single_thread"] = dict(value=T * one[0] / one[1], cores=1,
                                    sample=f"{one[0]} calls, {one[1]:.1f} s, thread pools limited to 1")
    return res


def bench_stack(args):
    """16 layers, 16 slots each, Zipf(1.1) routing, 64 tokens per step; waves of
    C (the paper's plan) and waves of C/2 with fills overlapping the previous
    wave's computation, each from empty caches over the same routing."""
    import torch
    from paper_2608_15383_amd import api
    from paper_2608_15383_amd.inputs import zipf_gumbel_logits

    torch.cuda.init()
    dm = api.dims(D_MODEL, D_FF, N_EXPERTS, TOP_K)
    L, T, C = 16, 64, 16
    steps = args.steps or 32
    warmup = args.warmup if args.warmup is not None else 4
    rec = api.expert_record_bytes(dm)
    log("stack: quantizing 16 x 64 experts into the pinned host bank")
    host, weights = quantized_host_bank(api, dm, torch, [2000 + l for l in range(L)])
    del weights
    torch.cuda.empty_cache()
    h2d_gbs = pinned_h2d_gbs(torch, host)
    banks = [torch.zeros(C * rec, dtype=torch.uint8, device="cuda") for _ in range(L)]
    rng = np.random.default_rng(4)
    perms = [rng.permutation(N_EXPERTS) for _ in range(L)]
    n_steps = warmup + steps
    z_all = np.stack([np.stack([zipf_gumbel_logits(T, N_EXPERTS, 1.1, perms[l], rng) for l in range(L)])
                      for _ in range(n_steps)])
    z_dev = torch.from_numpy(z_all).to("cuda")            # [steps][L][T][E]
    gen = torch.Generator(device="cuda").manual_seed(9)
    hs = [torch.randn((T, D_MODEL), dtype=torch.bfloat16, device="cuda", generator=gen) for _ in range(8)]
    y = torch.empty_like(hs[0])
    ws = torch.empty(api.workspace_bytes(dm, T), dtype=torch.uint8, device="cuda")
    log(f"stack ready: pinned H2D {h2d_gbs:.1f} GB/s")

    def hit_rate(x):
        tot = x.hits + x.misses
        return x.hits / tot if tot else 0.0

    def run_mode(overlap):
        caches = [api.Cache(dm, C, slot_bank=banks[l],
                            host_bank=host[l * N_EXPERTS * rec:(l + 1) * N_EXPERTS * rec])
                  for l in range(L)]
        for c in caches:
            c.set_wave_overlap(overlap)

        def step(s, st):
            for l in range(L):
                api.moe_forward(caches[l], hs[(s * L + l) % len(hs)], None, y, ws,
                                logits_override=z_dev[s, l], stats=st)

        first = api.Stats()
        step(0, first)
        torch.cuda.synchronize()
        for s in range(1, warmup):
            step(s, api.Stats())
        torch.cuda.synchronize()
        st = api.Stats()
        t0 = time.perf_counter()
        for s in range(warmup, n_steps):
            step(s, st)
        torch.cuda.synchronize()
        sec = time.perf_counter() - t0
        y_last = y.clone()
        api.profile_begin(1 << 16)
        step(warmup, api.Stats())
        prof = api.profile_end(1 << 16)
        for c in caches:
            c.close()
        kern = {}
        for name, t in prof:
            kern.setdefault(name, []).append(t)
        kern = {n: dict(avg_us=1e3 * float(np.mean(v)), launches=len(v)) for n, v in kern.items()}
        kernel_ms = sum(v["avg_us"] * v["launches"] for v in kern.values()) * 1e-3
        calls = steps * L
        achieved = st.h2d_bytes / sec / 1e9
        res = dict(tokens_per_s=T * steps / sec, ms_per_step=1e3 * sec / steps,
                   hit_rate_steady=hit_rate(st), hit_rate_cold_first_step=hit_rate(first),
                   h2d_bytes_per_layer_call=st.h2d_bytes / calls, waves_per_layer_call=st.waves / calls,
                   misses_per_layer_call=st.misses / calls, h2d_gbs_achieved=achieved,
                   host_link=dict(bound="host link", achieved=achieved, pinned_copy_gbs=h2d_gbs,
                                  frac=achieved / h2d_gbs),
                   kernels_ms_per_step=kernel_ms, kernels=kern,
                   dominant_kernel=max(kern, key=lambda n: kern[n]["avg_us"] * kern[n]["launches"]))
        log(f"overlap={overlap}: {res['tokens_per_s']:.0f} tokens/s, link {achieved:.1f} GB/s "
            f"({res['host_link']['frac']:.2f}), hit rate {res['hit_rate_steady']:.3f}, "
            f"{res['waves_per_layer_call']:.2f} waves per layer call")
        return res, y_last

    plain, y_plain = run_mode(False)
    over, y_over = run_mode(True)
    out = dict(metric=METRIC, value=over["tokens_per_s"], unit="tokens/s", n_gpus=1, steps=steps,
               warmup=warmup, ms_per_step=over["ms_per_step"], higher_is_better=True, scaling="weak",
               vs_baseline=None, dtype="bf16", data="synthetic",
               config=dict(workload="olmoe_stack16_zipf1.1_16slots", layers=L, tokens=T,
                           d_model=D_MODEL, d_ff=D_FF, n_experts=N_EXPERTS, top_k=TOP_K, slots=C,
                           group=128, weights="int4 group-128, fp16 scales", wave_overlap=True,
                           activations="8 pre-drawn N(0,1) token blocks cycled over layers and steps"),
               **{k: v for k, v in over.items() if k not in ("ms_per_step", "tokens_per_s")},
               no_overlap=plain, overlap_speedup=over["tokens_per_s"] / plain["tokens_per_s"],
               last_output_equal=bool(torch.equal(y_plain, y_over)))
    print(json.dumps(out), flush=True)


def bench_frontier(args):
    """Capacity and batch frontier of the 16-layer stack: C in {8, 16, 32, 64}
    slots per layer, T in {1, 2, 4, 8} tokens per step, Zipf(1.1) routing."""
    import torch
    from paper_2608_15383_amd import api
    from paper_2608_15383_amd.inputs import zipf_gumbel_logits

    torch.cuda.init()
    dm = api.dims(D_MODEL, D_FF, N_EXPERTS, TOP_K)
    L = 16
    steps = args.steps or 6
    warmup = args.warmup if args.warmup is not None else 2
    rec = api.expert_record_bytes(dm)
    log("frontier: quantizing 16 x 64 experts into the pinned host bank")
    host, weights = quantized_host_bank(api, dm, torch, [2000 + l for l in range(L)])
    del weights
    torch.cuda.empty_cache()
    rng = np.random.default_rng(4)
    perms = [rng.permutation(N_EXPERTS) for _ in range(L)]
    gen = torch.Generator(device="cuda").manual_seed(9)
    rows = []
    for C in (8, 16, 32, 64):
        banks = [torch.zeros(C * rec, dtype=torch.uint8, device="cuda") for _ in range(L)]
        caches = []
        for l in range(L):
            c = api.Cache(dm, C, slot_bank=banks[l],
                          host_bank=host[l * N_EXPERTS * rec:(l + 1) * N_EXPERTS * rec])
            if C == N_EXPERTS:
                c.preload_all()
            caches.append(c)
        for T in (1, 2, 4, 8):
            n_steps = warmup + steps
            z = torch.from_numpy(np.stack([np.stack([zipf_gumbel_logits(T, N_EXPERTS, 1.1, perms[l], rng)
                                                     for l in range(L)]) for _ in range(n_steps)])
                                 .astype(np.float32)).to("cuda")
            h = torch.randn((T, D_MODEL), dtype=torch.bfloat16, device="cuda", generator=gen)
            y = torch.empty_like(h)
            ws = torch.empty(api.workspace_bytes(dm, T), dtype=torch.uint8, device="cuda")

            def step(si, st):
                for l in range(L):
                    api.moe_forward(caches[l], h, None, y, ws, logits_override=z[si, l], stats=st)

            for si in range(warmup):
                step(si, api.Stats())
            torch.cuda.synchronize()
            st = api.Stats()
            t0 = time.perf_counter()
            for si in range(warmup, n_steps):
                step(si, st)
            torch.cuda.synchronize()
            sec = time.perf_counter() - t0
            tot = st.hits + st.misses
            row = dict(slots=C, tokens=T, tokens_per_s=T * steps / sec, ms_per_step=1e3 * sec / steps,
                       hit_rate=(st.hits / tot) if tot else 1.0,
                       h2d_mb_per_token=st.h2d_bytes / (T * steps) / 1e6,
                       h2d_gbs=st.h2d_bytes / sec / 1e9, waves_per_layer_call=st.waves / (steps * L),
                       slot_gib=L * C * rec / 2 ** 30)
            rows.append(row)
            log(f"C={C:2d} T={T}: {row['tokens_per_s']:8.1f} tokens/s, hit rate {row['hit_rate']:.2f}, "
                f"H2D {row['h2d_mb_per_token']:.1f} MB/token, {row['h2d_gbs']:.1f} GB/s")
        for c in caches:
            c.close()
        del caches, banks
        torch.cuda.empty_cache()
    head = next(r for r in rows if r["slots"] == 16 and r["tokens"] == 1)
    out = dict(metric=METRIC, value=head["tokens_per_s"], unit="tokens/s", n_gpus=1, steps=steps,
               warmup=warmup, ms_per_step=head["ms_per_step"], higher_is_better=True,
               scaling="weak", vs_baseline=None, dtype="bf16", data="synthetic",
               config=dict(workload="olmoe_stack16_zipf1.1_frontier", layers=L, d_model=D_MODEL,
                           d_ff=D_FF, n_experts=N_EXPERTS, top_k=TOP_K, group=128,
                           value_at=dict(slots=16, tokens=1),
                           weights="int4 group-128, fp16 scales"),
               frontier=rows)
    print(json.dumps(out), flush=True)


def bench_decoder(args):
    """Synthetic OLMoE-shaped decoder (16 layers of attention + the W4A16 layer,
    random weights) in the structure of the paper's runtime table: time to
    first token for a prompt and greedy decode tokens/s, at 64 slots per layer
    (every expert resident) and at 16 slots (pinned host bank of all 1024
    records).  The next token never leaves the GPU between steps."""
    import torch
    from paper_2608_15383_amd import api

    torch.cuda.init()
    L, H, Dh, V = 16, 16, 128, 50304
    prompt_len = 128
    gen_tokens = args.steps or 128
    reps = 3
    dm = api.dims(D_MODEL, D_FF, N_EXPERTS, TOP_K)
    dd = api.decoder_dims(L, H, Dh, V, prompt_len + gen_tokens + 1, dm)
    rec = api.expert_record_bytes(dm)
    g = torch.Generator(device="cuda").manual_seed(11)
    bf = dict(dtype=torch.bfloat16, device="cuda", generator=g)
    w = dict(embed=torch.randn((V, D_MODEL), **bf), lm_head=torch.randn((V, D_MODEL), **bf) * 0.02,
             final_norm=1 + torch.randn((D_MODEL,), **bf) * 0.1)
    w["attn_norm"] = [1 + torch.randn((D_MODEL,), **bf) * 0.1 for _ in range(L)]
    w["wqkv"] = [torch.randn((3 * D_MODEL, D_MODEL), **bf) * 0.02 for _ in range(L)]
    w["wo"] = [torch.randn((D_MODEL, D_MODEL), **bf) * 0.02 for _ in range(L)]
    w["moe_norm"] = [1 + torch.randn((D_MODEL,), **bf) * 0.1 for _ in range(L)]
    w["w_router"] = [torch.randn((N_EXPERTS, D_MODEL), **bf) * 0.02 for _ in range(L)]
    log("decoder: quantizing 16 x 64 experts")
    host, _ = quantized_host_bank(api, dm, torch, [3000 + l for l in range(L)])
    torch.cuda.empty_cache()
    prompt = torch.randint(0, V, (prompt_len,), dtype=torch.int32, device="cuda", generator=g)
    kv = torch.zeros(api.decoder_kv_bytes(dd), dtype=torch.uint8, device="cuda")
    ws = torch.empty(api.decoder_workspace_bytes(dd, prompt_len), dtype=torch.uint8, device="cuda")
    logits = torch.empty(V, dtype=torch.float32, device="cuda")
    toks = torch.empty(gen_tokens + 1, dtype=torch.int32, device="cuda")
    rows = []
    for C in (64, 16):
        banks = [torch.zeros(C * rec, dtype=torch.uint8, device="cuda") for _ in range(L)]
        caches = []
        for l in range(L):
            c = api.Cache(dm, C, slot_bank=banks[l],
                          host_bank=host[l * N_EXPERTS * rec:(l + 1) * N_EXPERTS * rec])
            if C == N_EXPERTS:
                c.preload_all()
            else:
                c.set_wave_overlap(True)
            caches.append(c)
        dec = api.Decoder(dd, w, caches, kv)
        ttft, tps, stats = [], [], api.Stats()
        for rep in range(reps + 1):           # the first repetition warms up
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            dec.forward(prompt, 0, logits, toks[0:1], ws)
            first = int(toks[0].item())       # the first token reaches the host
            t1 = time.perf_counter()
            st = api.Stats()
            for i in range(gen_tokens):
                dec.forward(toks[i:i + 1], prompt_len + i, logits, toks[i + 1:i + 2], ws, stats=st)
            torch.cuda.synchronize()
            t2 = time.perf_counter()
            if rep:
                ttft.append(t1 - t0)
                tps.append(gen_tokens / (t2 - t1))
                stats = st
        tot = stats.hits + stats.misses
        row = dict(slots=C, ttft_ms=1e3 * float(np.median(ttft)), decode_tokens_per_s=float(np.median(tps)),
                   ms_per_token=1e3 / float(np.median(tps)), prompt_tokens=prompt_len,
                   generated_tokens=gen_tokens, repetitions=reps, first_token=first,
                   hit_rate=(stats.hits / tot) if tot else None,
                   h2d_gib_per_request=stats.h2d_bytes / 2 ** 30,
                   slot_bank_gib=L * C * rec / 2 ** 30)
        rows.append(row)
        log(f"C={C}: TTFT {row['ttft_ms']:.2f} ms, decode {row['decode_tokens_per_s']:.1f} tokens/s, "
            f"hit rate {row['hit_rate']}, H2D {row['h2d_gib_per_request']:.2f} GiB per request")
        dec.close()
        for c in caches:
            c.close()
        del banks, caches
        torch.cuda.empty_cache()
    head = rows[0]
    out = dict(metric=METRIC, value=head["decode_tokens_per_s"], unit="tokens/s", n_gpus=1,
               steps=gen_tokens, warmup=1, ms_per_step=head["ms_per_token"], higher_is_better=True,
               scaling="weak", vs_baseline=None, dtype="bf16", data="synthetic",
               config=dict(workload="olmoe_synthetic_decoder", layers=L, heads=H, head_dim=Dh, vocab=V,
                           d_model=D_MODEL, d_ff=D_FF, n_experts=N_EXPERTS, top_k=TOP_K,
                           prompt_tokens=prompt_len, generated_tokens=gen_tokens,
                           value_at=dict(slots=64),
                           weights="random; experts int4 group-128 with fp16 scales, the rest bf16"),
               capacity=rows)
    print(json.dumps(out), flush=True)


def bench_copy(args):
    import torch

    torch.cuda.init()
    n = 1 << 29  # bf16 elements: 1 GiB read and 1 GiB written per copy
    src = torch.ones(n, dtype=torch.bfloat16, device="cuda")
    dst = torch.empty_like(src)
    steps = args.steps or 5
    for _ in range(args.warmup if args.warmup is not None else 1):
        dst.copy_(src)
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(steps):
        dst.copy_(src)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    nbytes = 2 * n
    print(json.dumps(dict(workload="copy", bytes_read_per_copy=nbytes, bytes_written_per_copy=nbytes,
                          ms_per_copy=ms, value=2 * nbytes / (ms * 1e-3) / 1e9, unit="GB/s",
                          steps=steps)), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(the layer runs on a single device).", file=sys.stderr)
        sys.exit(2)
    if args.workload == "multiwave":
        bench_multiwave(args)
    elif args.workload == "stack":
        bench_stack(args)
    elif args.workload == "copy":
        bench_copy(args)
    elif args.workload == "frontier":
        bench_frontier(args)
    elif args.workload == "decoder":
        bench_decoder(args)
    else:
        bench_layer(args)


if __name__ == "__main__":
    main()
