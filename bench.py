"""Benchmark of the MI355X fused W4A16 routed-expert layer on one GPU.

    python bench.py [--steps K] [--warmup W] [--workload decode|prefill] [--no-cpu-baseline]

A step is one full layer call (route, group, grouped gate/up+SwiGLU, grouped
down, combine) on OLMoE-shaped synthetic inputs (d_model 2048, d_ff 1024,
64 experts, top-8; weights ~N(0, 0.02) as bf16, quantized once to int4
group-128 before timing; activations ~N(0, 1)).  Prints one JSON line.

decode  : 1 token, all 64 experts resident; 16 distinct expert banks are
          rotated step by step so the 26 MB working set cannot sit in the
          256 MB last-level cache across steps.  value = algorithmic HBM GB/s.
prefill : 2048 tokens (16,384 token-expert pairs), all experts resident.
          value = expert TFLOP/s.
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


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=None)
    p.add_argument("--warmup", type=int, default=None)
    p.add_argument("--workload", default="decode", choices=["decode", "prefill"])
    p.add_argument("--no-cpu-baseline", action="store_true")
    return p.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def record_bytes():
    return 3 * D_MODEL * D_FF // 2 + 3 * D_MODEL * D_FF // 64


def w13_bytes():
    return D_FF * D_MODEL + D_FF * D_MODEL // 32


def w2_bytes():
    return D_MODEL * D_FF // 2 + D_MODEL * D_FF // 64


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
    calls, t0 = 0, time.perf_counter()
    y = None
    while True:
        for ex in experts.values():
            ex._hat.clear()          # dequantize again each call, as the GPU path does
        rr = O.route(hf, wrf, k)
        y = O.moe_forward(hf, experts, rr)
        calls += 1
        el = time.perf_counter() - t0
        if el >= budget_s or calls >= 1000:
            break
    per_call = el / calls
    value = alg_bytes / per_call / 1e9 if unit == "GB/s" else flops / per_call / 1e12
    return y, dict(value=value, unit=unit, cores=int(threads), kind="oracle",
                   sample=f"{calls} full layer calls of this workload ({hf.shape[0]} token(s)), "
                          f"{el:.1f} s, numpy fp64 with dequantization each call",
                   seconds_per_call=per_call)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(the layer runs on a single device).", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2608_15383_amd import api

    torch.cuda.init()
    dm = api.dims(D_MODEL, D_FF, N_EXPERTS, TOP_K)
    decode = args.workload == "decode"
    T = 1 if decode else 2048
    steps = args.steps or (400 if decode else 50)
    warmup = args.warmup if args.warmup is not None else (40 if decode else 5)
    n_banks = 16 if decode else 2
    log(f"workload={args.workload} T={T} banks={n_banks} steps={steps} warmup={warmup}")

    gen = torch.Generator(device="cuda").manual_seed(7)
    wr = (torch.randn((N_EXPERTS, D_MODEL), dtype=torch.bfloat16, device="cuda", generator=gen) * 0.02)
    h = torch.randn((T, D_MODEL), dtype=torch.bfloat16, device="cuda", generator=gen)
    y = torch.empty_like(h)
    ws = torch.empty(api.workspace_bytes(dm, T), dtype=torch.uint8, device="cuda")

    banks, caches, keep_weights = [], [], None
    for b in range(n_banks):
        bank, cache, weights = make_bank(api, dm, torch, 1000 + b)
        banks.append(bank)
        caches.append(cache)
        if b == 0 and not args.no_cpu_baseline:
            keep_weights = tuple(w.view(torch.int16).cpu().numpy().view(np.uint16) for w in weights)
        del weights
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    log("banks ready")

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
    log(f"timed {steps} steps: {ms * 1e3:.2f} us/step")

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
        k_bytes = n_distinct * w2_bytes() + P * D_FF * 2 + P * D_MODEL * 4
        k_flops = P * 2 * D_FF * D_MODEL
    else:
        k_bytes, k_flops = alg_bytes, flops
    if decode or "gemv" in dominant:
        ach = k_bytes / dur_s / 1e9
        roof = dict(bound="hbm", achieved=ach, peak=HBM_PEAK_GBS, unit="GB/s", frac=ach / HBM_PEAK_GBS,
                    traffic=None, kernel=dominant, alg_bytes_per_launch=k_bytes)
    else:
        ach = k_flops / dur_s / 1e12
        roof = dict(bound="mfma", achieved=ach, peak=BF16_PEAK_TFLOPS, unit="TFLOP/s",
                    frac=ach / BF16_PEAK_TFLOPS, traffic=None, kernel=dominant,
                    alg_flops_per_launch=k_flops)

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

    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        api.moe_forward(caches[0], h, wr, y, ws)
        torch.cuda.synchronize()
        y0 = y.view(torch.int16).cpu().numpy().view(np.uint16)
        h_np = h.view(torch.int16).cpu().numpy().view(np.uint16)
        wr_np = wr.view(torch.int16).cpu().numpy().view(np.uint16)
        if not decode:
            h_np = h_np[:8]            # bounded sample: 8 of the 2048 tokens
        yref, cpu = oracle_baseline(keep_weights, wr_np, h_np, TOP_K,
                                    alg_bytes if decode else None,
                                    8 * TOP_K * (flops // P), unit)
        from paper_2608_15383_amd.inputs import bf16_bits_to_f32
        yg = bf16_bits_to_f32(y0[:h_np.shape[0]]).astype(np.float64)
        out["parity_max_rel_err"] = float(np.abs(yg - yref).max() / np.abs(yref).max())
        if not decode:
            cpu["sample"] += "; 8 tokens of the 2048-token batch"
        out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
