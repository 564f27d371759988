"""Phase timestamps of the fused decode launch, for measurement.

    python -m paper_2608_15383_amd.phase_trace --build          # compile the traced library
    python -m paper_2608_15383_amd.phase_trace [--tokens 1,4]   # run it on the GPU, print tables

The traced library is the product sources compiled with -DEMOE_PHASE_TRACE into
_build/trace/: every workgroup of a fused launch reads the wall clock (100 MHz) as it passes
its phases, keeps the readings in LDS and copies them out as it exits (decode.hip,
EMOE_PHASE).  For each token count the run makes 300 warm-up and 400 timed layer calls on 16
rotating resident OLMoE-shaped banks (d_model 2048, d_ff 1024, 64 experts, top-8), then reads
the timestamps of the last call and prints, per role and phase, min / median / p90 / max in
microseconds after the earliest workgroup start.  The clock reads and the copy-out cost a
little time (the per-call figure is printed beside the tables).
"""
from __future__ import annotations

import argparse
import ctypes as C
import os
import sys

import numpy as np

from . import _lib
from . import build as _build

TRACE_DIR = os.path.join(_build.BUILD, "trace")
TRACE_LIB = os.path.join(TRACE_DIR, "libexactmoe_trace.so")


def build_traced() -> str:
    return _build.build(defines=("EMOE_PHASE_TRACE",), lib=TRACE_LIB, objdir=TRACE_DIR)


def _stat(name, ticks, base):
    v = (ticks[ticks > 0] - base) / 100.0
    if len(v) == 0:
        return
    print(f"  {name:34s} min {v.min():7.2f}  med {np.median(v):7.2f}  p90 "
          f"{np.percentile(v, 90):7.2f}  max {v.max():7.2f}")


def trace(tokens: int, banks: int = 16):
    import torch
    from . import api
    dm = api.dims(2048, 1024, 64, 8)
    g = torch.Generator(device="cuda").manual_seed(1)
    kw = dict(dtype=torch.bfloat16, device="cuda", generator=g)
    caches, bank_mem = [], []
    for _ in range(banks):
        wg = torch.randn((64, 1024, 2048), **kw) * 0.02
        wu = torch.randn((64, 1024, 2048), **kw) * 0.02
        wd = torch.randn((64, 2048, 1024), **kw) * 0.02
        bank = torch.empty(64 * api.expert_record_bytes(dm), dtype=torch.uint8, device="cuda")
        api.quantize_experts(dm, wg, wu, wd, bank)
        del wg, wu, wd
        c = api.Cache(dm, 64, slot_bank=bank)
        c.preload_all()
        caches.append(c)
        bank_mem.append(bank)
    wr = torch.randn((64, 2048), **kw) * 0.02
    h = torch.randn((tokens, 2048), **kw)
    y = torch.empty_like(h)
    ws = torch.empty(api.workspace_bytes(dm, tokens), dtype=torch.uint8, device="cuda")
    for i in range(300):
        api.moe_forward(caches[i % banks], h, wr, y, ws)
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for i in range(400):
        api.moe_forward(caches[i % banks], h, wr, y, ws)
    t1.record()
    torch.cuda.synchronize()
    per_call = t0.elapsed_time(t1) / 400 * 1e3
    lib = _lib.lib()
    fn = lib.emoe_debug_phase_trace
    fn.argtypes, fn.restype = [C.c_void_p, C.c_int32], C.c_int32
    n_max = 1024
    tr = np.zeros(n_max * 16, np.uint64)
    assert fn(tr.ctypes.data, n_max) == 0
    tr = tr.reshape(n_max, 16).astype(np.int64)
    w0, w1 = int(tr[0, 14]), int(tr[0, 15])
    n_router, n_gate, n_work = w0 & 0xffff, (w0 >> 16) & 0xffff, (w0 >> 32) & 0xffff
    ppi, down_r, tail_r = w1 & 0xffff, (w1 >> 16) & 0xffff, (w1 >> 32) & 0xffff
    lag, tail_pairs = (w1 >> 48) & 0xff, (w1 >> 56) & 0xff
    n = n_router + n_work
    tr = tr[:n]
    base = tr[:, 0].min()
    chunks = -(-(1024 // 16) // ppi)
    j = np.arange(n) - n_router
    gate = (j >= 0) & (j < n_gate)
    tail = j >= n_gate
    k = 8
    per_pair = -(-(2048 // 16) // tail_r)
    # The pair whose down row blocks a worker computes.
    P = tokens * k
    gate_pair = j // max(chunks, 1) - lag
    down_pair = np.where(gate, np.where(gate_pair < P - tail_pairs, gate_pair, -1),
                         P - tail_pairs + (j - n_gate) // per_pair)
    down_gate = gate & (down_pair >= 0)
    comb = (down_gate | tail) & (down_pair % k == k - 1)
    print(f"T={tokens}: {per_call:.2f} us per layer call (traced build); grid {n} workgroups: "
          f"{n_router} router, {n_gate} gate/up workers ({ppi} row-block pair(s) each, then "
          f"{down_r} down row block(s) of the pair {lag} before, none in the last "
          f"{tail_pairs - lag} pair(s)), {n_work - n_gate} tail workers ({tail_r} row block(s) "
          f"each of the last {tail_pairs} pair(s))")
    R = tr[:n_router]
    print(" router workgroups")
    _stat("start", R[:, 0], base)
    _stat("logits stored", R[:, 1], base)
    print(" gate/up workers")
    _stat("start", tr[gate, 0], base)
    if tokens == 1:
        _stat("logits seen (wavefront 0)", tr[gate, 1], base)
    _stat("top-k done", tr[gate, 2], base)
    _stat("gate/up item done (activations out)", tr[gate, 4], base)
    for name, sel in (("gate/up workers, down part", down_gate), ("tail workers", tail)):
        print(f" {name}")
        _stat("down part reached", tr[sel, 3], base)
        _stat("activation row staged", tr[sel, 5], base)
        _stat("down tiles computed", tr[sel, 6], base)
        _stat("end", tr[sel, 9], base)
    print(" combining workers (last pair of a token)")
    _stat("other outputs of the token seen", tr[comb, 7], base)
    _stat("end", tr[comb, 9], base)
    print(f" bounded waits that gave up: {sum(c.sync_timeouts() for c in caches)}")
    for c in caches:
        c.close()


def main():
    p = argparse.ArgumentParser()
    p.add_argument("--build", action="store_true", help="compile the traced library and exit")
    p.add_argument("--tokens", default="1,4")
    args = p.parse_args()
    if args.build:
        print(build_traced())
        return
    if not os.path.exists(TRACE_LIB):
        sys.exit(f"{TRACE_LIB} is missing: run `python -m paper_2608_15383_amd.phase_trace --build`")
    import torch  # HIP runtime before the library, as elsewhere
    torch.cuda.init()
    _lib.LIB_PATH = TRACE_LIB
    for t in (int(x) for x in args.tokens.split(",")):
        trace(t)


if __name__ == "__main__":
    main()
