"""Helpers of the GPU parity tests: device upload, the library calls, and a
lazily quantized oracle expert bank."""
from __future__ import annotations

import numpy as np
import torch

import oracle as O
from paper_2608_15383_amd import api
from paper_2608_15383_amd.inputs import bf16_bits_to_f32

TOL = 2e-2  # max|y - y_ref| <= TOL * max|y_ref|


def dev(a: np.ndarray) -> torch.Tensor:
    """Upload a uint16 (bf16 bits) / int32 / float32 numpy array to cuda:0."""
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda:0")


def host_bits(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


def quantize(dm: api.Dims, lay, experts=None) -> torch.Tensor:
    """GPU-quantize the layer's experts into a packed bank (device uint8)."""
    sel = slice(None) if experts is None else experts
    wg, wu, wd = dev(lay.w_gate[sel]), dev(lay.w_up[sel]), dev(lay.w_down[sel])
    n = wg.shape[0]
    rec = torch.empty(n * api.expert_record_bytes(dm), dtype=torch.uint8, device="cuda:0")
    api.quantize_experts(dm, wg, wu, wd, rec)
    torch.cuda.synchronize()
    return rec


class LazyExperts:
    """experts[e] -> oracle QuantizedExpert, quantized on first use (oracle only)."""

    def __init__(self, lay):
        self.lay = lay
        self.cache = {}

    def __getitem__(self, e):
        e = int(e)
        if e not in self.cache:
            self.cache[e] = O.quantize_expert(bf16_bits_to_f32(self.lay.w_gate[e]),
                                              bf16_bits_to_f32(self.lay.w_up[e]),
                                              bf16_bits_to_f32(self.lay.w_down[e]))
        return self.cache[e]


def dims_of(shape) -> api.Dims:
    return api.dims(shape.d_model, shape.d_ff, shape.n_experts, shape.top_k)


def assert_close_rel(y, ref, label=""):
    """max|y - ref| <= TOL * max|ref| (prints both error measures)."""
    mx, mean = rel_err(y, ref)
    print(f"{label}: max|err|/max|ref| = {mx:.3e}, mean rel = {mean:.3e}", flush=True)
    assert mx <= TOL, (label, mx)


def rel_err(y: np.ndarray, ref: np.ndarray):
    """(max|err| / max|ref|, mean|err| / mean|ref|)."""
    err = np.abs(y.astype(np.float64) - ref)
    return float(err.max() / np.abs(ref).max()), float(err.mean() / np.abs(ref).mean())


class Layer:
    """A fully resident layer on the GPU (C = E, Sec. 3.3) plus its workspace."""

    def __init__(self, dm: api.Dims, lay, max_tokens: int):
        self.dm = dm
        self.lay = lay
        self.bank = quantize(dm, lay)
        self.cache = api.Cache(dm, dm.n_experts, slot_bank=self.bank)
        self.cache.preload_all()
        self.wr = dev(lay.w_router)
        self.ws = torch.empty(api.workspace_bytes(dm, max_tokens), dtype=torch.uint8, device="cuda:0")
        self.tokens = 0

    def forward(self, h_bits: np.ndarray, logits=None, path=api.EMOE_PATH_AUTO, renormalize=True,
                cache=None, sequential=False, stats=None):
        h = dev(h_bits)
        self.tokens = h.shape[0]
        y = torch.empty_like(h)
        lo = None if logits is None else dev(np.asarray(logits, np.float32))
        api.moe_forward(cache or self.cache, h, self.wr, y, self.ws, logits_override=lo,
                        renormalize=renormalize, path=path, stats=stats, sequential=sequential)
        torch.cuda.synchronize()
        return bf16_bits_to_f32(host_bits(y))

    def pair_out(self, pairs: int, mfma: bool) -> np.ndarray:
        """Pair outputs of the last call as float32 [pairs][d_model] (the MFMA
        path stores them in bf16, the GEMV path in fp32)."""
        d = self.dm.d_model
        if mfma:
            return bf16_bits_to_f32(self.ws_array("pair_out", pairs * d, np.uint16)).reshape(pairs, d)
        return self.ws_array("pair_out", pairs * d, np.float32).reshape(pairs, d)

    def ws_array(self, name: str, count: int, dtype) -> np.ndarray:
        """Copy of a workspace array written by the last forward call."""
        off = getattr(api.workspace_layout(self.dm, self.tokens), name)
        nbytes = count * np.dtype(dtype).itemsize
        return self.ws[off:off + nbytes].cpu().numpy().view(dtype).copy()
