"""Thin Python binding of libexactmoe.so with the C ABI's names.

PyTorch only supplies device memory, pinned host memory and streams; every
step of the layer runs in the HIP library.  Tensors holding bf16 data may be
torch.bfloat16 or int16/uint16 bit patterns; they are passed by data_ptr().
"""
from __future__ import annotations

import ctypes as C

import numpy as np

from . import _lib
from ._lib import (DecoderDims, DecoderWeights, Dims, Stats, WsLayout, check, lib,
                   EMOE_PATH_AUTO, EMOE_PATH_GEMV, EMOE_PATH_MFMA, EMOE_PATH_MIXED,
                   EMOE_MIXED_MFMA_ROWS, ExactMoEError)


def _ptr(t) -> int | None:
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def dims(d_model: int, d_ff: int, n_experts: int, top_k: int) -> Dims:
    return Dims(d_model, d_ff, n_experts, top_k)


def check_dims(dm: Dims) -> None:
    check(lib().emoe_check_dims(C.byref(dm)))


def expert_record_bytes(dm: Dims) -> int:
    return int(lib().emoe_expert_record_bytes(C.byref(dm)))


def workspace_layout(dm: Dims, max_tokens: int) -> WsLayout:
    out = WsLayout()
    check(lib().emoe_workspace_layout(C.byref(dm), max_tokens, C.byref(out)))
    return out


def workspace_bytes(dm: Dims, max_tokens: int) -> int:
    return int(lib().emoe_workspace_bytes(C.byref(dm), max_tokens))


def quantize_experts(dm: Dims, w_gate, w_up, w_down, records, stream=None) -> None:
    """emoe_quantize_experts: device bf16 weights -> device packed records."""
    n = w_gate.shape[0]
    check(lib().emoe_quantize_experts(C.byref(dm), n, _ptr(w_gate), _ptr(w_up), _ptr(w_down),
                                      _ptr(records), _stream(stream)))


def unpack_expert(dm: Dims, record: np.ndarray) -> dict:
    """emoe_unpack_expert on a host copy of one record (numpy uint8)."""
    d, f = dm.d_model, dm.d_ff
    out = dict(q_gate=np.empty((f, d), np.int8), s_gate=np.empty((f, d // 128), np.uint16),
               q_up=np.empty((f, d), np.int8), s_up=np.empty((f, d // 128), np.uint16),
               q_down=np.empty((d, f), np.int8), s_down=np.empty((d, f // 128), np.uint16))
    rec = np.ascontiguousarray(record, dtype=np.uint8)
    check(lib().emoe_unpack_expert(C.byref(dm), rec.ctypes.data, *[out[k].ctypes.data for k in
                                   ("q_gate", "s_gate", "q_up", "s_up", "q_down", "s_down")]))
    return out


def pack_expert(dm: Dims, q_gate, s_gate, q_up, s_up, q_down, s_down) -> np.ndarray:
    """emoe_pack_expert: plain codes/scales (host) -> one packed record (numpy uint8)."""
    rec = np.zeros(expert_record_bytes(dm), np.uint8)
    arrs = [np.ascontiguousarray(a) for a in (q_gate, s_gate, q_up, s_up, q_down, s_down)]
    check(lib().emoe_pack_expert(C.byref(dm), *[a.ctypes.data for a in arrs], rec.ctypes.data))
    return rec


def route(dm: Dims, tokens: int, h, w_router, logits_override, renormalize: bool, logits,
          topk_ids, topk_w, counts, offsets, sorted_pairs, active, n_active, stream=None) -> None:
    """emoe_route: Eq. 1 logits, top-k, mixture weights and grouping on the device."""
    check(lib().emoe_route(C.byref(dm), tokens, _ptr(h), _ptr(w_router), _ptr(logits_override),
                           int(bool(renormalize)), _ptr(logits), _ptr(topk_ids), _ptr(topk_w),
                           _ptr(counts), _ptr(offsets), _ptr(sorted_pairs), _ptr(active),
                           _ptr(n_active), _stream(stream)))


class Cache:
    """emoe_cache_*: one layer's slot cache (Sec. 3.3)."""

    def __init__(self, dm: Dims, capacity: int, slot_bank=None, host_bank=None):
        self.dims = dm
        self.capacity = capacity
        self._keep = (slot_bank, host_bank)
        handle = C.c_void_p()
        check(lib().emoe_cache_create(C.byref(dm), capacity, _ptr(slot_bank), _ptr(host_bank),
                                      C.byref(handle)))
        self.handle = handle

    def close(self) -> None:
        if self.handle:
            lib().emoe_cache_destroy(self.handle)
            self.handle = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def preload_all(self, stream=None) -> None:
        check(lib().emoe_cache_preload_all(self.handle, _stream(stream)))

    def state(self):
        e, c = self.dims.n_experts, self.capacity
        so, eo, st = np.empty(e, np.int32), np.empty(c, np.int32), np.empty(c, np.int64)
        check(lib().emoe_cache_state(self.handle, so.ctypes.data, eo.ctypes.data, st.ctypes.data))
        return so, eo, st

    def sync_timeouts(self) -> int:
        """emoe_cache_sync_timeouts: bounded device waits that gave up (0 when healthy)."""
        n = C.c_int64()
        check(lib().emoe_cache_sync_timeouts(self.handle, C.byref(n)))
        return n.value

    def set_wave_overlap(self, enable: bool) -> None:
        """emoe_cache_set_wave_overlap: waves of C/2 when the active set does not fit,
        so each wave's fills proceed while the previous wave computes."""
        check(lib().emoe_cache_set_wave_overlap(self.handle, int(bool(enable))))

    def set_wave_delay(self, microseconds: int) -> None:
        """emoe_test_set_wave_delay: spin before each wave's projections (test hook)."""
        check(lib().emoe_test_set_wave_delay(self.handle, int(microseconds)))

    def set_decode_waits(self, spin_limit: int = 1 << 20, unmatched: bool = False) -> None:
        """emoe_test_set_decode_waits: the fused decode launch's waits give up after
        `spin_limit` polls; with `unmatched` they wait for a tag no writer uses (test hook)."""
        check(lib().emoe_test_set_decode_waits(self.handle, int(spin_limit), int(bool(unmatched))))

    def plan_waves(self, counts) -> list[list[int]]:
        e = self.dims.n_experts
        cnt = np.ascontiguousarray(counts, np.int32)
        we, wo, nw = np.empty(e, np.int32), np.empty(e + 1, np.int32), C.c_int32()
        check(lib().emoe_plan_waves(self.handle, cnt.ctypes.data, we.ctypes.data, wo.ctypes.data,
                                    C.byref(nw)))
        return [we[wo[i]:wo[i + 1]].tolist() for i in range(nw.value)]

    def build_slot_map(self, wave, stats: Stats | None = None):
        e = self.dims.n_experts
        w = np.ascontiguousarray(wave, np.int32)
        sm = np.empty(e, np.int32)
        fe, fs = np.empty(max(len(w), 1), np.int32), np.empty(max(len(w), 1), np.int32)
        nf = C.c_int32()
        check(lib().emoe_build_slot_map(self.handle, w.ctypes.data, len(w), sm.ctypes.data,
                                        fe.ctypes.data, fs.ctypes.data, C.byref(nf),
                                        C.byref(stats) if stats is not None else None))
        return sm, list(zip(fe[:nf.value].tolist(), fs[:nf.value].tolist()))

    def fill_slots(self, fills, stream=None) -> None:
        fe = np.array([a for a, _ in fills], np.int32)
        fs = np.array([b for _, b in fills], np.int32)
        check(lib().emoe_fill_slots(self.handle, fe.ctypes.data, fs.ctypes.data, len(fills),
                                    _stream(stream)))


def moe_forward(cache: Cache, h, w_router, y, workspace, logits_override=None,
                renormalize: bool = True, path: int = EMOE_PATH_AUTO, stats: Stats | None = None,
                stream=None, sequential: bool = False) -> None:
    """emoe_moe_forward (or emoe_moe_forward_sequential): y = the MoE layer of Eq. 2."""
    fn = lib().emoe_moe_forward_sequential if sequential else lib().emoe_moe_forward
    tokens = h.shape[0]
    nbytes = workspace.numel() * workspace.element_size()
    check(fn(cache.handle, tokens, _ptr(h), _ptr(w_router), _ptr(logits_override),
             int(bool(renormalize)), path, _ptr(y), _ptr(workspace), nbytes, _stream(stream),
             C.byref(stats) if stats is not None else None))


def moe_forward_noalloc(cache: Cache, h, w_router, y, logits_override=None,
                        renormalize: bool = True, path: int = EMOE_PATH_AUTO,
                        stats: Stats | None = None, stream=None) -> None:
    """emoe_moe_forward_noalloc: the layer call with the library's own scratch workspace."""
    check(lib().emoe_moe_forward_noalloc(cache.handle, h.shape[0], _ptr(h), _ptr(w_router),
                                         _ptr(logits_override), int(bool(renormalize)), path,
                                         _ptr(y), _stream(stream),
                                         C.byref(stats) if stats is not None else None))


def moe_forward_sequential(cache: Cache, h, w_router, y, workspace, **kw) -> None:
    moe_forward(cache, h, w_router, y, workspace, sequential=True, **kw)


def test_fail_copy_after(copies: int) -> None:
    """emoe_test_fail_copy_after: make the slot copy after `copies` more fail (-1 disarms)."""
    check(lib().emoe_test_fail_copy_after(int(copies)))


def decoder_dims(n_layers: int, n_heads: int, head_dim: int, vocab: int, max_positions: int,
                 moe: Dims, rope_base: float = 10000.0, rms_eps: float = 1e-5,
                 renormalize: bool = True) -> DecoderDims:
    return DecoderDims(n_layers, n_heads, head_dim, vocab, max_positions, rope_base, rms_eps,
                       int(bool(renormalize)), moe)


def decoder_kv_bytes(dd: DecoderDims) -> int:
    return int(lib().emoe_decoder_kv_bytes(C.byref(dd)))


def decoder_workspace_bytes(dd: DecoderDims, max_tokens: int) -> int:
    return int(lib().emoe_decoder_workspace_bytes(C.byref(dd), max_tokens))


class Decoder:
    """emoe_decoder_*: the synthetic decoder around one slot cache per layer.

    weights: dict of device bf16 tensors: embed [V][d], lm_head [V][d],
    final_norm [d], and per-layer lists attn_norm, wqkv [3d][d], wo [d][d],
    moe_norm, w_router [E][d].  caches: list of Cache (one per layer).
    kv: device buffer of decoder_kv_bytes(dd) bytes."""

    def __init__(self, dd: DecoderDims, weights: dict, caches, kv):
        n = dd.n_layers
        arr = lambda name: (C.c_void_p * n)(*[_ptr(t) for t in weights[name]])
        self._arrays = {k: arr(k) for k in ("attn_norm", "wqkv", "wo", "moe_norm", "w_router")}
        cast = lambda a: C.cast(a, C.POINTER(C.c_void_p))
        w = DecoderWeights(_ptr(weights["embed"]), _ptr(weights["lm_head"]),
                           _ptr(weights["final_norm"]), cast(self._arrays["attn_norm"]),
                           cast(self._arrays["wqkv"]), cast(self._arrays["wo"]),
                           cast(self._arrays["moe_norm"]), cast(self._arrays["w_router"]))
        handles = (C.c_void_p * n)(*[c.handle.value for c in caches])
        self.dims = dd
        self._keep = (weights, caches, kv, handles)
        h = C.c_void_p()
        check(lib().emoe_decoder_create(C.byref(dd), C.byref(w), C.cast(handles, C.POINTER(C.c_void_p)),
                                        _ptr(kv), C.byref(h)))
        self.handle = h

    def close(self) -> None:
        if self.handle:
            lib().emoe_decoder_destroy(self.handle)
            self.handle = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def forward(self, tokens, pos0: int, logits, next_token, workspace, stream=None,
                stats: Stats | None = None) -> None:
        """emoe_decoder_forward: tokens (device int32 [T]) at positions pos0 .. pos0+T-1."""
        nbytes = workspace.numel() * workspace.element_size()
        check(lib().emoe_decoder_forward(self.handle, _ptr(tokens), tokens.shape[0], pos0,
                                         _ptr(logits), _ptr(next_token), _ptr(workspace), nbytes,
                                         _stream(stream),
                                         C.byref(stats) if stats is not None else None))


def profile_begin(max_kernels: int) -> None:
    """emoe_profile_begin: time each kernel the layer calls launch from this thread."""
    check(lib().emoe_profile_begin(max_kernels))


def profile_end(max_out: int = 1 << 16) -> list[tuple[str, float]]:
    """emoe_profile_end: [(kernel name, milliseconds)] in launch order."""
    kinds = np.empty(max_out, np.int32)
    ms = np.empty(max_out, np.float32)
    n = C.c_int32()
    check(lib().emoe_profile_end(kinds.ctypes.data, ms.ctypes.data, max_out, C.byref(n)))
    m = min(n.value, max_out)
    return [(_lib.KERNEL_NAMES[k], float(t)) for k, t in zip(kinds[:m], ms[:m])]


__all__ = ["Dims", "Stats", "WsLayout", "ExactMoEError", "EMOE_PATH_AUTO", "EMOE_PATH_GEMV",
           "EMOE_PATH_MFMA", "EMOE_PATH_MIXED", "EMOE_MIXED_MFMA_ROWS", "dims", "check_dims", "expert_record_bytes", "workspace_layout",
           "workspace_bytes", "quantize_experts", "unpack_expert", "pack_expert", "route", "Cache",
           "moe_forward", "moe_forward_noalloc", "decoder_dims", "decoder_kv_bytes",
           "decoder_workspace_bytes", "Decoder", "moe_forward_sequential", "test_fail_copy_after", "profile_begin", "profile_end", "lib"]
