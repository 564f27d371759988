"""ctypes declarations of libexactmoe.so (include/exactmoe.h).

Argument marshalling only: every step of the layer runs in the library.
Loading fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libexactmoe.so")

EMOE_OK, EMOE_EINVAL, EMOE_ESHAPE, EMOE_ERANGE, EMOE_ECAPACITY, EMOE_EHIP, EMOE_ESTATE = \
    0, -1, -2, -3, -4, -5, -6
EMOE_GROUP = 128
EMOE_MAX_EXPERTS = 256
EMOE_PATH_AUTO, EMOE_PATH_GEMV, EMOE_PATH_MFMA, EMOE_PATH_MIXED = 0, 1, 2, 3
EMOE_MIXED_MFMA_ROWS = 16
EMOE_GEMV_MAX_TOKENS = 4
EMOE_NOALLOC_SCRATCH_BYTES = 32 << 20


class Dims(C.Structure):
    _fields_ = [("d_model", C.c_int32), ("d_ff", C.c_int32), ("n_experts", C.c_int32),
                ("top_k", C.c_int32)]


class Stats(C.Structure):
    _fields_ = [(n, C.c_int64) for n in ("layer_calls", "waves", "hits", "misses", "h2d_bytes",
                                          "grouped_gemm_calls", "seq_expert_calls",
                                          "kernel_launches")]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


class WsLayout(C.Structure):
    _fields_ = [(n, C.c_size_t) for n in ("logits", "topk_ids", "topk_w", "counts", "offsets",
                                          "sorted_pairs", "active", "n_active", "tile_offsets",
                                          "pair_pos", "act", "pair_out", "act_bias",
                                          "chunk_counts", "tok_bias", "total")]


class DecoderDims(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("n_heads", C.c_int32), ("head_dim", C.c_int32),
                ("vocab", C.c_int32), ("max_positions", C.c_int32), ("rope_base", C.c_float),
                ("rms_eps", C.c_float), ("renormalize", C.c_int32), ("moe", Dims)]


class DecoderWeights(C.Structure):
    _fields_ = [("embed", C.c_void_p), ("lm_head", C.c_void_p), ("final_norm", C.c_void_p),
                ("attn_norm", C.POINTER(C.c_void_p)), ("wqkv", C.POINTER(C.c_void_p)),
                ("wo", C.POINTER(C.c_void_p)), ("moe_norm", C.POINTER(C.c_void_p)),
                ("w_router", C.POINTER(C.c_void_p))]


_vp = C.c_void_p
_i32 = C.c_int32
_i32p = C.POINTER(C.c_int32)
_i64p = C.POINTER(C.c_int64)
_dimsp = C.POINTER(Dims)

# name -> (restype, argtypes); mirrors include/exactmoe.h
SIGNATURES = {
    "emoe_status_string": (C.c_char_p, [_i32]),
    "emoe_last_error": (C.c_char_p, []),
    "emoe_check_dims": (_i32, [_dimsp]),
    "emoe_expert_record_bytes": (C.c_size_t, [_dimsp]),
    "emoe_workspace_layout": (_i32, [_dimsp, _i32, C.POINTER(WsLayout)]),
    "emoe_workspace_bytes": (C.c_size_t, [_dimsp, _i32]),
    "emoe_quantize_experts": (_i32, [_dimsp, _i32, _vp, _vp, _vp, _vp, _vp]),
    "emoe_unpack_expert": (_i32, [_dimsp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "emoe_pack_expert": (_i32, [_dimsp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "emoe_route": (_i32, [_dimsp, _i32, _vp, _vp, _vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                          _vp, _vp]),
    "emoe_cache_create": (_i32, [_dimsp, _i32, _vp, _vp, C.POINTER(_vp)]),
    "emoe_cache_destroy": (_i32, [_vp]),
    "emoe_cache_preload_all": (_i32, [_vp, _vp]),
    "emoe_cache_state": (_i32, [_vp, _vp, _vp, _vp]),
    "emoe_cache_set_wave_overlap": (_i32, [_vp, _i32]),
    "emoe_cache_sync_timeouts": (_i32, [_vp, _i64p]),
    "emoe_plan_waves": (_i32, [_vp, _vp, _vp, _vp, _i32p]),
    "emoe_build_slot_map": (_i32, [_vp, _vp, _i32, _vp, _vp, _vp, _i32p, C.POINTER(Stats)]),
    "emoe_fill_slots": (_i32, [_vp, _vp, _vp, _i32, _vp]),
    "emoe_moe_forward": (_i32, [_vp, _i32, _vp, _vp, _vp, _i32, _i32, _vp, _vp, C.c_size_t, _vp,
                                C.POINTER(Stats)]),
    "emoe_moe_forward_sequential": (_i32, [_vp, _i32, _vp, _vp, _vp, _i32, _i32, _vp, _vp,
                                           C.c_size_t, _vp, C.POINTER(Stats)]),
    "emoe_moe_forward_noalloc": (_i32, [_vp, _i32, _vp, _vp, _vp, _i32, _i32, _vp, _vp,
                                        C.POINTER(Stats)]),
    "emoe_test_fail_copy_after": (_i32, [C.c_int64]),
    "emoe_test_set_wave_delay": (_i32, [_vp, _i32]),
    "emoe_test_set_decode_waits": (_i32, [_vp, _i32, _i32]),
    "emoe_debug_fused_plan": (_i32, [_dimsp, _i32, _i32, _vp, _vp, _i32]),
    "emoe_decoder_kv_bytes": (C.c_size_t, [C.POINTER(DecoderDims)]),
    "emoe_decoder_workspace_bytes": (C.c_size_t, [C.POINTER(DecoderDims), _i32]),
    "emoe_decoder_create": (_i32, [C.POINTER(DecoderDims), C.POINTER(DecoderWeights),
                                   C.POINTER(_vp), _vp, C.POINTER(_vp)]),
    "emoe_decoder_destroy": (_i32, [_vp]),
    "emoe_decoder_forward": (_i32, [_vp, _vp, _i32, _i32, _vp, _vp, _vp, C.c_size_t, _vp,
                                    C.POINTER(Stats)]),
    "emoe_profile_begin": (_i32, [_i32]),
    "emoe_profile_end": (_i32, [_vp, _vp, _i32, _i32p]),
}

KERNEL_NAMES = ["router", "topk", "group", "gateup_gemv", "down_gemv", "gateup_mfma", "down_mfma",
                "combine", "decode_fused", "row_bias", "group_count"]

_lib = None


class ExactMoEError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} (status {status})")
        self.status = status


def lib() -> C.CDLL:
    """Load libexactmoe.so once; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: run `python -m paper_2608_15383_amd.build`")
        h = C.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(h, name)
            fn.restype = res
            fn.argtypes = args
        _lib = h
    return _lib


def check(status: int) -> None:
    if status != EMOE_OK:
        msg = lib().emoe_last_error().decode() or lib().emoe_status_string(status).decode()
        raise ExactMoEError(status, msg)
