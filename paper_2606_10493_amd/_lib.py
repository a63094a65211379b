"""ctypes declarations of libmoe.so (mirrors include/moe.h)."""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmoe.so")

MOE_OK = 0
MOE_ERR_INVALID_ARG = -1
MOE_ERR_UNSUPPORTED_SHAPE = -2
MOE_ERR_WORKSPACE = -3
MOE_ERR_HIP = -4

MOE_REGIME_AUTO = 0
MOE_REGIME_DECODE = 1
MOE_REGIME_PREFILL = 2
MOE_DECODE_MAX_TOKENS = 64

MOE_NOALLOC_SCRATCH_BYTES = 32 << 20

MOE_DEV_BAD_EXPERT_ID = 1
MOE_DEV_DUP_EXPERT_ID = 2

MOE_SOP_WAIT_OFF = 1
MOE_SOP_COPY = 2
MOE_SOP_RECORD_ON = 3
MOE_SOP_WAIT_ON = 4
MOE_SOP_LAUNCH = 5
MOE_SOP_RECORD_OFF = 6


class MoeDims(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("inter", ctypes.c_int32),
                ("n_experts", ctypes.c_int32), ("topk", ctypes.c_int32)]


class MoeRouterCfg(ctypes.Structure):
    _fields_ = [("n_group", ctypes.c_int32), ("topk_group", ctypes.c_int32), ("routed_scaling", ctypes.c_float),
                ("shared_expert", ctypes.c_int32)]


class MoeStreamOp(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int32), ("a", ctypes.c_int32), ("b", ctypes.c_int32), ("c", ctypes.c_int32)]


class MoEError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        super().__init__(f"{_status_name(status)}: {detail}")


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run `python paper_2606_10493_amd/build.py`")

# torch brings its own HIP runtime (soname libamdhip64.so.7).  Loading it
# first makes libmoe.so bind to that same runtime, so the streams and device
# memory torch hands over belong to the runtime that launches the kernels.
# Loading libmoe.so first would pull a second HIP runtime into the process.
import torch  # noqa: E402,F401

lib = ctypes.CDLL(LIB_PATH)

_P = ctypes.c_void_p
_I = ctypes.c_int32
_S = ctypes.c_size_t
_ST = ctypes.c_int

_SIGS = {
    "moe_status_string": (ctypes.c_char_p, [_ST]),
    "moe_last_error": (ctypes.c_char_p, []),
    "moe_quant_act": (_ST, [_P, _I, _I, _P, _P, _P]),
    "moe_quant_rows_f32": (_ST, [_P, _I, _I, _P, _P, _P]),
    "moe_quant_weight": (_ST, [_P, _I, _I, _I, _P, _P, _P]),
    "moe_pack_weight": (_ST, [_P, _I, _I, _I, _P, _P]),
    "moe_permute_workspace": (_S, [_I, _I, _I]),
    "moe_permute": (_ST, [_P, _I, _I, _I, _P, _P, _P, _P, _P, _S, _P]),
    "moe_expert_ffn_workspace": (_S, [MoeDims, _I, _ST]),
    "moe_expert_ffn": (_ST, [MoeDims, _I, _ST, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _S, _P]),
    "moe_combine": (_ST, [_P, _P, _P, _I, _I, _I, _P, _P]),
    "moe_ffn_layer_workspace": (_S, [MoeDims, _I, _ST]),
    "moe_ffn_layer": (_ST, [MoeDims, _I, _ST, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _S, _P]),
    "moe_ffn_layer_noalloc": (_ST, [MoeDims, _I, _ST, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "moe_expert_ffn_w8a16_workspace": (_S, [MoeDims, _I]),
    "moe_expert_ffn_w8a16": (_ST, [MoeDims, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _S, _P]),
    "moe_router_workspace": (_S, [_I, _I, _I]),
    "moe_router": (_ST, [_P, _I, _I, _P, _P, _I, _I, MoeRouterCfg, _P, _P, _P, _S, _P]),
    "moe_stream_ctx_create": (_ST, [_I, ctypes.POINTER(ctypes.c_void_p)]),
    "moe_stream_ctx_destroy": (None, [_P]),
    "moe_ring_bytes": (_S, [MoeDims, _I]),
    "moe_ring_scale_bytes": (_S, [MoeDims, _I]),
    "moe_ffn_streamed_workspace": (_S, [MoeDims, _I, _I]),
    "moe_stream_schedule": (_ST, [MoeDims, _I, _I, _I, _P, _P, _I, ctypes.POINTER(ctypes.c_int32)]),
    "moe_ffn_streamed": (_ST, [MoeDims, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _S,
                                _P, _P]),
    "moe_profile_begin": (_ST, [_I]),
    "moe_profile_end": (_I, []),
    "moe_profile_get": (_ST, [_I, ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_char_p)]),
}

EXPORTED_SYMBOLS = tuple(_SIGS)

for _name, (_res, _args) in _SIGS.items():
    _f = getattr(lib, _name)
    _f.restype = _res
    _f.argtypes = _args


def _status_name(status: int) -> str:
    return lib.moe_status_string(status).decode()


def check(status: int) -> None:
    if status != MOE_OK:
        raise MoEError(status, lib.moe_last_error().decode())
