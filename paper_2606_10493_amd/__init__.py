"""MI355X (gfx950) routed-expert FP8 MoE FFN.

Thin Python binding of libmoe.so (the C ABI in include/moe.h).  Functions
carry the C names and only marshal arguments: every step of the layer runs
in the library's HIP kernels.  torch tensors supply device memory and
streams; nothing here computes.  If libmoe.so is missing the import fails:
build it with ``python paper_2606_10493_amd/build.py``.
"""
from __future__ import annotations

import ctypes
import os

from ._lib import (  # noqa: F401
    LIB_PATH, MoEError, lib, MOE_OK, MOE_ERR_INVALID_ARG, MOE_ERR_UNSUPPORTED_SHAPE,
    MOE_ERR_WORKSPACE, MOE_ERR_HIP, MOE_REGIME_AUTO, MOE_REGIME_DECODE, MOE_REGIME_PREFILL,
    MOE_DEV_BAD_EXPERT_ID, MOE_DEV_DUP_EXPERT_ID, MOE_DECODE_MAX_TOKENS, MOE_NOALLOC_SCRATCH_BYTES, MoeDims,
    MoeRouterCfg, MoeStreamOp, MOE_SOP_WAIT_OFF, MOE_SOP_COPY, MOE_SOP_RECORD_ON, MOE_SOP_WAIT_ON, MOE_SOP_LAUNCH,
    MOE_SOP_RECORD_OFF,
    EXPORTED_SYMBOLS,
)
from ._lib import check as _check


def _ptr(t):
    return ctypes.c_void_p(0 if t is None else t.data_ptr())


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _nbytes(t):
    return 0 if t is None else t.numel() * t.element_size()


def _need(t, dtype_bytes, name):
    if t is not None:
        if not t.is_cuda:
            raise ValueError(f"{name} must be a device tensor")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        if t.element_size() != dtype_bytes:
            raise ValueError(f"{name} has element size {t.element_size()}, expected {dtype_bytes}")


def moe_status_string(status: int) -> str:
    return lib.moe_status_string(status).decode()


def moe_last_error() -> str:
    return lib.moe_last_error().decode()


def moe_quant_act(x_bf16, q, s, stream=None):
    """x_bf16 [rows, cols] (bf16 or 16-bit view) -> q uint8 [rows, cols], s fp32 [rows, cols/128]."""
    _need(x_bf16, 2, "x_bf16"); _need(q, 1, "q"); _need(s, 4, "s")
    rows, cols = x_bf16.shape
    _check(lib.moe_quant_act(_ptr(x_bf16), rows, cols, _ptr(q), _ptr(s), _stream(stream)))


def moe_quant_rows_f32(x, q, s, stream=None):
    _need(x, 4, "x"); _need(q, 1, "q"); _need(s, 4, "s")
    rows, cols = x.shape
    _check(lib.moe_quant_rows_f32(_ptr(x), rows, cols, _ptr(q), _ptr(s), _stream(stream)))


def moe_quant_weight(w, q, s, stream=None):
    """w fp32 [n_mats, rows, cols] (or [rows, cols]) -> q uint8 same shape, s fp32 [.., rows/128, cols/128]."""
    _need(w, 4, "w"); _need(q, 1, "q"); _need(s, 4, "s")
    shape = w.shape if w.dim() == 3 else (1, *w.shape)
    _check(lib.moe_quant_weight(_ptr(w), shape[0], shape[1], shape[2], _ptr(q), _ptr(s), _stream(stream)))


def moe_pack_weight(q, packed, stream=None):
    """q uint8 [n_mats, rows, cols] (or [rows, cols]) row-major -> packed operand tiles (same size)."""
    _need(q, 1, "q"); _need(packed, 1, "packed")
    shape = q.shape if q.dim() == 3 else (1, *q.shape)
    if packed.numel() != q.numel():
        raise MoEError(MOE_ERR_INVALID_ARG, "moe_pack_weight: packed must have as many bytes as q")
    _check(lib.moe_pack_weight(_ptr(q), shape[0], shape[1], shape[2], _ptr(packed), _stream(stream)))


def moe_permute_workspace(T: int, k: int, E: int) -> int:
    return int(lib.moe_permute_workspace(T, k, E))


def moe_permute(topk_ids, n_experts, expert_offsets, sorted_src, dest_row, dev_status=None, ws=None,
                stream=None):
    _need(topk_ids, 4, "topk_ids"); _need(expert_offsets, 4, "expert_offsets")
    _need(sorted_src, 4, "sorted_src"); _need(dest_row, 4, "dest_row")
    _need(dev_status, 4, "dev_status"); _need(ws, 1, "ws")
    T, k = topk_ids.shape
    _check(lib.moe_permute(_ptr(topk_ids), T, k, n_experts, _ptr(expert_offsets), _ptr(sorted_src),
                           _ptr(dest_row), _ptr(dev_status), _ptr(ws), _nbytes(ws), _stream(stream)))


def moe_expert_ffn_workspace(dims: MoeDims, T: int, regime: int = MOE_REGIME_AUTO) -> int:
    return int(lib.moe_expert_ffn_workspace(dims, T, regime))


def moe_expert_ffn(dims: MoeDims, T: int, regime: int, qx, sx, expert_offsets, sorted_src,
                   w_gate, s_gate, w_up, s_up, w_down, s_down, y_rows, ws, stream=None):
    for t, nb, n in ((qx, 1, "qx"), (sx, 4, "sx"), (expert_offsets, 4, "expert_offsets"),
                     (sorted_src, 4, "sorted_src"), (w_gate, 1, "w_gate"), (s_gate, 4, "s_gate"),
                     (w_up, 1, "w_up"), (s_up, 4, "s_up"), (w_down, 1, "w_down"), (s_down, 4, "s_down"),
                     (y_rows, 4, "y_rows"), (ws, 1, "ws")):
        _need(t, nb, n)
    _check(lib.moe_expert_ffn(dims, T, regime, _ptr(qx), _ptr(sx), _ptr(expert_offsets), _ptr(sorted_src),
                              _ptr(w_gate), _ptr(s_gate), _ptr(w_up), _ptr(s_up), _ptr(w_down),
                              _ptr(s_down), _ptr(y_rows), _ptr(ws), _nbytes(ws), _stream(stream)))


def moe_expert_ffn_w8a16_workspace(dims: MoeDims, T: int) -> int:
    return int(lib.moe_expert_ffn_w8a16_workspace(dims, T))


def moe_expert_ffn_w8a16(dims: MoeDims, T: int, x_bf16, expert_offsets, sorted_src,
                         w_gate, s_gate, w_up, s_up, w_down, s_down, y_rows, ws, stream=None):
    """Decode-regime expert FFN with bf16 activations (the W8A16 GEMV numerics)."""
    for t, nb, n in ((x_bf16, 2, "x_bf16"), (expert_offsets, 4, "expert_offsets"), (sorted_src, 4, "sorted_src"),
                     (w_gate, 1, "w_gate"), (s_gate, 4, "s_gate"), (w_up, 1, "w_up"), (s_up, 4, "s_up"),
                     (w_down, 1, "w_down"), (s_down, 4, "s_down"), (y_rows, 4, "y_rows"), (ws, 1, "ws")):
        _need(t, nb, n)
    _check(lib.moe_expert_ffn_w8a16(dims, T, _ptr(x_bf16), _ptr(expert_offsets), _ptr(sorted_src), _ptr(w_gate),
                                    _ptr(s_gate), _ptr(w_up), _ptr(s_up), _ptr(w_down), _ptr(s_down), _ptr(y_rows),
                                    _ptr(ws), _nbytes(ws), _stream(stream)))


def moe_router_workspace(T: int, H: int, E: int) -> int:
    return int(lib.moe_router_workspace(T, H, E))


def moe_router(x_bf16, w_router_bf16, bias, topk_ids, topk_w, n_group=1, topk_group=1, routed_scaling=1.0,
               ws=None, stream=None, shared_expert=-1):
    """x_bf16 [T, H], w_router_bf16 [E, H] (bf16 or 16-bit views), bias fp32 [E] or None
    -> topk_ids int32 [T, k], topk_w fp32 [T, k]; with shared_expert >= 0 both are
    [T, k + 1] and the last slot is (shared_expert, 1.0)."""
    _need(x_bf16, 2, "x_bf16"); _need(w_router_bf16, 2, "w_router_bf16"); _need(bias, 4, "bias")
    _need(topk_ids, 4, "topk_ids"); _need(topk_w, 4, "topk_w"); _need(ws, 1, "ws")
    T, H = x_bf16.shape
    E = w_router_bf16.shape[0]
    k = topk_ids.shape[1] - (1 if shared_expert >= 0 else 0)
    if topk_w.shape != topk_ids.shape:
        raise ValueError("topk_w must have the shape of topk_ids")
    cfg = MoeRouterCfg(n_group, topk_group, routed_scaling, shared_expert)
    _check(lib.moe_router(_ptr(x_bf16), T, H, _ptr(w_router_bf16), _ptr(bias), E, k, cfg, _ptr(topk_ids),
                          _ptr(topk_w), _ptr(ws), _nbytes(ws), _stream(stream)))


def moe_combine(y_rows, dest_row, topk_w, out_bf16, stream=None):
    _need(y_rows, 4, "y_rows"); _need(dest_row, 4, "dest_row"); _need(topk_w, 4, "topk_w")
    _need(out_bf16, 2, "out_bf16")
    T, k = topk_w.shape
    H = out_bf16.shape[1]
    _check(lib.moe_combine(_ptr(y_rows), _ptr(dest_row), _ptr(topk_w), T, k, H, _ptr(out_bf16),
                           _stream(stream)))


def moe_ffn_layer_workspace(dims: MoeDims, T: int, regime: int = MOE_REGIME_AUTO) -> int:
    return int(lib.moe_ffn_layer_workspace(dims, T, regime))


def moe_ffn_layer(dims: MoeDims, T: int, regime: int, x_bf16, topk_ids, topk_w, w_gate, s_gate, w_up, s_up,
                  w_down, s_down, out_bf16, dev_status, ws, stream=None):
    """The whole resident layer in one library call (see include/moe.h)."""
    for t, nb, n in ((x_bf16, 2, "x_bf16"), (topk_ids, 4, "topk_ids"), (topk_w, 4, "topk_w"),
                     (w_gate, 1, "w_gate"), (s_gate, 4, "s_gate"), (w_up, 1, "w_up"), (s_up, 4, "s_up"),
                     (w_down, 1, "w_down"), (s_down, 4, "s_down"), (out_bf16, 2, "out_bf16"),
                     (dev_status, 4, "dev_status"), (ws, 1, "ws")):
        _need(t, nb, n)
    _check(lib.moe_ffn_layer(dims, T, regime, _ptr(x_bf16), _ptr(topk_ids), _ptr(topk_w), _ptr(w_gate),
                             _ptr(s_gate), _ptr(w_up), _ptr(s_up), _ptr(w_down), _ptr(s_down), _ptr(out_bf16),
                             _ptr(dev_status), _ptr(ws), _nbytes(ws), _stream(stream)))


def moe_ffn_layer_noalloc(dims: MoeDims, T: int, regime: int, x_bf16, topk_ids, topk_w, w_gate, s_gate, w_up, s_up,
                          w_down, s_down, out_bf16, dev_status=None, stream=None):
    """moe_ffn_layer with the library's per-GPU scratch array instead of a workspace (see include/moe.h)."""
    for t, nb, n in ((x_bf16, 2, "x_bf16"), (topk_ids, 4, "topk_ids"), (topk_w, 4, "topk_w"),
                     (w_gate, 1, "w_gate"), (s_gate, 4, "s_gate"), (w_up, 1, "w_up"), (s_up, 4, "s_up"),
                     (w_down, 1, "w_down"), (s_down, 4, "s_down"), (out_bf16, 2, "out_bf16"),
                     (dev_status, 4, "dev_status")):
        _need(t, nb, n)
    _check(lib.moe_ffn_layer_noalloc(dims, T, regime, _ptr(x_bf16), _ptr(topk_ids), _ptr(topk_w), _ptr(w_gate),
                                     _ptr(s_gate), _ptr(w_up), _ptr(s_up), _ptr(w_down), _ptr(s_down),
                                     _ptr(out_bf16), _ptr(dev_status), _stream(stream)))


class StreamContext:
    """Owns the per-slot ON/OFF events of moe_ffn_streamed (created once, at setup)."""

    def __init__(self, ring_slots: int):
        h = ctypes.c_void_p()
        _check(lib.moe_stream_ctx_create(ring_slots, ctypes.byref(h)))
        self.handle = h
        self.slots = ring_slots

    def close(self):
        if self.handle:
            lib.moe_stream_ctx_destroy(self.handle)
            self.handle = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:  # interpreter shutdown
            pass


def moe_ring_bytes(dims: MoeDims, ring_slots: int) -> int:
    return int(lib.moe_ring_bytes(dims, ring_slots))


def moe_ring_scale_bytes(dims: MoeDims, ring_slots: int) -> int:
    return int(lib.moe_ring_scale_bytes(dims, ring_slots))


def moe_ffn_streamed_workspace(dims: MoeDims, T: int, chunk_tokens: int) -> int:
    return int(lib.moe_ffn_streamed_workspace(dims, T, chunk_tokens))


def moe_stream_schedule(dims: MoeDims, T: int, chunk_tokens: int, ring_slots: int, off_recorded=None):
    """The ring schedule moe_ffn_streamed enqueues for one layer (host only).

    Returns (ops, off_recorded): ops a list of (op, a, b, c) tuples in
    enqueue order (MOE_SOP_* codes, fields as in include/moe.h), and the
    per-slot OFF-record flags the call leaves in the context (pass them to
    the next layer's call on the same ring)."""
    rec = (ctypes.c_uint8 * ring_slots)(*(bytes(ring_slots) if off_recorded is None else off_recorded))
    n = ctypes.c_int32(0)
    st = lib.moe_stream_schedule(dims, T, chunk_tokens, ring_slots, ctypes.cast(rec, ctypes.c_void_p), None, 0,
                                 ctypes.byref(n))
    if st not in (MOE_OK, MOE_ERR_WORKSPACE):
        _check(st)
    ops = (MoeStreamOp * max(n.value, 1))()
    _check(lib.moe_stream_schedule(dims, T, chunk_tokens, ring_slots, ctypes.cast(rec, ctypes.c_void_p),
                                   ctypes.cast(ops, ctypes.c_void_p), n.value, ctypes.byref(n)))
    return [(o.op, o.a, o.b, o.c) for o in ops[:n.value]], bytes(rec)


def _need_pinned(t, dtype_bytes, name):
    if t.is_cuda or not t.is_pinned():
        raise ValueError(f"{name} must be a pinned host tensor")
    if not t.is_contiguous() or t.element_size() != dtype_bytes:
        raise ValueError(f"{name} must be contiguous with element size {dtype_bytes}")


def moe_ffn_streamed(dims: MoeDims, chunk_tokens: int, x_bf16, topk_ids, topk_w, host_weights, dev_ring,
                     dev_ring_scales, ctx: "StreamContext", out_bf16, dev_status, ws, compute_stream=None,
                     copy_stream=None):
    """host_weights = (w_gate, s_gate, w_up, s_up, w_down, s_down) pinned host tensors."""
    T = x_bf16.shape[0]
    _need(x_bf16, 2, "x_bf16"); _need(topk_ids, 4, "topk_ids"); _need(topk_w, 4, "topk_w")
    _need(dev_ring, 1, "dev_ring"); _need(dev_ring_scales, 4, "dev_ring_scales")
    _need(out_bf16, 2, "out_bf16"); _need(dev_status, 4, "dev_status"); _need(ws, 1, "ws")
    for t, nb, n in zip(host_weights, (1, 4, 1, 4, 1, 4),
                        ("host_w_gate", "host_s_gate", "host_w_up", "host_s_up", "host_w_down", "host_s_down")):
        _need_pinned(t, nb, n)
    if dev_ring.numel() < moe_ring_bytes(dims, ctx.slots):
        raise ValueError("dev_ring is smaller than moe_ring_bytes(dims, ctx.slots)")
    if dev_ring_scales.numel() * 4 < moe_ring_scale_bytes(dims, ctx.slots):
        raise ValueError("dev_ring_scales is smaller than moe_ring_scale_bytes(dims, ctx.slots)")
    hw = [_ptr(t) for t in host_weights]
    _check(lib.moe_ffn_streamed(dims, T, chunk_tokens, _ptr(x_bf16), _ptr(topk_ids), _ptr(topk_w), *hw,
                                _ptr(dev_ring), _ptr(dev_ring_scales), ctx.handle, _ptr(out_bf16), _ptr(dev_status),
                                _ptr(ws), _nbytes(ws), _stream(compute_stream), _stream(copy_stream)))


def moe_profile_begin(max_launches: int) -> None:
    _check(lib.moe_profile_begin(max_launches))


def moe_profile_end():
    """Stop recording; returns [(kernel name, ms), ...] in launch order."""
    n = lib.moe_profile_end()
    out = []
    for i in range(n):
        ms = ctypes.c_float()
        name = ctypes.c_char_p()
        _check(lib.moe_profile_get(i, ctypes.byref(ms), ctypes.byref(name)))
        out.append((name.value.decode(), float(ms.value)))
    return out


from .layer import MoELayerBuffers, run_layer  # noqa: E402,F401
