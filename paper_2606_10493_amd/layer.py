"""One routed-expert layer call through the C ABI, with torch-allocated buffers.

``MoELayerBuffers`` owns the device buffers of one (dims, tokens) shape;
``run_layer`` enqueues moe_quant_act -> moe_permute -> moe_expert_ffn ->
moe_combine on one stream (with ``w8a16``: moe_permute ->
moe_expert_ffn_w8a16 -> moe_combine, bf16 activations, decode regime;
with ``fused``: one moe_ffn_layer call, whose intermediates live in its
workspace).  Nothing is computed in Python.
"""
from __future__ import annotations

import torch

from . import _lib
from ._lib import MoeDims


class MoELayerBuffers:
    def __init__(self, hidden: int, inter: int, n_experts: int, topk: int, tokens: int,
                 regime: int = _lib.MOE_REGIME_AUTO, device="cuda", with_status: bool = True, w8a16: bool = False,
                 fused: bool = False):
        if fused and w8a16:
            raise ValueError("moe_ffn_layer runs the W8A8 layer; W8A16 goes through the separate calls")
        self.dims = MoeDims(hidden, inter, n_experts, topk)
        self.tokens = tokens
        self.regime = regime
        self.fused = fused
        self.w8a16 = w8a16
        t, h, k, e = tokens, hidden, topk, n_experts
        dev = torch.device(device)
        self.dev_status = torch.zeros(1, dtype=torch.int32, device=dev) if with_status else None
        self.out = torch.empty((t, h), dtype=torch.int16, device=dev)
        if fused:
            lws = _lib.lib.moe_ffn_layer_workspace(self.dims, t, regime)
            self.layer_ws = torch.empty(max(lws, 256), dtype=torch.uint8, device=dev)
            return
        self.qx = torch.empty((t, h), dtype=torch.uint8, device=dev)
        self.sx = torch.empty((t, h // 128), dtype=torch.float32, device=dev)
        self.expert_offsets = torch.empty(e + 1, dtype=torch.int32, device=dev)
        self.sorted_src = torch.empty(t * k, dtype=torch.int32, device=dev)
        self.dest_row = torch.empty(t * k, dtype=torch.int32, device=dev)
        pws = _lib.lib.moe_permute_workspace(t, k, e)
        self.perm_ws = torch.empty(max(pws, 1), dtype=torch.uint8, device=dev)
        fws = (_lib.lib.moe_expert_ffn_w8a16_workspace(self.dims, t) if w8a16
               else _lib.lib.moe_expert_ffn_workspace(self.dims, t, regime))
        self.ffn_ws = torch.empty(max(fws, 256), dtype=torch.uint8, device=dev)
        self.y_rows = torch.empty((t * k, h), dtype=torch.float32, device=dev)


def run_layer(buf: MoELayerBuffers, x_bf16, topk_ids, topk_w, weights, stream=None):
    """weights = (w_gate, s_gate, w_up, s_up, w_down, s_down) device tensors."""
    from . import moe_quant_act, moe_permute, moe_expert_ffn, moe_expert_ffn_w8a16, moe_combine, moe_ffn_layer
    wg, sg, wu, su, wd, sd = weights
    if buf.fused:
        moe_ffn_layer(buf.dims, buf.tokens, buf.regime, x_bf16, topk_ids, topk_w, wg, sg, wu, su, wd, sd, buf.out,
                      buf.dev_status, buf.layer_ws, stream)
        return buf.out
    if not buf.w8a16:
        moe_quant_act(x_bf16, buf.qx, buf.sx, stream)
    moe_permute(topk_ids, buf.dims.n_experts, buf.expert_offsets, buf.sorted_src, buf.dest_row,
                buf.dev_status, buf.perm_ws, stream)
    if buf.w8a16:
        moe_expert_ffn_w8a16(buf.dims, buf.tokens, x_bf16, buf.expert_offsets, buf.sorted_src,
                             wg, sg, wu, su, wd, sd, buf.y_rows, buf.ffn_ws, stream)
    else:
        moe_expert_ffn(buf.dims, buf.tokens, buf.regime, buf.qx, buf.sx, buf.expert_offsets, buf.sorted_src,
                       wg, sg, wu, su, wd, sd, buf.y_rows, buf.ffn_ws, stream)
    moe_combine(buf.y_rows, buf.dest_row, topk_w, buf.out, stream)
    return buf.out
