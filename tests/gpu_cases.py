"""Helpers of the GPU parity tests: seeded inputs on both sides, oracle runs.

Weights are drawn in fp32 by ``synth``; the GPU quantizes them with
moe_quant_weight (then packs them into operand tiles with moe_pack_weight,
the layout the FFN kernels read) and the oracle with its own
quantize_weight.  The oracle never receives a value produced by the HIP
library.
"""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import synth


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def require_gpu():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need an MI355X; run them with -m gpu on a GPU machine")
    import paper_2606_10493_amd as moe  # noqa: F401  (fails loudly if libmoe.so is missing)
    return moe


def to_dev(a: np.ndarray, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.view(dtype)
    return t.cuda()


def bf16_dev(bits: np.ndarray):
    return to_dev(bits.view(np.int16))


def pack_reference(q: np.ndarray) -> np.ndarray:
    """The operand-tile layout of moe_pack_weight, by its definition: the 16
    bytes at 1024h + 512(kq%2) + 256(kq//2) + 16r of tile (g, b) hold
    q[16g + r, 128b + 64h + 16kq + j], j = 0..15."""
    n, rows, cols = q.shape
    t = q.reshape(n, rows // 16, 16, cols // 128, 2, 2, 2, 16)   # n, g, r, b, h, kq//2, kq%2, j
    return np.ascontiguousarray(t.transpose(0, 1, 3, 4, 6, 5, 2, 7)).reshape(n, rows, cols)


def quantize_weights_gpu(moe, wg, wu, wd):
    """fp32 host stacks -> device (packed q, s) triples quantized and packed by the library."""
    out = []
    for w in (wg, wu, wd):
        e, n, k = w.shape
        dw = to_dev(w)
        q = torch.empty((e, n, k), dtype=torch.uint8, device="cuda")
        s = torch.empty((e, n // 128, k // 128), dtype=torch.float32, device="cuda")
        moe.moe_quant_weight(dw, q, s)
        packed = torch.empty_like(q)
        moe.moe_pack_weight(q, packed)
        out += [packed, s]
        del dw, q
    torch.cuda.synchronize()
    return tuple(out)


def generated_layer_gpu(moe, w: synth.Workload, layer: int = 0):
    """Full layer: fp32 experts drawn on the GPU one by one, quantized and packed in place."""
    e, i, h = w.n_experts, w.inter, w.hidden
    qg = torch.empty((e, i, h), dtype=torch.uint8, device="cuda")
    qu = torch.empty((e, i, h), dtype=torch.uint8, device="cuda")
    qd = torch.empty((e, h, i), dtype=torch.uint8, device="cuda")
    sg = torch.empty((e, i // 128, h // 128), dtype=torch.float32, device="cuda")
    su = torch.empty((e, i // 128, h // 128), dtype=torch.float32, device="cuda")
    sd = torch.empty((e, h // 128, i // 128), dtype=torch.float32, device="cuda")
    tmp = torch.empty((max(i, h) * max(i, h),), dtype=torch.uint8, device="cuda")
    for x in range(e):
        for which, (q, s) in enumerate(((qg, sg), (qu, su), (qd, sd))):
            f = synth.expert_weight_device(w, layer, x, which)
            rowmajor = tmp[:f.numel()].view(f.shape)
            moe.moe_quant_weight(f, rowmajor, s[x])
            moe.moe_pack_weight(rowmajor, q[x])
    torch.cuda.synchronize()
    return qg, sg, qu, su, qd, sd


def oracle_expert_weights(w: synth.Workload, experts, layer: int = 0):
    """Oracle-side weights of some experts: re-drawn in fp32, quantized by the oracle."""
    res = {}
    for x in experts:
        mats = []
        for which in range(3):
            f = synth.expert_weight_device(w, layer, int(x), which).cpu().numpy()
            mats += list(oracle.quantize_weight(f))
        res[int(x)] = tuple(mats)
    return res


def oracle_tokens(x_bits, ids, wts, tokens, ow):
    """Oracle output rows (bf16 bits) of some tokens, from per-expert weights ow."""
    qx, sx = oracle.quant_act(x_bits[tokens])
    k = ids.shape[1]
    outs = []
    for r, t in enumerate(tokens):
        ys = []
        for j in range(k):
            qg, sg, qu, su, qd, sd = ow[int(ids[t, j])]
            ys.append(oracle.expert_rows(qx[r:r + 1], sx[r:r + 1], qg, sg, qu, su, qd, sd)[0])
        outs.append(oracle.combine(np.stack(ys), np.arange(k, dtype=np.int32), wts[t:t + 1])[0])
    return np.stack(outs)


def rel_err(got_f32: np.ndarray, ref_f32: np.ndarray) -> float:
    den = float(np.max(np.abs(ref_f32)))
    return float(np.max(np.abs(got_f32.astype(np.float64) - ref_f32))) / (den if den > 0 else 1.0)


def bits_to_f32(t: torch.Tensor) -> np.ndarray:
    return oracle.bf16_to_f32(t.cpu().numpy().view(np.uint16))


def oracle_expert_weights_pooled(w: synth.Workload, experts, layer: int = 0, batch: int = 16):
    """oracle_expert_weights for many experts: the fp32 matrices are re-drawn on
    the GPU in batches and quantized by the oracle on a pool of CPU processes."""
    import oracle_pool
    experts = [int(e) for e in experts]
    jobs = [(e, which) for e in experts for which in range(3)]
    mats = {}
    for i in range(0, len(jobs), batch):
        part = jobs[i:i + batch]
        f32s = [synth.expert_weight_device(w, layer, e, which).cpu().numpy() for e, which in part]
        for key, qs in zip(part, oracle_pool.quantize_weights(f32s)):
            mats[key] = qs
        del f32s
    return {e: mats[(e, 0)] + mats[(e, 1)] + mats[(e, 2)] for e in experts}


def oracle_tokens_grouped(x_bits, ids, wts, tokens, ow):
    """Oracle output rows (bf16 bits) of some tokens, the layer's steps in order:
    quantize the tokens, sort their slots by expert, run each expert once over
    its rows, combine in slot order (the experts of the tokens, relabelled in
    ascending order, so the sort and the combine order are those of the layer)."""
    tokens = list(tokens)
    qx, sx = oracle.quant_act(x_bits[tokens])
    sub = np.asarray(ids[tokens])
    k = sub.shape[1]
    uniq = sorted(set(sub.reshape(-1).tolist()))
    relabel = np.vectorize({e: i for i, e in enumerate(uniq)}.get)(sub).astype(np.int32)
    offsets, src, dest = oracle.permute(relabel, len(uniq))
    y = np.zeros((len(tokens) * k, x_bits.shape[1]), np.float32)
    for i, e in enumerate(uniq):
        p0, p1 = int(offsets[i]), int(offsets[i + 1])
        rows = src[p0:p1] // k
        y[p0:p1] = oracle.expert_rows(qx[rows], sx[rows], *ow[e])
    return oracle.combine(y, dest, np.asarray(wts[tokens]))
