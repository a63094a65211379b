"""CPU oracle of the routed-expert FP8 MoE FFN.  TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import or run this module.  The GPU library never does: it
shares no code, table or constant generator with this file.

It is a plain, slow, numpy statement of what one routed-expert MoE layer
computes, written from the paper:

* Background and Motivation, "FP8 Block Scaling Format": weights are FP8
  E4M3 with shared fp32 scale factors; on the GPU path activations are
  quantized to FP8 and the GEMM runs FP8 x FP8 with FP32 accumulation.
* AVX-512 FP8 GEMV Kernel, "FP8 Format and Dequantization Strategy": the
  E4M3FN format (1 sign, 4 exponent, 3 mantissa bits).
* AVX-512 FP8 GEMV Kernel, "Tiling and Scale-Block Optimizations": K is
  walked in 128-element scale blocks, all partial products of a block are
  accumulated first and the block's scale is applied once.
* Fine-grained CPU Parallelism for MoE Inference, Figure mlp-flow and
  "Operator Fusion for Quantized Inference": an expert is gate and up
  (independent), SiLU(gate) times up, then down; the expert outputs are
  accumulated with the router weights in F32 and converted back to the
  hidden type.
* Distributed Stream-loading Prefill (standard EP workflow) and Multi-GPU
  Parallelism: tokens are sorted by expert into per-expert token lists.

Readings where the paper is silent (each also listed in the design notes):
OCP E4M3 with max 448 and NaN at S.1111.111 (the paper describes the
format as free of NaNs; read as free of infinities, the OCP "FN" variant); the scale is a multiplicative dequantization
factor s = amax/448; x/s is a correctly rounded fp32 division; rounding to
e4m3 is to nearest with ties to the even code, |v| > 448 saturates to 448,
the sign of zero is kept; an all-zero block gets s = 0 and signed-zero
codes; the input of the down projection is also quantized (W8A8 for both
GEMMs); the per-expert sort is stable in the flat index t*k+j; combine sums
in slot order in fp32 from +0.0 and rounds once to bf16.

Precision: every value is fp32 except one step.  The dot product of a 128-
element block of e4m3 codes is formed exactly (fp64 holds every partial sum
of products of two e4m3 values exactly: they are multiples of 2^-18 below
2^25), then rounded once to fp32; the per-block scale product and the
accumulation over blocks (ascending) are fp32.  Inputs must be finite.
"""
from __future__ import annotations

import concurrent.futures as _cf
import math
import os

import numpy as np

BLOCK = 128
E4M3_MAX = 448.0

f32 = np.float32


# --------------------------------------------------------------------------
# FP8 E4M3 (OCP "FN" variant) -- AVX-512 FP8 GEMV Kernel, FP8 format.
# --------------------------------------------------------------------------
def _e4m3_value(code: int) -> float:
    """Value of one e4m3 code by the OCP definition (bias 7, no infinities)."""
    sign = code >> 7
    exp = (code >> 3) & 0xF
    man = code & 0x7
    if exp == 15 and man == 7:
        return math.nan
    if exp == 0:
        mag = math.ldexp(man / 8.0, -6)          # subnormal: 2^-6 * m/8
    else:
        mag = math.ldexp(1.0 + man / 8.0, exp - 7)
    return -mag if sign else mag


E4M3_TABLE = np.array([_e4m3_value(c) for c in range(256)], dtype=np.float64)
# Non-negative finite magnitudes, ascending with the code: codes 0x00..0x7E.
_E4M3_POS = E4M3_TABLE[:0x7F].copy()


def e4m3_decode(codes: np.ndarray) -> np.ndarray:
    """e4m3 codes -> exact values (fp64; every e4m3 value is exact in fp32 too)."""
    return E4M3_TABLE[np.asarray(codes, dtype=np.uint8)]


def e4m3_encode(v: np.ndarray) -> np.ndarray:
    """Round fp32 values to e4m3 codes.

    Nearest representable value, ties to the even code (the code whose
    mantissa LSB is 0), |v| > 448 saturates to 448, sign kept (so -0 and
    negative values that round to zero give 0x80).  Large arrays are split
    into chunks handled on a thread pool; each element is independent.
    """
    v = np.asarray(v, dtype=np.float32)
    if v.size > _PAR_MIN:
        flat = v.reshape(-1)
        out = np.empty(flat.shape, dtype=np.uint8)
        step = _PAR_MIN

        def work(i0):
            out[i0:i0 + step] = _encode_chunk(flat[i0:i0 + step])

        with _cf.ThreadPoolExecutor(max_workers=os.cpu_count() or 1) as ex:
            list(ex.map(work, range(0, flat.size, step)))
        return out.reshape(v.shape)
    return _encode_chunk(v)


_PAR_MIN = 1 << 20


def _encode_chunk(v: np.ndarray) -> np.ndarray:
    sign = (np.signbit(v).astype(np.uint8) << 7).astype(np.uint8)
    a = np.minimum(np.abs(v.astype(np.float64)), E4M3_MAX)
    hi = np.searchsorted(_E4M3_POS, a, side="left")       # first value >= a
    hi = np.minimum(hi, 0x7E)
    lo = np.maximum(hi - 1, 0)
    d_hi = _E4M3_POS[hi] - a
    d_lo = a - _E4M3_POS[lo]
    take_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    code = np.where(take_hi, hi, lo).astype(np.uint8)
    return code | sign


# --------------------------------------------------------------------------
# bf16 <-> fp32 (the hidden type of the layer)
# --------------------------------------------------------------------------
def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> the exact fp32 values."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def f32_to_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    return ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)


# --------------------------------------------------------------------------
# Block quantization -- FP8 Block Scaling Format; scale blocks of 128.
# --------------------------------------------------------------------------
def _quantize_groups(xg: np.ndarray):
    """Quantize groups along the last axis; xg fp32 [..., n]. Returns (q, s)."""
    a = np.max(np.abs(xg), axis=-1)                        # exact
    s = (a.astype(np.float32) / f32(E4M3_MAX)).astype(np.float32)
    s_b = s[..., None]
    v = np.divide(xg, s_b, out=np.array(xg, dtype=np.float32, copy=True),
                  where=s_b > 0).astype(np.float32)        # s == 0: keep the signed zeros
    return e4m3_encode(v), s


def quantize_rows(x: np.ndarray):
    """Per row, per 128 consecutive channels: x fp32 [R, K] -> (q u8 [R,K], s f32 [R,K/128])."""
    x = np.asarray(x, dtype=np.float32)
    r, k = x.shape
    if k % BLOCK:
        raise ValueError("K must be a multiple of 128")
    q, s = _quantize_groups(x.reshape(r, k // BLOCK, BLOCK))
    return q.reshape(r, k), s


def quant_act(x_bf16: np.ndarray):
    """Activation quantization of bf16 tokens [T, H] (bf16 -> exact fp32 -> quantize_rows)."""
    return quantize_rows(bf16_to_f32(x_bf16))


def quantize_weight(w: np.ndarray):
    """128x128 block quantization of one matrix w fp32 [N, K] -> (q u8 [N,K], s f32 [N/128, K/128])."""
    w = np.asarray(w, dtype=np.float32)
    n, k = w.shape
    if n % BLOCK or k % BLOCK:
        raise ValueError("weight dims must be multiples of 128")
    g = w.reshape(n // BLOCK, BLOCK, k // BLOCK, BLOCK).transpose(0, 2, 1, 3)
    q, s = _quantize_groups(g.reshape(n // BLOCK, k // BLOCK, BLOCK * BLOCK))
    q = q.reshape(n // BLOCK, k // BLOCK, BLOCK, BLOCK).transpose(0, 2, 1, 3).reshape(n, k)
    return np.ascontiguousarray(q), s


def quantize_experts(w: np.ndarray):
    """quantize_weight over a stack [E, N, K]."""
    qs, ss = zip(*(quantize_weight(m) for m in w))
    return np.stack(qs), np.stack(ss)


# --------------------------------------------------------------------------
# Permutation -- sort tokens by expert into per-expert token lists.
# --------------------------------------------------------------------------
def check_routing(ids: np.ndarray, n_experts: int):
    ids = np.asarray(ids)
    if ids.ndim != 2:
        raise ValueError("topk_ids must be [T, k]")
    if ids.size and (ids.min() < 0 or ids.max() >= n_experts):
        raise ValueError("expert id out of range")
    s = np.sort(ids, axis=1)
    if ids.shape[1] > 1 and np.any(s[:, 1:] == s[:, :-1]):
        raise ValueError("duplicate expert id within a token's top-k")


def permute(ids: np.ndarray, n_experts: int):
    """Stable counting sort of the flat slots f = t*k + j by expert id.

    Returns (expert_offsets [E+1], sorted_src [T*k] = f at sorted position p,
    dest_row [T*k] = sorted position of slot f), all int32.
    """
    check_routing(ids, n_experts)
    flat = np.asarray(ids, dtype=np.int64).reshape(-1)
    counts = np.bincount(flat, minlength=n_experts)
    offsets = np.zeros(n_experts + 1, dtype=np.int64)
    np.cumsum(counts, out=offsets[1:])
    order = np.argsort(flat, kind="stable")
    dest = np.empty_like(order)
    dest[order] = np.arange(flat.size)
    return offsets.astype(np.int32), order.astype(np.int32), dest.astype(np.int32)


# --------------------------------------------------------------------------
# Block-scaled FP8 GEMM (FP32 accumulation, one scale per 128-K block).
# --------------------------------------------------------------------------
def block_scaled_matmul(a_q, a_s, w_q, w_s) -> np.ndarray:
    """C[m,n] = sum_b fl32(a_s[m,b]*w_s[n/128,b]) * fl32(exact sum_{i in b} a[m,i]*w[n,i]).

    a_q u8 [M,K], a_s f32 [M,K/128]; w_q u8 [N,K] (row n is output n,
    K contiguous), w_s f32 [N/128, K/128].  Blocks b are accumulated in
    ascending order in fp32, starting from +0.0.
    """
    a = e4m3_decode(a_q)
    w = e4m3_decode(w_q)
    m, k = a.shape
    n = w.shape[0]
    acc = np.zeros((m, n), dtype=np.float32)
    for b in range(k // BLOCK):
        sl = slice(b * BLOCK, (b + 1) * BLOCK)
        d = (a[:, sl] @ w[:, sl].T).astype(np.float32)     # exact, then one rounding
        scale = (a_s[:, b][:, None].astype(np.float32)
                 * np.repeat(w_s[:, b], BLOCK)[None, :].astype(np.float32)).astype(np.float32)
        acc = (acc + (d * scale).astype(np.float32)).astype(np.float32)
    return acc


def silu_mul(g: np.ndarray, u: np.ndarray) -> np.ndarray:
    """h = g * sigmoid(g) * u in fp32, sigmoid(g) = 1 / (1 + exp(-g))."""
    g = np.asarray(g, dtype=np.float32)
    with np.errstate(over="ignore"):
        sig = (f32(1.0) / (f32(1.0) + np.exp(-g))).astype(np.float32)
    return ((g * sig).astype(np.float32) * np.asarray(u, dtype=np.float32)).astype(np.float32)


def expert_rows(qx, sx, q_gate, s_gate, q_up, s_up, q_down, s_down, want_intermediates=False):
    """One expert applied to rows of quantized activations.

    gate and up projections, SiLU(gate)*up, quantization of h per row per
    128 channels, then the down projection.  Returns y fp32 [M, H] (and the
    intermediates G, U, h, qh, sh when asked).
    """
    g = block_scaled_matmul(qx, sx, q_gate, s_gate)
    u = block_scaled_matmul(qx, sx, q_up, s_up)
    h = silu_mul(g, u)
    qh, sh = quantize_rows(h)
    y = block_scaled_matmul(qh, sh, q_down, s_down)
    if want_intermediates:
        return y, dict(g=g, u=u, h=h, qh=qh, sh=sh)
    return y


def expert_ffn(qx, sx, expert_offsets, sorted_src, topk, weights, experts=None,
               want_intermediates=False):
    """Expert FFN over the expert-sorted rows.

    weights = (q_gate [E,I,H], s_gate [E,I/128,H/128], q_up, s_up,
    q_down [E,H,I], s_down [E,H/128,I/128]).  Row p of the result belongs
    to token sorted_src[p] // topk and to the expert e with
    expert_offsets[e] <= p < expert_offsets[e+1].  Returns y_rows fp32
    [T*k, H] (rows of experts not in ``experts`` stay zero when a subset is
    given).
    """
    qg, sg, qu, su, qd, sd = weights
    n_rows = int(expert_offsets[-1])
    hidden = qd.shape[1]
    inter = qd.shape[2]
    y = np.zeros((n_rows, hidden), dtype=np.float32)
    inter_rows = None
    if want_intermediates:
        inter_rows = dict(g=np.zeros((n_rows, inter), np.float32),
                          u=np.zeros((n_rows, inter), np.float32),
                          h=np.zeros((n_rows, inter), np.float32),
                          qh=np.zeros((n_rows, inter), np.uint8),
                          sh=np.zeros((n_rows, inter // BLOCK), np.float32))
    n_exp = len(expert_offsets) - 1
    for e in range(n_exp) if experts is None else experts:
        p0, p1 = int(expert_offsets[e]), int(expert_offsets[e + 1])
        if p1 == p0:
            continue
        tok = np.asarray(sorted_src[p0:p1]) // topk
        out = expert_rows(qx[tok], sx[tok], qg[e], sg[e], qu[e], su[e], qd[e], sd[e],
                          want_intermediates)
        if want_intermediates:
            y[p0:p1], d = out
            for key in inter_rows:
                inter_rows[key][p0:p1] = d[key]
        else:
            y[p0:p1] = out
    return (y, inter_rows) if want_intermediates else y


def combine(y_rows, dest_row, topk_w) -> np.ndarray:
    """out[t] = bf16(sum over slots j in order of w[t,j] * y_rows[dest_row[t*k+j]]).

    fp32 products and sums from +0.0, one round-to-nearest-even to bf16.
    Returns bf16 bit patterns [T, H].
    """
    topk_w = np.asarray(topk_w, dtype=np.float32)
    t, k = topk_w.shape
    dest = np.asarray(dest_row).reshape(t, k)
    acc = np.zeros((t, y_rows.shape[1]), dtype=np.float32)
    for j in range(k):
        acc = (acc + (topk_w[:, j][:, None] * y_rows[dest[:, j]]).astype(np.float32)).astype(np.float32)
    return f32_to_bf16(acc)


def prepare_weights(w_gate, w_up, w_down):
    """fp32 expert stacks -> (q_gate, s_gate, q_up, s_up, q_down, s_down)."""
    qg, sg = quantize_experts(w_gate)
    qu, su = quantize_experts(w_up)
    qd, sd = quantize_experts(w_down)
    return qg, sg, qu, su, qd, sd


def moe_layer(x_bf16, topk_ids, topk_w, weights, want_intermediates=False):
    """The whole routed-expert layer: quantize -> permute -> expert FFN -> combine."""
    n_exp = weights[0].shape[0]
    topk = topk_ids.shape[1]
    qx, sx = quant_act(x_bf16)
    offsets, sorted_src, dest_row = permute(topk_ids, n_exp)
    res = expert_ffn(qx, sx, offsets, sorted_src, topk, weights,
                     want_intermediates=want_intermediates)
    y, inter = res if want_intermediates else (res, None)
    out = combine(y, dest_row, topk_w)
    if want_intermediates:
        return out, dict(qx=qx, sx=sx, offsets=offsets, sorted_src=sorted_src,
                         dest_row=dest_row, y=y, **inter)
    return out


# --------------------------------------------------------------------------
# W8A16 -- the paper's CPU GEMV numerics (AVX-512 FP8 GEMV Kernel: FP8 weights
# expanded to BF16, BF16 x BF16 dot products accumulated in FP32, the block's
# scale applied once to the accumulated block sum; Tiling and Scale-Block
# Optimizations: K walked in 128-element blocks).  Activations stay bf16; h
# is rounded to bf16 (the hidden type) before the down projection.
# --------------------------------------------------------------------------
def block_scaled_matmul_w8a16(a_bf16, w_q, w_s) -> np.ndarray:
    """C[m,n] = sum_b fl32(w_s[n/128,b] * fl32(exact sum_{i in b} a[m,i]*w[n,i])).

    a_bf16 uint16 bf16 bits [M,K]; w_q u8 [N,K]; w_s f32 [N/128, K/128].
    A bf16 x e4m3 product has at most 12 significant bits, so fp64 holds the
    block sums exactly for activations within a 2^40 range of one another
    (any realistic data); blocks are accumulated in ascending order in fp32.
    """
    a = bf16_to_f32(a_bf16).astype(np.float64)
    w = e4m3_decode(w_q)
    m, k = a.shape
    n = w.shape[0]
    acc = np.zeros((m, n), dtype=np.float32)
    for b in range(k // BLOCK):
        sl = slice(b * BLOCK, (b + 1) * BLOCK)
        d = (a[:, sl] @ w[:, sl].T).astype(np.float32)
        scale = np.repeat(w_s[:, b], BLOCK)[None, :].astype(np.float32)
        acc = (acc + (d * scale).astype(np.float32)).astype(np.float32)
    return acc


def expert_rows_w8a16(x_bf16, q_gate, s_gate, q_up, s_up, q_down, s_down, want_intermediates=False):
    """One expert on bf16 activation rows: gate, up, h = bf16(SiLU(G) * U), down."""
    g = block_scaled_matmul_w8a16(x_bf16, q_gate, s_gate)
    u = block_scaled_matmul_w8a16(x_bf16, q_up, s_up)
    h = f32_to_bf16(silu_mul(g, u))
    y = block_scaled_matmul_w8a16(h, q_down, s_down)
    if want_intermediates:
        return y, dict(g=g, u=u, h=h)
    return y


def expert_ffn_w8a16(x_bf16, expert_offsets, sorted_src, topk, weights, experts=None):
    """W8A16 expert FFN over the expert-sorted rows (same layout as expert_ffn)."""
    qg, sg, qu, su, qd, sd = weights
    n_rows = int(expert_offsets[-1])
    y = np.zeros((n_rows, qd.shape[1]), dtype=np.float32)
    for e in range(len(expert_offsets) - 1) if experts is None else experts:
        p0, p1 = int(expert_offsets[e]), int(expert_offsets[e + 1])
        if p1 == p0:
            continue
        tok = np.asarray(sorted_src[p0:p1]) // topk
        y[p0:p1] = expert_rows_w8a16(x_bf16[tok], qg[e], sg[e], qu[e], su[e], qd[e], sd[e])
    return y


def moe_layer_w8a16(x_bf16, topk_ids, topk_w, weights):
    """The routed-expert layer with W8A16 numerics: permute -> expert FFN -> combine."""
    offsets, sorted_src, dest_row = permute(topk_ids, weights[0].shape[0])
    y = expert_ffn_w8a16(np.asarray(x_bf16), offsets, sorted_src, topk_ids.shape[1], weights)
    return combine(y, dest_row, topk_w)


def moe_layer_dense(x_bf16, topk_ids, topk_w, weights):
    """Every expert on every token, masked by routing; no permutation.

    Uses the same per-row functions as ``moe_layer``; the result must equal
    it bit for bit, which checks the permutation and combine bookkeeping.
    """
    qg, sg, qu, su, qd, sd = weights
    check_routing(topk_ids, qg.shape[0])
    qx, sx = quant_act(x_bf16)
    t, k = topk_ids.shape
    acc = np.zeros((t, qd.shape[1]), dtype=np.float32)
    dense = [expert_rows(qx, sx, qg[e], sg[e], qu[e], su[e], qd[e], sd[e])
             for e in range(qg.shape[0])]
    rows = np.arange(t)
    for j in range(k):
        yj = np.stack([dense[topk_ids[r, j]][r] for r in rows])
        acc = (acc + (topk_w[:, j][:, None].astype(np.float32) * yj).astype(np.float32)).astype(np.float32)
    return f32_to_bf16(acc)
