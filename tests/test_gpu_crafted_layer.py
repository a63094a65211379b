"""GPU: the whole layer on crafted values that make every scale count.

The other layer tests draw activations ~N(0,1) and weights ~N(0,0.02), so
every 128-block carries a similar scale, and an operand that took the scale
of a neighbouring block (a wrong scale index, a transposed scale table, a
K block paired with the wrong scale) would move the output by a few per
cent, which can hide inside a 2e-2 bound.  Here each (token, 128-channel)
block of the activations is scaled by 2^a with a in [-16, 16] and each
128x128 block of every weight matrix by 2^b with b in [-8, 8], so any such
mix-up changes an output by orders of magnitude.  Also in the layer: a token
of zeros (its output must be exactly zero), a token with one non-zero block,
an all-zero weight block (scale 0), and a slot with routing weight 0.

Bar (FP8 Block Scaling Format, W8A8 with fp32 promotion): per token,
max|out - ref| / max|ref| <= 2e-2 against the oracle (the tokens' output
maxima span more than 2^40, so one global maximum would hide the small
ones); the
quantized activations, the permutation and the device-quantized weights bit
for bit; both regimes, through the four calls and through moe_ffn_layer.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_cases import bf16_dev, bits_to_f32, log, pack_reference, quantize_weights_gpu, require_gpu, to_dev

TOL = 2e-2
H, I, E, K, T = 512, 256, 8, 2, 24


@pytest.fixture(scope="module")
def moe():
    return require_gpu()


def _crafted(seed=11):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, H)).astype(np.float32)
    x *= np.repeat(np.exp2(rng.integers(-16, 17, (T, H // 128))).astype(np.float32), 128, axis=1)
    x[0] = 0.0                       # a token of zeros
    x[1, 128:] = 0.0                 # one non-zero block
    xb = synth.bf16_bits_from_f32(x)

    def blocks(shape):
        w = 0.02 * rng.standard_normal(shape).astype(np.float32)
        sc = np.exp2(rng.integers(-8, 9, (shape[0], shape[1] // 128, shape[2] // 128))).astype(np.float32)
        return w * np.repeat(np.repeat(sc, 128, axis=1), 128, axis=2)

    wg, wu, wd = blocks((E, I, H)), blocks((E, I, H)), blocks((E, H, I))
    wg[3, 128:256, 256:384] = 0.0    # an all-zero weight block: scale 0
    wd[5, :128, :128] = 0.0
    ids = np.stack([rng.choice(E, K, replace=False) for _ in range(T)]).astype(np.int32)
    ids[2] = [3, 5]                  # a token through both zero blocks
    logits = rng.standard_normal((T, K)).astype(np.float32)
    wts = (1.0 / (1.0 + np.exp(-logits))).astype(np.float32)
    wts /= wts.sum(axis=1, keepdims=True)
    wts[4, 1] = 0.0                  # a slot with routing weight 0
    return xb, ids, wts.astype(np.float32), (wg, wu, wd)


def _per_token_err(got, ref):
    errs = []
    for t in range(got.shape[0]):
        m = np.max(np.abs(ref[t]))
        if m == 0:
            assert np.all(got[t] == 0), f"token {t}: the reference is zero, the output is not"
            errs.append(0.0)
        else:
            errs.append(float(np.max(np.abs(got[t] - ref[t])) / m))
    return np.array(errs)


def test_crafted_inputs_expose_a_misplaced_scale():
    """CPU, the oracle only: a scale table with two blocks swapped, or the
    activation scales of one K block shifted to its neighbour, moves some
    token's output far beyond the bound on these inputs."""
    xb, ids, wts, (wg, wu, wd) = _crafted()
    ow = oracle.prepare_weights(wg, wu, wd)
    ref = oracle.bf16_to_f32(oracle.moe_layer(xb, ids, wts, ow))
    sg = ow[1].copy()
    sg[:, :, [0, 1]] = sg[:, :, [1, 0]]          # W_gate scales of K blocks 0 and 1 swapped
    bad = oracle.bf16_to_f32(oracle.moe_layer(xb, ids, wts, (ow[0], sg) + tuple(ow[2:])))
    assert _per_token_err(bad, ref).max() > 50 * TOL
    qx, sx = oracle.quant_act(xb)
    offsets, sorted_src, dest_row = oracle.permute(ids, E)
    sx_bad = sx.copy()
    sx_bad[:, 2] = sx[:, 3]                      # activation block 2 promoted with block 3's scale
    y = oracle.expert_ffn(qx, sx_bad, offsets, sorted_src, K, ow)
    y = y[0] if isinstance(y, tuple) else y
    bad2 = oracle.bf16_to_f32(oracle.combine(y, dest_row, wts))
    assert _per_token_err(bad2, ref).max() > 50 * TOL


@pytest.mark.gpu
@pytest.mark.parametrize("regime", ["decode", "prefill"])
@pytest.mark.parametrize("fused", [False, True], ids=["four_calls", "moe_ffn_layer"])
def test_layer_on_crafted_scales(moe, regime, fused):
    xb, ids, wts, (wg, wu, wd) = _crafted()
    rg = moe.MOE_REGIME_DECODE if regime == "decode" else moe.MOE_REGIME_PREFILL
    ow = oracle.prepare_weights(wg, wu, wd)
    dweights = quantize_weights_gpu(moe, wg, wu, wd)
    for j, (dq, rq) in enumerate(zip(dweights, ow)):
        assert np.array_equal(dq.cpu().numpy(), pack_reference(rq) if j % 2 == 0 else rq)
    assert ow[1][3, 1, 2] == 0.0 and ow[5][5, 0, 0] == 0.0  # the zero blocks have scale 0
    ref, inter = oracle.moe_layer(xb, ids, wts, ow, want_intermediates=True)
    buf = moe.MoELayerBuffers(H, I, E, K, T, rg, fused=fused)
    moe.run_layer(buf, bf16_dev(xb), to_dev(ids), to_dev(wts), dweights)
    torch.cuda.synchronize()
    assert int(buf.dev_status.item()) == 0
    if not fused:
        assert np.array_equal(buf.qx.cpu().numpy(), inter["qx"])
        assert np.array_equal(buf.sx.cpu().numpy(), inter["sx"])
        assert np.array_equal(buf.sorted_src.cpu().numpy(), inter["sorted_src"])
    got = bits_to_f32(buf.out)
    errs = _per_token_err(got, oracle.bf16_to_f32(ref))
    mags = np.abs(got).max(axis=1)
    log(f"crafted layer {regime} {'fused' if fused else 'four calls'}: worst token {int(errs.argmax())} "
        f"err {errs.max():.3e}; token output maxima 2^{np.log2(mags[mags > 0]).min():.0f}.."
        f"2^{np.log2(mags.max()):.0f}")
    assert errs.max() <= TOL


def _crafted_fullsize(seed=12, E=4, K=2):
    """The same construction at the DeepSeek-V3 widths (H = 7168, I = 2048)
    over 4 experts: gate/up run 56 K blocks (the prefill GEMM's 16-slot
    row-scale batch, the decode kernel's K halves), down 16."""
    h, i = 7168, 2048
    rng = np.random.default_rng(seed)

    def blocks(shape):
        w = 0.02 * rng.standard_normal(shape, dtype=np.float32)
        sc = np.exp2(rng.integers(-8, 9, (shape[0], shape[1] // 128, shape[2] // 128))).astype(np.float32)
        w *= np.repeat(np.repeat(sc, 128, axis=1), 128, axis=2)
        return w

    wg, wu, wd = blocks((E, i, h)), blocks((E, i, h)), blocks((E, h, i))
    wg[1, :128, -128:] = 0.0
    return (wg, wu, wd), rng


@pytest.fixture(scope="module")
def fullsize(moe):
    log("crafted full-width layer: drawing and quantizing 4 experts at H=7168, I=2048")
    (wg, wu, wd), rng = _crafted_fullsize()
    ow = oracle.prepare_weights(wg, wu, wd)
    dweights = quantize_weights_gpu(moe, wg, wu, wd)
    for j, (dq, rq) in enumerate(zip(dweights, ow)):
        assert np.array_equal(dq.cpu().numpy(), pack_reference(rq) if j % 2 == 0 else rq)
    return ow, dweights, rng


@pytest.mark.gpu
@pytest.mark.parametrize("regime,tokens", [("decode", 48), ("prefill", 300)])
def test_fullwidth_layer_on_crafted_scales(moe, fullsize, regime, tokens):
    """48 decode tokens (about 24 rows per expert) and 300 prefill tokens
    (150 rows per expert: two m-tiles each), one moe_ffn_layer call each,
    every token against the oracle with the per-token bound."""
    ow, dweights, rng0 = fullsize
    rng = np.random.default_rng(100 + tokens)
    h, i, e, k = 7168, 2048, 4, 2
    x = rng.standard_normal((tokens, h)).astype(np.float32)
    x *= np.repeat(np.exp2(rng.integers(-16, 17, (tokens, h // 128))).astype(np.float32), 128, axis=1)
    x[0] = 0.0
    xb = synth.bf16_bits_from_f32(x)
    ids = np.stack([rng.choice(e, k, replace=False) for _ in range(tokens)]).astype(np.int32)
    wts = rng.uniform(0.1, 1.0, (tokens, k)).astype(np.float32)
    rg = moe.MOE_REGIME_DECODE if regime == "decode" else moe.MOE_REGIME_PREFILL
    log(f"crafted full-width {regime}: T={tokens}")
    ref = oracle.bf16_to_f32(oracle.moe_layer(xb, ids, wts, ow))
    buf = moe.MoELayerBuffers(h, i, e, k, tokens, rg, fused=True)
    moe.run_layer(buf, bf16_dev(xb), to_dev(ids), to_dev(wts), dweights)
    torch.cuda.synchronize()
    assert int(buf.dev_status.item()) == 0
    errs = _per_token_err(bits_to_f32(buf.out), ref)
    log(f"crafted full-width {regime}: worst token {int(errs.argmax())} err {errs.max():.3e}")
    assert errs.max() <= TOL
