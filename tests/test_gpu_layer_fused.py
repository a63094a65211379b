"""GPU: the one-call layer (moe_ffn_layer) against the four-call path and the oracle.

moe_ffn_layer runs the arithmetic of moe_quant_act -> moe_permute ->
moe_expert_ffn -> moe_combine in fewer launches (quantization and the slot
sort in one launch for T <= 256; in the decode regime with T * k <= 16 the
down projection and the combine in one launch, each workgroup combining its
output columns of every active expert in LDS).  Bar: its output equals the four-call path's bit for bit,
and the oracle's within 2e-2 (max|out - ref| / max|ref|).
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_cases import (bf16_dev, bits_to_f32, generated_layer_gpu, log, quantize_weights_gpu, rel_err,
                       require_gpu, to_dev)

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.fixture(scope="module")
def moe():
    return require_gpu()


def _layer_inputs(h, i, e, k, t, routing, seed=0):
    w = synth.Workload("fused", h, i, e, k, t, routing, 1.0 if routing == "zipf" else 0.0, "sigmoid", seed=seed)
    x = synth.activations(w)
    ids, wts = synth.routing(w)
    return w, x, ids, wts


def _run(moe, w, x, ids, wts, dweights, regime, fused):
    buf = moe.MoELayerBuffers(w.hidden, w.inter, w.n_experts, w.topk, w.tokens, regime, fused=fused)
    moe.run_layer(buf, bf16_dev(x), to_dev(ids), to_dev(wts), dweights)
    torch.cuda.synchronize()
    return buf


CASES = [
    # (hidden, inter, experts, topk, tokens, routing, regime)
    (256, 128, 8, 2, 1, "uniform", "decode"),
    (1024, 512, 16, 4, 4, "uniform", "decode"),     # h quantized in the down kernel
    (1024, 512, 16, 4, 5, "zipf", "decode"),        # separate h quantization
    (768, 384, 32, 8, 2, "zipf", "decode"),         # T * k = 16, three K blocks over four waves
    (512, 256, 4, 4, 2, "uniform", "decode"),       # k == E, T = 2: every expert has both tokens
    (768, 384, 32, 8, 4, "zipf", "decode"),         # T * k = 32: separate down and combine
    (768, 384, 32, 8, 17, "uniform", "decode"),     # two token operands, separate down and combine
    (768, 384, 32, 8, 33, "zipf", "decode"),        # four token operands
    (768, 384, 32, 8, 64, "zipf", "decode"),        # decode limit
    (256, 128, 4, 4, 5, "uniform", "decode"),       # k == E
    (512, 256, 8, 2, 65, "zipf", "prefill"),
    (512, 256, 8, 2, 256, "uniform", "prefill"),    # last one-launch prologue
    (512, 256, 8, 2, 257, "zipf", "prefill"),       # separate quantization and sort
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c[:5])) + c[5] + "_" + c[6])
def test_fused_layer_equals_four_calls_and_oracle(moe, case):
    h, i, e, k, t, routing, regime = case
    rg = moe.MOE_REGIME_DECODE if regime == "decode" else moe.MOE_REGIME_PREFILL
    w, x, ids, wts = _layer_inputs(h, i, e, k, t, routing)
    wg, wu, wd = synth.weights_host(w)
    dweights = quantize_weights_gpu(moe, wg, wu, wd)
    log(f"fused layer {case}")
    a = _run(moe, w, x, ids, wts, dweights, rg, fused=True)
    b = _run(moe, w, x, ids, wts, dweights, rg, fused=False)
    assert int(a.dev_status.item()) == 0
    assert np.array_equal(a.out.cpu().numpy(), b.out.cpu().numpy())
    ref = oracle.moe_layer(x, ids, wts, oracle.prepare_weights(wg, wu, wd))
    err = rel_err(bits_to_f32(a.out), oracle.bf16_to_f32(ref))
    log(f"  out rel err {err:.3e}")
    assert err <= TOL


def test_fused_layer_back_to_back_calls_share_a_workspace(moe):
    """Two calls in a row on one workspace (the combine counters are cleared
    by every call), the second with fewer tokens; then the first again."""
    w, x, ids, wts = _layer_inputs(1024, 512, 16, 4, 48, "zipf", seed=2)
    wg, wu, wd = synth.weights_host(w)
    dweights = quantize_weights_gpu(moe, wg, wu, wd)
    buf = moe.MoELayerBuffers(w.hidden, w.inter, w.n_experts, w.topk, w.tokens, moe.MOE_REGIME_DECODE, fused=True)
    dims = buf.dims
    outs = []
    for t in (48, 3, 48):
        out = torch.empty((t, w.hidden), dtype=torch.int16, device="cuda")
        moe.moe_ffn_layer(dims, t, moe.MOE_REGIME_DECODE, bf16_dev(x[:t]), to_dev(ids[:t]), to_dev(wts[:t]),
                          *dweights, out, buf.dev_status, buf.layer_ws)
        outs.append(out)
    torch.cuda.synchronize()
    for t, out in zip((48, 3, 48), outs):
        ref = _run(moe, w.with_tokens(t), x[:t], ids[:t], wts[:t], dweights, moe.MOE_REGIME_DECODE, fused=False)
        assert np.array_equal(out.cpu().numpy(), ref.out.cpu().numpy()), t


@pytest.mark.parametrize("regime,tokens", [("decode", 24), ("prefill", 24), ("decode", 2), ("decode", 3)])
def test_fused_layer_reports_bad_ids(moe, regime, tokens):
    """Bad routing ids are reported and parked as by the separate sort, also
    for the smallest batches (T = 2, 3: one-row experts, fused down + combine)."""
    rg = moe.MOE_REGIME_DECODE if regime == "decode" else moe.MOE_REGIME_PREFILL
    w, x, ids, wts = _layer_inputs(512, 256, 8, 2, tokens, "uniform", seed=6)
    ids = ids.copy()
    bad = (0, 1) if tokens <= 3 else (3, 7)
    ids[bad[0], 1] = 8                  # out of range
    ids[bad[1], 1] = ids[bad[1], 0]     # repeated in one token
    wg, wu, wd = synth.weights_host(w)
    dweights = quantize_weights_gpu(moe, wg, wu, wd)
    a = _run(moe, w, x, ids, wts, dweights, rg, fused=True)
    b = _run(moe, w, x, ids, wts, dweights, rg, fused=False)
    st = int(a.dev_status.item())
    assert st == int(b.dev_status.item())
    assert st & moe.MOE_DEV_BAD_EXPERT_ID and st & moe.MOE_DEV_DUP_EXPERT_ID
    good = [t for t in range(w.tokens) if t not in bad]  # outputs of the bad tokens are unspecified
    assert np.array_equal(a.out.cpu().numpy()[good], b.out.cpu().numpy()[good])


@pytest.mark.parametrize("bad_kind", ["range", "dup", "both"])
def test_one_token_layer_reports_bad_ids(moe, bad_kind):
    """One token (no sort launch): an id outside [0, E) and an id repeated in
    the token's top-k set the same dev_status bits as the sort does."""
    w, x, ids, wts = _layer_inputs(512, 256, 16, 4, 1, "uniform", seed=8)
    ids = ids.copy()
    if bad_kind in ("range", "both"):
        ids[0, 1] = 16 if bad_kind == "range" else -3
    if bad_kind in ("dup", "both"):
        ids[0, 3] = ids[0, 0]
    wg, wu, wd = synth.weights_host(w)
    dweights = quantize_weights_gpu(moe, wg, wu, wd)
    a = _run(moe, w, x, ids, wts, dweights, moe.MOE_REGIME_DECODE, fused=True)
    b = _run(moe, w, x, ids, wts, dweights, moe.MOE_REGIME_DECODE, fused=False)
    st = int(a.dev_status.item())
    assert st == int(b.dev_status.item())
    want = {"range": moe.MOE_DEV_BAD_EXPERT_ID, "dup": moe.MOE_DEV_DUP_EXPERT_ID,
            "both": moe.MOE_DEV_BAD_EXPERT_ID | moe.MOE_DEV_DUP_EXPERT_ID}[bad_kind]
    assert st == want


def test_fused_layer_zero_tokens_and_small_workspace(moe):
    w, x, ids, wts = _layer_inputs(256, 128, 8, 2, 4, "uniform")
    wg, wu, wd = synth.weights_host(w)
    dweights = quantize_weights_gpu(moe, wg, wu, wd)
    dims = moe.MoeDims(w.hidden, w.inter, w.n_experts, w.topk)
    out = torch.empty((4, w.hidden), dtype=torch.int16, device="cuda")
    ws = torch.empty(256, dtype=torch.uint8, device="cuda")
    moe.moe_ffn_layer(dims, 0, moe.MOE_REGIME_AUTO, bf16_dev(x[:0]), to_dev(ids[:0]), to_dev(wts[:0]), *dweights,
                      out[:0], None, ws)
    with pytest.raises(moe.MoEError):
        moe.moe_ffn_layer(dims, 4, moe.MOE_REGIME_AUTO, bf16_dev(x), to_dev(ids), to_dev(wts), *dweights, out,
                          None, ws)
    torch.cuda.synchronize()


@pytest.fixture(scope="module")
def deepseek_layer(moe):
    log("generating the full DeepSeek-V3 expert layer on the GPU")
    return generated_layer_gpu(moe, synth.WORKLOADS["decode1"], layer=0)


@pytest.mark.parametrize("name", ["decode1", "decode2", "decode4", "decode64_zipf"])
def test_fused_layer_deepseek_decode_equals_four_calls(moe, deepseek_layer, name):
    """The DeepSeek-V3 layer in one call equals the four calls bit for bit:
    at one token the two-launch path (gate/up with its own quantization and
    no sort, then the fused down + combine), at two tokens the sort with the
    fused down + combine (T * k = 16), beyond it the separate kernels."""
    import dataclasses
    w = (dataclasses.replace(synth.WORKLOADS["decode4"], name="decode2", tokens=2) if name == "decode2"
         else synth.WORKLOADS[name])
    x = synth.activations(w)
    ids, wts = synth.routing(w)
    log(f"deepseek fused {name}")
    a = _run(moe, w, x, ids, wts, deepseek_layer, moe.MOE_REGIME_AUTO, fused=True)
    b = _run(moe, w, x, ids, wts, deepseek_layer, moe.MOE_REGIME_AUTO, fused=False)
    assert int(a.dev_status.item()) == 0
    assert np.array_equal(a.out.cpu().numpy(), b.out.cpu().numpy())


@pytest.mark.parametrize("h,i,e,k,t,regime", [
    (256, 128, 1, 1, 3, "decode"),        # a single expert
    (256, 128, 1, 1, 300, "prefill"),
    (256, 128, 1024, 32, 2, "decode"),    # E = 1024, k = 32: the widest sort
    (256, 128, 1024, 16, 1, "decode"),    # E = 1024, T * k = 16: fused down + combine over four 256-expert chunks
    (256, 128, 300, 8, 2, "decode"),      # E = 300: fused down + combine, a partial second chunk
    (256, 128, 32, 16, 1, "decode"),      # one token, k = 16: the most slots of the one-token path
    (8192, 256, 8, 4, 1, "decode"),       # one token at the largest H the one-token path takes
    (8320, 256, 8, 4, 1, "decode"),       # one token with H > 8192: through the sort
    (128, 128, 4, 2, 1, "decode"),        # one token, one K block: a gate/up wave without blocks
    (256, 128, 1024, 32, 40, "prefill"),
    (384, 128, 8, 2, 9, "decode"),        # H a multiple of 128 but not of 256 (decode only)
    (8448, 256, 4, 2, 40, "prefill"),     # K = 8448 > 8192: row scales beyond one 16-load batch
], ids=lambda v: str(v))
def test_fused_layer_edge_shapes(moe, h, i, e, k, t, regime):
    rg = moe.MOE_REGIME_DECODE if regime == "decode" else moe.MOE_REGIME_PREFILL
    w, x, ids, wts = _layer_inputs(h, i, e, k, t, "uniform", seed=11)
    wg, wu, wd = synth.weights_host(w)
    dweights = quantize_weights_gpu(moe, wg, wu, wd)
    a = _run(moe, w, x, ids, wts, dweights, rg, fused=True)
    b = _run(moe, w, x, ids, wts, dweights, rg, fused=False)
    assert int(a.dev_status.item()) == 0
    assert np.array_equal(a.out.cpu().numpy(), b.out.cpu().numpy())
    ref = oracle.moe_layer(x, ids, wts, oracle.prepare_weights(wg, wu, wd))
    assert rel_err(bits_to_f32(a.out), oracle.bf16_to_f32(ref)) <= TOL


def test_fused_layer_prefill_rejects_h_not_multiple_of_256(moe):
    w, x, ids, wts = _layer_inputs(384, 128, 8, 2, 9, "uniform")
    wg, wu, wd = synth.weights_host(w)
    dweights = quantize_weights_gpu(moe, wg, wu, wd)
    buf = moe.MoELayerBuffers(w.hidden, w.inter, w.n_experts, w.topk, w.tokens, moe.MOE_REGIME_PREFILL, fused=True)
    with pytest.raises(moe.MoEError):
        moe.run_layer(buf, bf16_dev(x), to_dev(ids), to_dev(wts), dweights)
    torch.cuda.synchronize()



def test_fused_layer_prefill_rejects_k_beyond_its_limit(moe):
    """K <= 24576 in the prefill regime (the [2][K/128] weight-scale table is
    loaded one entry per thread); H = 24832 is rejected before anything runs
    (the decode regime stops at H = 16384)."""
    w, x, ids, wts = _layer_inputs(24832, 128, 2, 1, 4, "uniform")
    wg, wu, wd = synth.weights_host(w)
    dweights = quantize_weights_gpu(moe, wg, wu, wd)
    buf = moe.MoELayerBuffers(w.hidden, w.inter, w.n_experts, w.topk, w.tokens, moe.MOE_REGIME_PREFILL, fused=True)
    with pytest.raises(moe.MoEError):
        moe.run_layer(buf, bf16_dev(x), to_dev(ids), to_dev(wts), dweights)
    torch.cuda.synchronize()
