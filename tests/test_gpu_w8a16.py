"""GPU parity of the W8A16 decode FFN (moe_expert_ffn_w8a16) against the
oracle's W8A16 mode (bf16 activations, FP8 weights expanded to bf16, fp32
block sums post-scaled by the weight scale, bf16 h).

Bar: max|out - ref| / max|ref| <= 2e-2 on the bf16 layer output; every e4m3
code expands exactly (a crafted layer whose up projection holds all 254
finite codes, read back element by element).
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_cases import (bits_to_f32, generated_layer_gpu, log, oracle_expert_weights, quantize_weights_gpu, rel_err,
                       require_gpu, to_dev)

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.fixture(scope="module")
def moe():
    return require_gpu()


def _layer(moe, w, x, ids, wts, dev_weights):
    buf = moe.MoELayerBuffers(w.hidden, w.inter, w.n_experts, w.topk, x.shape[0], w8a16=True)
    moe.run_layer(buf, to_dev(x.view(np.int16)), to_dev(ids), to_dev(wts), dev_weights)
    torch.cuda.synchronize()
    assert int(buf.dev_status.item()) == 0
    return buf


@pytest.mark.parametrize("tokens", [16, 1, 5, 64])
def test_w8a16_small_layers(moe, tokens):
    w = synth.Workload("w8a16_small", 512, 256, 16, 4, tokens, "zipf", 1.0)
    x = synth.activations(w)
    ids, wts = synth.routing(w)
    wg, wu, wd = synth.weights_host(w)
    buf = _layer(moe, w, x, ids, wts, quantize_weights_gpu(moe, wg, wu, wd))
    ref = oracle.bf16_to_f32(oracle.moe_layer_w8a16(x, ids, wts, oracle.prepare_weights(wg, wu, wd)))
    err = rel_err(bits_to_f32(buf.out), ref)
    log(f"w8a16 T={tokens}: out rel err {err:.3e}")
    assert err <= TOL


def test_w8a16_tiny_layer(moe):
    w = synth.WORKLOADS["tiny"]
    x = synth.activations(w)
    ids, wts = synth.routing(w)
    wg, wu, wd = synth.weights_host(w)
    buf = _layer(moe, w, x, ids, wts, quantize_weights_gpu(moe, wg, wu, wd))
    ref = oracle.bf16_to_f32(oracle.moe_layer_w8a16(x, ids, wts, oracle.prepare_weights(wg, wu, wd)))
    assert rel_err(bits_to_f32(buf.out), ref) <= TOL


@pytest.mark.parametrize("name", ["decode1", "decode4"])
def test_w8a16_deepseek_decode(moe, name):
    w = synth.WORKLOADS[name]
    x = synth.activations(w)
    ids, wts = synth.routing(w)
    log(f"w8a16 {name}: drawing the full layer on the GPU")
    buf = _layer(moe, w, x, ids, wts, generated_layer_gpu(moe, w))
    ow = oracle_expert_weights(w, sorted(set(ids.reshape(-1).tolist())))
    outs = []
    for t in range(w.tokens):
        ys = [oracle.expert_rows_w8a16(x[t:t + 1], *ow[int(e)])[0] for e in ids[t]]
        outs.append(oracle.combine(np.stack(ys), np.arange(w.topk, dtype=np.int32), wts[t:t + 1])[0])
    err = rel_err(bits_to_f32(buf.out), oracle.bf16_to_f32(np.stack(outs)))
    log(f"  out rel err {err:.3e}")
    assert err <= TOL


def test_w8a16_every_e4m3_code_expands_exactly(moe):
    """One expert, one token x = e_0.  W_gate[:, 0] = 1 and W_up[n, 0] = the
    value of code n (NaN codes replaced by 0), each 128x128 block holding a
    448 elsewhere so that its scale is exactly 1; W_down is the identity
    (plus a 448 per block in columns whose h is zero).  Then y[n] =
    bf16(SiLU(1) * value(code n)): a wrong expansion of any code shows."""
    H = I = 256
    vals = oracle.E4M3_TABLE.astype(np.float64).copy()
    vals[~np.isfinite(vals)] = 0.0
    wg = np.zeros((1, I, H), np.float32)
    wu = np.zeros((1, I, H), np.float32)
    wd = np.zeros((1, H, I), np.float32)
    wg[0, :, 0] = 1.0
    wu[0, :, 0] = vals.astype(np.float32)
    for r in (0, 128):
        for c in (1, 129):
            wg[0, r, c] = 448.0
            wu[0, r, c] = 448.0
    wd[0] = np.eye(H, dtype=np.float32)
    for r in (0, 128):
        for c in (0, 128):          # h[0] = h[128] = 0 (codes 0x00 and 0x80)
            wd[0, r + 1, c] = 448.0
    x = np.zeros((1, H), np.float32)
    x[0, 0] = 1.0
    xb = synth.bf16_bits_from_f32(x)
    w = synth.Workload("w8a16_codes", H, I, 1, 1, 1, "uniform")
    ids = np.zeros((1, 1), np.int32)
    wts = np.ones((1, 1), np.float32)
    buf = _layer(moe, w, xb, ids, wts, quantize_weights_gpu(moe, wg, wu, wd))
    got = buf.y_rows.cpu().numpy()[0]
    weights = oracle.prepare_weights(wg, wu, wd)
    assert np.all(weights[1] == 1.0) and np.all(weights[3] == 1.0) and np.all(weights[5] == 1.0)
    ref = oracle.expert_rows_w8a16(xb, *[m[0] for m in weights])[0]
    silu1 = np.float32(1.0) / (np.float32(1.0) + np.exp(np.float32(-1.0)))
    expect = oracle.bf16_to_f32(oracle.f32_to_bf16((silu1 * vals.astype(np.float32)).astype(np.float32)))
    assert np.allclose(ref, expect, rtol=1e-2, atol=0)
    assert np.allclose(got, ref, rtol=1e-2, atol=0)
    assert np.array_equal(np.signbit(got[vals != 0]), np.signbit(vals[vals != 0]))
