"""GPU: moe_ffn_layer_noalloc (the library's per-GPU scratch array in place of
a caller workspace) against moe_ffn_layer with its own workspace.

Both run the same kernels, so the outputs must be identical bit for bit; a
few tokens are also checked against the CPU oracle (2e-2).  Each case makes
two calls in a row on one GPU, the second with fewer tokens, so the second
call runs over the scratch contents the first one left.  The layer has the
DeepSeek-V3 widths (H = 7168, I = 2048, k = 8) over 16 experts, so the
64-token decode call uses about 19 MB of the 32 MiB array.
"""
import pytest
import torch

import oracle
import synth
from gpu_cases import (bf16_dev, bits_to_f32, generated_layer_gpu, log, oracle_expert_weights, oracle_tokens,
                       rel_err, require_gpu)

pytestmark = pytest.mark.gpu
TOL = 2e-2
W = synth.Workload("noalloc16", 7168, 2048, 16, 8, 64, "zipf", 1.0)


@pytest.fixture(scope="module")
def moe():
    return require_gpu()


@pytest.fixture(scope="module")
def layer(moe):
    log("noalloc: drawing a 16-expert layer at H=7168, I=2048 on the GPU")
    return generated_layer_gpu(moe, W)


def _inputs(T):
    w = W.with_tokens(T)
    x = synth.activations(w)
    ids, wts = synth.routing(w)
    return x, ids, wts


def _both(moe, T, regime, layer):
    x, ids, wts = _inputs(T)
    dx, dids, dw = bf16_dev(x), torch.from_numpy(ids).cuda(), torch.from_numpy(wts).cuda()
    d = moe.MoeDims(W.hidden, W.inter, W.n_experts, W.topk)
    ref = torch.empty((T, W.hidden), dtype=torch.int16, device="cuda")
    ws = torch.empty(max(256, moe.moe_ffn_layer_workspace(d, T, regime)), dtype=torch.uint8, device="cuda")
    st_ref = torch.zeros(1, dtype=torch.int32, device="cuda")
    moe.moe_ffn_layer(d, T, regime, dx, dids, dw, *layer, ref, st_ref, ws)
    got = torch.empty((T, W.hidden), dtype=torch.int16, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    moe.moe_ffn_layer_noalloc(d, T, regime, dx, dids, dw, *layer, got, st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0 and int(st_ref.item()) == 0
    return x, ids, wts, ref, got


@pytest.mark.parametrize("regime_name,t_first,t_second", [("decode", 64, 3), ("prefill", 128, 65)])
def test_noalloc_equals_layer_on_two_calls(moe, layer, regime_name, t_first, t_second):
    regime = moe.MOE_REGIME_DECODE if regime_name == "decode" else moe.MOE_REGIME_PREFILL
    for T in (t_first, t_second):
        log(f"noalloc {regime_name}: T={T}")
        x, ids, wts, ref, got = _both(moe, T, regime, layer)
        assert torch.equal(got, ref), f"{regime_name} T={T}: noalloc output differs from moe_ffn_layer"
        toks = [0, T // 2, T - 1]
        ow = oracle_expert_weights(W, sorted(set(ids[toks].reshape(-1).tolist())))
        ref_o = oracle_tokens(x, ids, wts, toks, ow)
        err = rel_err(bits_to_f32(got)[toks], oracle.bf16_to_f32(ref_o))
        log(f"noalloc {regime_name}: T={T} vs oracle on tokens {toks}: {err:.3e}")
        assert err <= TOL


def test_noalloc_rejects_a_call_beyond_its_scratch(moe, layer):
    T = 512   # prefill workspace of 512 tokens x 8 slots is about 120 MB
    d = moe.MoeDims(W.hidden, W.inter, W.n_experts, W.topk)
    assert moe.moe_ffn_layer_workspace(d, T, moe.MOE_REGIME_PREFILL) > moe.MOE_NOALLOC_SCRATCH_BYTES
    x, ids, wts = _inputs(T)
    out = torch.empty((T, W.hidden), dtype=torch.int16, device="cuda")
    with pytest.raises(moe.MoEError) as ei:
        moe.moe_ffn_layer_noalloc(d, T, moe.MOE_REGIME_PREFILL, bf16_dev(x), torch.from_numpy(ids).cuda(),
                                  torch.from_numpy(wts).cuda(), *layer, out)
    assert ei.value.status == moe.MOE_ERR_WORKSPACE and "scratch" in str(ei.value)


@pytest.mark.parametrize("regime_name,T", [("decode", 4), ("prefill", 100)])
def test_noalloc_call_replays_from_a_hip_graph(moe, layer, regime_name, T):
    """The callers this entry point is for: one call captured in a HIP graph
    (nothing allocated inside it), replayed three times.  Before each replay
    the static input gets new activations, and eager work runs on the same
    GPU (moe_ffn_layer with its own workspace on the new input, for the
    reference, and a noalloc call of another size, which rewrites the
    scratch array); every replay must equal the reference bit for bit."""
    import numpy as np

    regime = moe.MOE_REGIME_DECODE if regime_name == "decode" else moe.MOE_REGIME_PREFILL
    d = moe.MoeDims(W.hidden, W.inter, W.n_experts, W.topk)
    x0, ids, wts = _inputs(T)
    dx, dids, dw = bf16_dev(x0), torch.from_numpy(ids).cuda(), torch.from_numpy(wts).cuda()
    out = torch.empty((T, W.hidden), dtype=torch.int16, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    moe.moe_ffn_layer_noalloc(d, T, regime, dx, dids, dw, *layer, out, st)  # first call on the device: set-up
    torch.cuda.synchronize()
    log(f"noalloc graph {regime_name}: capturing T={T}")
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(g, stream=side):
        moe.moe_ffn_layer_noalloc(d, T, regime, dx, dids, dw, *layer, out, st)
    torch.cuda.synchronize()

    xo, ido, wo = _inputs(3)
    other = torch.empty((3, W.hidden), dtype=torch.int16, device="cuda")
    ws = torch.empty(max(256, moe.moe_ffn_layer_workspace(d, T, regime)), dtype=torch.uint8, device="cuda")
    rng = np.random.default_rng(17)
    for rep in range(3):
        x = synth.bf16_bits_from_f32(rng.standard_normal((T, W.hidden)).astype(np.float32) * (1.0 + rep))
        dx.copy_(bf16_dev(x))
        ref = torch.empty_like(out)
        st_ref = torch.zeros(1, dtype=torch.int32, device="cuda")
        moe.moe_ffn_layer(d, T, regime, dx, dids, dw, *layer, ref, st_ref, ws)
        moe.moe_ffn_layer_noalloc(d, 3, moe.MOE_REGIME_DECODE, bf16_dev(xo), torch.from_numpy(ido).cuda(),
                                  torch.from_numpy(wo).cuda(), *layer, other)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        log(f"noalloc graph {regime_name}: replay {rep}")
        assert int(st.item()) == 0 and int(st_ref.item()) == 0
        assert torch.equal(out, ref), f"replay {rep} differs from the eager call on the same input"
