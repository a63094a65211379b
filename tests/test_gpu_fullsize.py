"""GPU parity at the full DeepSeek-V3 layer shape (H = 7168, I = 2048, E = 256,
k = 8) on whole experts and many tokens, against the CPU oracle.

* 8192-token prefill chunk (uniform routing): qx and sx of all 8192 tokens
  bit for bit; every row and all 7168 columns of y_rows for four complete
  experts (the smallest, the largest and two others), each expert within
  the bound on its own.
* 64-token batched decode (Zipf 1.0): the output of 16 tokens chosen to
  include twelve experts that have a single row, and y_rows of every expert
  those tokens touch (46 experts), each within the bound on its own.
* 32768-token prefill with Zipf(0.8) routing (the streamed workload, whose
  output equals the resident prefill path bit for bit, checked in
  test_gpu_streamed): y_rows of two complete mid-size experts and a 1024-row
  slice of the largest expert (18326 rows) that crosses many of its m-tiles,
  plus the bit-exact qx/sx of every token those rows read.

Cost on the host: the oracle re-draws each expert it needs on the GPU and
quantizes its three matrices (14.7M values each, a few seconds per matrix)
on a pool of CPU processes; about 60 expert quantizations and 10k oracle
activation rows over the module, a minute or two on 16 cores.
"""
import numpy as np
import pytest
import torch

import oracle
import oracle_pool
import synth
from gpu_cases import (bf16_dev, bits_to_f32, generated_layer_gpu, log, oracle_expert_weights_pooled,
                       oracle_tokens_grouped, rel_err, require_gpu, to_dev)

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.fixture(scope="module")
def moe():
    return require_gpu()


@pytest.fixture(scope="module")
def layer(moe):
    log("full-size parity: drawing the DeepSeek-V3 expert layer on the GPU")
    return generated_layer_gpu(moe, synth.WORKLOADS["decode1"], layer=0)


def _run(moe, w, x, ids, wts, layer, regime):
    buf = moe.MoELayerBuffers(w.hidden, w.inter, w.n_experts, w.topk, w.tokens, regime)
    moe.run_layer(buf, bf16_dev(x), to_dev(ids), to_dev(wts), layer)
    torch.cuda.synchronize()
    assert int(buf.dev_status.item()) == 0
    return buf


def _check_expert_rows(name, buf, qx, sx, ids, ow, experts, row_slices=None):
    """y_rows of the given experts (all rows, or a slice) against oracle.expert_rows."""
    k = ids.shape[1]
    off = buf.expert_offsets.cpu().numpy()
    src = buf.sorted_src.cpu().numpy()
    for e in experts:
        p0, p1 = int(off[e]), int(off[e + 1])
        if row_slices and e in row_slices:
            a, b = row_slices[e]
            p0, p1 = p0 + a, p0 + b
        tok = src[p0:p1] // k
        ref = oracle.expert_rows(qx[tok], sx[tok], *ow[e])
        got = buf.y_rows[p0:p1].cpu().numpy()
        err = rel_err(got, ref)
        big = float(np.max(np.abs(got.astype(np.float64) - ref)))
        log(f"  {name}: expert {e} rows {p0}..{p1 - 1} ({p1 - p0}): rel err {err:.3e} (max abs {big:.3e})")
        assert err <= TOL, (e, err)


# ----------------------------------------------------------- prefill 8192
@pytest.fixture(scope="module")
def prefill8k(moe, layer):
    w = synth.WORKLOADS["prefill8k"]
    x = synth.activations(w)
    ids, wts = synth.routing(w)
    log("prefill8k: the layer on 8192 tokens (four calls, prefill regime)")
    buf = _run(moe, w, x, ids, wts, layer, moe.MOE_REGIME_PREFILL)
    return w, x, ids, wts, buf


def test_prefill8k_quantized_activations_of_every_token(prefill8k):
    w, x, ids, wts, buf = prefill8k
    qx_ref, sx_ref = oracle_pool.quant_act_rows(x)
    assert np.array_equal(buf.sx.cpu().numpy().view(np.uint32), sx_ref.view(np.uint32))
    assert np.array_equal(buf.qx.cpu().numpy(), qx_ref)
    off, src, dst = oracle.permute(ids, w.n_experts)
    assert np.array_equal(buf.expert_offsets.cpu().numpy(), off)
    assert np.array_equal(buf.sorted_src.cpu().numpy(), src)
    assert np.array_equal(buf.dest_row.cpu().numpy(), dst)


def test_prefill8k_complete_experts(prefill8k):
    w, x, ids, wts, buf = prefill8k
    counts = np.bincount(ids.reshape(-1), minlength=w.n_experts)
    experts = sorted({int(np.argmin(counts)), int(np.argmax(counts)), 0, w.n_experts - 1})
    log(f"prefill8k: complete experts {experts} with {counts[experts].tolist()} rows")
    ow = oracle_expert_weights_pooled(w, experts)
    toks = sorted(set(np.concatenate([np.nonzero((ids == e).any(axis=1))[0] for e in experts]).tolist()))
    qx = np.zeros((w.tokens, w.hidden), np.uint8)
    sx = np.zeros((w.tokens, w.hidden // 128), np.float32)
    qx[toks], sx[toks] = oracle_pool.quant_act_rows(x[toks])
    _check_expert_rows("prefill8k", buf, qx, sx, ids, ow, experts)


# ------------------------------------------------ batched decode, 64 tokens
def _decode_sample(ids, n_tokens=16, n_single=4):
    """Tokens chosen greedily to touch few experts: first n_single tokens that
    hold an expert with a single row, then any, each adding the fewest new
    experts (ties to the lower token)."""
    counts = np.bincount(ids.reshape(-1), minlength=int(ids.max()) + 1)
    single = set(np.nonzero(counts == 1)[0].tolist())
    chosen, union = [], set()
    pools = [[t for t in range(ids.shape[0]) if single & set(ids[t].tolist())]] * n_single + \
            [list(range(ids.shape[0]))] * (n_tokens - n_single)
    for cand in pools:
        t = min((t for t in cand if t not in chosen), key=lambda t: (len(union | set(ids[t].tolist())), t))
        chosen.append(t)
        union |= set(ids[t].tolist())
    return sorted(chosen), sorted(union), sorted(e for e in union if counts[e] == 1)


@pytest.fixture(scope="module")
def decode64(moe, layer):
    w = synth.WORKLOADS["decode64_zipf"]
    x = synth.activations(w)
    ids, wts = synth.routing(w)
    buf = _run(moe, w, x, ids, wts, layer, moe.MOE_REGIME_DECODE)
    tokens, experts, single = _decode_sample(ids)
    log(f"decode64_zipf: tokens {tokens}: {len(experts)} experts, {len(single)} of them with a single row")
    assert len(tokens) == 16 and len(single) >= 4
    qx, sx = oracle.quant_act(x)
    assert np.array_equal(buf.qx.cpu().numpy(), qx) and np.array_equal(buf.sx.cpu().numpy(), sx)
    return w, x, ids, wts, buf, tokens, qx, sx


@pytest.mark.parametrize("half", [0, 1])
def test_decode64_zipf_sixteen_tokens_and_their_experts(decode64, half):
    """Half of the 16 sampled tokens per test (about 25 experts to quantize
    on the host each): their outputs, and every row of their experts."""
    w, x, ids, wts, buf, tokens, qx, sx = decode64
    toks = tokens[8 * half: 8 * half + 8]
    experts = sorted(set(ids[toks].reshape(-1).tolist()))
    single = [e for e in experts if int((ids == e).sum()) == 1]
    log(f"decode64_zipf: tokens {toks}: {len(experts)} experts, single-row experts {single}")
    ow = oracle_expert_weights_pooled(w, experts)
    _check_expert_rows("decode64_zipf", buf, qx, sx, ids, ow, experts)
    ref = oracle_tokens_grouped(x, ids, wts, toks, ow)
    err = rel_err(bits_to_f32(buf.out)[toks], oracle.bf16_to_f32(ref))
    log(f"decode64_zipf: output of tokens {toks}: rel err {err:.3e}")
    assert err <= TOL


# ------------------------------------- 32768-token prefill, Zipf(0.8) routing
def test_prefill32k_zipf_complete_and_sliced_experts(moe, layer):
    w = synth.WORKLOADS["prefill32k_streamed"]
    x = synth.activations(w)
    ids, wts = synth.routing(w)
    log("prefill32k: the resident prefill layer on 32768 tokens")
    buf = _run(moe, w, x, ids, wts, layer, moe.MOE_REGIME_PREFILL)
    counts = np.bincount(ids.reshape(-1), minlength=w.n_experts)
    order = np.argsort(counts, kind="stable")
    mids = [int(order[w.n_experts // 2]), int(order[w.n_experts // 2 + 1])]
    big = int(order[-1])
    assert counts[big] > 10000
    # rows 4700 .. 5723 of the largest expert: its rows are dealt to 128-row
    # m-tiles in 32-row groups (18326 rows: 141 tiles of 128 rows, then 3 of
    # 96), so the slice crosses 8 tile boundaries
    a = 4700
    slices = {big: (a, a + 1024)}
    log(f"prefill32k: experts {mids} complete ({counts[mids].tolist()} rows), expert {big} rows {a}..{a + 1023} "
        f"of {counts[big]}")
    experts = mids + [big]
    ow = oracle_expert_weights_pooled(w, experts)
    off = buf.expert_offsets.cpu().numpy()
    src = buf.sorted_src.cpu().numpy()
    rows = [src[off[e]:off[e + 1]] for e in mids] + [src[off[big] + a:off[big] + a + 1024]]
    toks = np.unique(np.concatenate(rows) // w.topk)
    qx = np.zeros((w.tokens, w.hidden), np.uint8)
    sx = np.zeros((w.tokens, w.hidden // 128), np.float32)
    qx[toks], sx[toks] = oracle_pool.quant_act_rows(x[toks])
    assert np.array_equal(buf.qx.cpu().numpy()[toks], qx[toks])
    assert np.array_equal(buf.sx.cpu().numpy()[toks].view(np.uint32), sx[toks].view(np.uint32))
    _check_expert_rows("prefill32k", buf, qx, sx, ids, ow, experts, slices)
