"""GPU parity of the router (moe_router) against the CPU router oracle.

The oracle takes each decision on fp32 keys computed from exactly summed
logits; the GPU sums the logits in fp32 on the MFMA.  Keys therefore agree
to about 1e-6, and a token whose k-th and (k+1)-th candidate keys (or whose
last kept and first dropped group scores) lie closer than EPS can flip: for
those tokens the GPU choice is checked to be a valid choice under the
oracle's keys within EPS; every other token must match bit for bit in ids,
and its weights within 1e-5.
"""
import numpy as np
import pytest
import torch

import synth
from gpu_cases import log, require_gpu, to_dev
from oracle import router_oracle as ro

pytestmark = pytest.mark.gpu
EPS = 2e-5


@pytest.fixture(scope="module")
def moe():
    return require_gpu()


def _gpu_router(moe, x, wr, bias, k, n_group, topk_group, scaling):
    t = x.shape[0]
    ids = torch.full((t, k), -1, dtype=torch.int32, device="cuda")
    wts = torch.zeros((t, k), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(1, moe.moe_router_workspace(t, x.shape[1], wr.shape[0])), dtype=torch.uint8, device="cuda")
    db = None if bias is None else to_dev(bias)
    moe.moe_router(to_dev(x.view(np.int16)), to_dev(wr.view(np.int16)), db, ids, wts, n_group, topk_group, scaling,
                   ws)
    torch.cuda.synchronize()
    return ids.cpu().numpy(), wts.cpu().numpy()


def _margins(sel, n_group, topk_group, k):
    """Per token: the smallest of the gap between the last kept and first
    dropped group score and the gaps between consecutive keys of the k + 1
    best experts of the kept groups (the ids are listed by key, so a near
    tie inside the top k reorders them)."""
    t, e = sel.shape
    if n_group > 1:
        gs = np.sort(ro.group_scores(sel, n_group), axis=1)[:, ::-1]
        ggap = gs[:, topk_group - 1] - gs[:, topk_group] if topk_group < n_group else np.full(t, np.inf)
    else:
        ggap = np.full(t, np.inf)
    m = min(k + 1, topk_group * (e // n_group))
    ids, _ = ro.select_experts(sel, None, m, n_group, topk_group)
    if m < 2:
        kgap = np.full(t, np.inf)
    else:
        ks = np.take_along_axis(sel, ids, axis=1)
        kgap = np.min(ks[:, :-1] - ks[:, 1:], axis=1)
    return np.minimum(ggap, kgap)


def _check(name, x, wr, bias, k, n_group, topk_group, scaling, moe):
    ids, wts = _gpu_router(moe, x, wr, bias, k, n_group, topk_group, scaling)
    r_ids, r_w, inter = ro.router(x, wr, bias, k, n_group, topk_group, scaling, want_intermediates=True)
    sel = inter["scores"] + (0 if bias is None else bias[None, :])
    close = _margins(sel.astype(np.float32), n_group, topk_group, k) < EPS
    same = np.all(ids == r_ids, axis=1)
    log(f"router {name}: T={x.shape[0]} tokens differing {int((~same).sum())}, near ties {int(close.sum())}")
    assert np.all(same | close), "ids differ on a token without a near tie"
    assert close.mean() <= 0.15  # most tokens are compared bit for bit
    assert np.allclose(wts[same], r_w[same], rtol=0, atol=1e-5 * scaling)
    e_all = sel.shape[1]
    gsize = e_all // n_group
    gscore = ro.group_scores(sel, n_group) if n_group > 1 else None
    scores = inter["scores"]
    for t in np.nonzero(~same)[0]:  # near ties: a valid choice under the oracle keys within EPS
        row = ids[t].tolist()
        got = set(row)
        assert len(got) == k and all(0 <= e < e_all for e in row)
        # groups: at most topk_group of them, each scoring within EPS of the
        # topk_group-th best group; completed with the best other groups
        used = sorted(set(e // gsize for e in row))
        assert len(used) <= topk_group
        if gscore is not None:
            thr = np.sort(gscore[t])[::-1][topk_group - 1]
            assert all(gscore[t, g] >= thr - EPS for g in used), (t, used)
            rest = [g for g in np.argsort(-gscore[t], kind="stable").tolist() if g not in used]
            kept = set(used) | set(rest[:topk_group - len(used)])
        else:
            kept = {0}
        # experts: no expert of a kept group left out beats a chosen one by more than EPS
        chosen_min = min(sel[t, row])
        others = [sel[t, e] for e in range(e_all) if e not in got and e // gsize in kept]
        assert not others or max(others) <= chosen_min + EPS
        # listed by decreasing key (within EPS)
        keys = sel[t, row]
        assert np.all(keys[:-1] >= keys[1:] - EPS)
        # weights of the chosen ids: oracle scores normalised in slot order
        sv = scores[t, row].astype(np.float32)
        tot = np.float32(0.0)
        for v in sv:
            tot = np.float32(tot + v)
        w_ref = (sv / tot * np.float32(scaling)).astype(np.float32)
        assert np.allclose(wts[t], w_ref, rtol=0, atol=1e-5 * scaling), (t, wts[t], w_ref)


def test_router_tiny_plain_topk(moe):
    w = synth.WORKLOADS["tiny"]
    x = synth.activations(w)
    wr, _ = synth.router_params(w)
    _check("tiny", x, wr, None, w.topk, 1, 1, 1.0, moe)


@pytest.mark.parametrize("tokens", [1, 4, 17, 64, 257])
def test_router_deepseek_grouped(moe, tokens):
    w = synth.WORKLOADS["prefill8k"].with_tokens(tokens)
    x = synth.activations(w)
    wr, bias = synth.router_params(w, bias_std=0.05)
    _check(f"deepseek T={tokens}", x, wr, bias, 8, 8, 4, 2.5, moe)


def test_router_deepseek_8192_tokens(moe):
    w = synth.WORKLOADS["prefill8k"]
    x = synth.activations(w)
    wr, bias = synth.router_params(w, bias_std=0.05)
    _check("deepseek T=8192", x, wr, bias, 8, 8, 4, 1.0, moe)


def test_router_many_experts_wide_topk(moe):
    w = synth.Workload("router_wide", 1024, 256, 1024, 32, 40, "uniform")
    x = synth.activations(w)
    wr, bias = synth.router_params(w, bias_std=0.02)
    _check("E=1024 k=32", x, wr, bias, 32, 64, 16, 1.0, moe)


@pytest.mark.parametrize("tokens", [255, 256, 300])
def test_router_ragged_expert_tile_tiled_logits(moe, tokens):
    """E = 320 (one full and one ragged 256-expert tile), tokens around the
    switch to the LDS-tiled logits kernel and a ragged 128-token tail."""
    w = synth.Workload("router_ragged", 1024, 256, 320, 6, tokens, "uniform")
    x = synth.activations(w)
    wr, bias = synth.router_params(w, bias_std=0.02)
    _check(f"E=320 T={tokens}", x, wr, bias, 6, 1, 1, 1.0, moe)


@pytest.mark.parametrize("hidden", [1120, 1344, 1376])
def test_router_tiled_logits_step_counts(moe, hidden):
    """Hidden sizes whose K slices hold 5, 6 and 43 steps of 32: the tiled
    logits kernel's four-slot ring ends on a partial round of 1, 2 and 3 steps."""
    w = synth.Workload("router_steps", hidden, 256, 256, 8, 300, "uniform")
    x = synth.activations(w)
    wr, bias = synth.router_params(w, bias_std=0.05)
    _check(f"H={hidden} T=300", x, wr, bias, 8, 8, 4, 2.5, moe)


@pytest.mark.parametrize("hidden", [1024, 1056, 1088])
def test_router_256_token_tiles(moe, hidden):
    """32868 tokens (256-token logits tiles from 32768 on, the last one
    ragged), E = 320 (one full and one ragged 256-expert tile), one K slice
    of 32, 33 and 34 steps: the three-slot ring ends on a partial round of
    2, 0 and 1 steps."""
    w = synth.Workload("router_big", hidden, 256, 320, 6, 32868, "uniform")
    x = synth.activations(w)
    wr, bias = synth.router_params(w, bias_std=0.02)
    _check(f"E=320 T=32868 H={hidden}", x, wr, bias, 6, 1, 1, 1.0, moe)


def test_router_many_experts_many_tokens(moe):
    w = synth.Workload("router_wide_tiled", 1024, 256, 1024, 32, 260, "uniform")
    x = synth.activations(w)
    wr, bias = synth.router_params(w, bias_std=0.02)
    _check("E=1024 k=32 T=260", x, wr, bias, 32, 64, 16, 1.0, moe)


@pytest.mark.parametrize("experts,n_group,topk_group,k", [(256, 2, 1, 8), (384, 8, 3, 6)])
def test_router_groups_not_aligned_to_lanes(moe, experts, n_group, topk_group, k):
    """Groups of 128 and of 48 experts (not a power of two up to 64): the
    group scores take the general per-group reduction."""
    w = synth.Workload("router_groups", 1024, 256, experts, k, 70, "uniform")
    x = synth.activations(w)
    wr, bias = synth.router_params(w, bias_std=0.02)
    _check(f"E={experts} groups={n_group}", x, wr, bias, k, n_group, topk_group, 1.0, moe)


def test_router_zero_tokens_and_bad_config(moe):
    w = synth.WORKLOADS["tiny"]
    wr, _ = synth.router_params(w)
    ids = torch.empty((0, 2), dtype=torch.int32, device="cuda")
    wts = torch.empty((0, 2), dtype=torch.float32, device="cuda")
    x0 = torch.empty((0, w.hidden), dtype=torch.int16, device="cuda")
    moe.moe_router(x0, to_dev(wr.view(np.int16)), None, ids, wts, 1, 1, 1.0, None)
    x = to_dev(synth.activations(w).view(np.int16))
    ids = torch.empty((w.tokens, 2), dtype=torch.int32, device="cuda")
    wts = torch.empty((w.tokens, 2), dtype=torch.float32, device="cuda")
    with pytest.raises(moe.MoEError):
        moe.moe_router(x, to_dev(wr.view(np.int16)), None, ids, wts, 3, 1, 1.0, None)   # 3 does not divide 8
    with pytest.raises(moe.MoEError):
        moe.moe_router(x, to_dev(wr.view(np.int16)), None, ids, wts, 1, 1, 1.0, None)   # no workspace


@pytest.mark.parametrize("tokens,regime", [(48, "decode"), (300, "prefill")])
def test_router_shared_expert_full_layer(moe, tokens, regime):
    """Router with the shared expert appended as slot k (id E, weight 1.0)
    feeding the whole layer on E + 1 expert stacks, against the oracle gate
    and layer; tokens whose routing matches exactly are compared."""
    import oracle
    from gpu_cases import bits_to_f32, quantize_weights_gpu, rel_err
    E, k = 16, 4
    w = synth.Workload("router_shared", 512, 256, E, k, tokens, "uniform")
    w_stack = synth.Workload("router_shared_stack", 512, 256, E + 1, k, tokens, "uniform")
    x = synth.activations(w)
    wr, bias = synth.router_params(w, bias_std=0.05)
    ids_ref, w_ref = ro.router(x, wr, bias, k, 4, 2, 2.5, shared_expert=E)
    d_ids = torch.empty((tokens, k + 1), dtype=torch.int32, device="cuda")
    d_w = torch.empty((tokens, k + 1), dtype=torch.float32, device="cuda")
    ws = torch.empty(moe.moe_router_workspace(tokens, w.hidden, E), dtype=torch.uint8, device="cuda")
    moe.moe_router(to_dev(x.view(np.int16)), to_dev(wr.view(np.int16)), to_dev(bias), d_ids, d_w, 4, 2, 2.5, ws,
                   shared_expert=E)
    wg, wu, wd = synth.weights_host(w_stack)
    dev_weights = quantize_weights_gpu(moe, wg, wu, wd)
    reg = moe.MOE_REGIME_DECODE if regime == "decode" else moe.MOE_REGIME_PREFILL
    buf = moe.MoELayerBuffers(w.hidden, w.inter, E + 1, k + 1, tokens, reg)
    moe.run_layer(buf, to_dev(x.view(np.int16)), d_ids, d_w, dev_weights)
    torch.cuda.synchronize()
    assert int(buf.dev_status.item()) == 0
    got_ids = d_ids.cpu().numpy()
    assert np.all(got_ids[:, k] == E) and np.all(d_w.cpu().numpy()[:, k] == 1.0)
    same = np.all(got_ids == ids_ref, axis=1)
    log(f"router + shared expert, {regime}: tokens with identical routing {int(same.sum())}/{tokens}")
    assert same.mean() >= 0.9
    ref = oracle.bf16_to_f32(oracle.moe_layer(x, ids_ref, w_ref, oracle.prepare_weights(wg, wu, wd)))
    err = rel_err(bits_to_f32(buf.out)[same], ref[same])
    log(f"  out rel err vs oracle {err:.3e}")
    assert err <= 2e-2
