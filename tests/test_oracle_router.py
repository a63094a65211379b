"""CPU pins of the router (gate) oracle.

The paper gives no gate formula or example (Background, Mixture-of-Experts
names only plain and grouped top-k), so the selection is pinned to hand-worked cases
of the reading (tests/golden/router_select_cases.txt), to a brute-force
statement by pairwise comparisons on small inputs, and to plain top-k
(numpy's sort) when there is one group; the logits to torch's fp64 matmul
and the sigmoid to torch's.
"""
import os

import numpy as np
import pytest
import torch

from oracle import router_oracle as ro

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "router_select_cases.txt")


def _cases():
    out = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        name, cfg, scores, bias, ids, wts = [p.strip() for p in line.split(";")]
        e, g, tg, k, sc = cfg.split()
        out.append((name, int(e), int(g), int(tg), int(k), float(sc),
                    np.array(scores.split(), np.float32), np.array(bias.split(), np.float32),
                    np.array(ids.split(), np.int32), np.array(wts.split(), np.float64)))
    return out


@pytest.mark.parametrize("case", _cases(), ids=lambda c: c[0])
def test_selection_matches_hand_worked_cases(case):
    name, e, g, tg, k, sc, scores, bias, ids, wts = case
    got_ids, got_w = ro.select_experts(scores[None, :], bias, k, g, tg, sc)
    assert np.array_equal(got_ids[0], ids)
    assert np.allclose(got_w[0], wts, rtol=0, atol=2e-6)


def _brute_force(scores, bias, k, n_group, topk_group, scaling):
    """Pairwise-comparison statement of the selection (no sorting), one token."""
    e = len(scores)
    sel = [np.float32(scores[i] + bias[i]) for i in range(e)]
    per = e // n_group
    gsc = []
    for gi in range(n_group):
        vals = sel[gi * per:(gi + 1) * per]
        best = max(range(per), key=lambda i: (vals[i], -i))
        second = max([i for i in range(per) if i != best], key=lambda i: (vals[i], -i))
        gsc.append(np.float32(vals[best] + vals[second]))

    def beats(a, b, va, vb):
        return va > vb or (va == vb and a < b)

    kept = [sum(beats(h, gi, gsc[h], gsc[gi]) for h in range(n_group)) < topk_group for gi in range(n_group)]
    cand = [i for i in range(e) if kept[i // per]]
    rank = {i: sum(beats(j, i, sel[j], sel[i]) for j in cand) for i in cand}
    ids = sorted([i for i in cand if rank[i] < k], key=lambda i: rank[i])
    total = np.float32(0)
    for i in ids:
        total = np.float32(total + np.float32(scores[i]))
    w = [np.float32(np.float32(np.float32(scores[i]) / total) * np.float32(scaling)) for i in ids]
    return np.array(ids, np.int32), np.array(w, np.float32)


@pytest.mark.parametrize("e,n_group,topk_group,k", [(16, 4, 2, 4), (32, 8, 4, 8), (12, 3, 3, 5), (8, 1, 1, 3)])
def test_selection_equals_brute_force(e, n_group, topk_group, k):
    rng = np.random.default_rng(e * 100 + k)
    for trial in range(40):
        # coarse values so that equal keys and equal group scores occur
        scores = (rng.integers(0, 6, size=e) / 8.0).astype(np.float32)
        bias = (rng.integers(-2, 3, size=e) / 16.0).astype(np.float32) if trial % 2 else np.zeros(e, np.float32)
        ids, w = ro.select_experts(scores[None, :], bias, k, n_group, topk_group, 1.5)
        bid, bw = _brute_force(scores, bias, k, n_group, topk_group, 1.5)
        assert np.array_equal(ids[0], bid), (scores, bias)
        assert np.array_equal(w[0], bw)


def test_one_group_is_plain_top_k():
    rng = np.random.default_rng(3)
    s = rng.random((50, 64)).astype(np.float32)
    ids, w = ro.select_experts(s, None, 6, 1, 1)
    ref = np.argsort(-s, axis=1, kind="stable")[:, :6]
    assert np.array_equal(ids, ref)
    assert np.allclose(w.sum(axis=1), 1.0, atol=1e-6)


def test_invariants_grouped_deepseek_shape():
    rng = np.random.default_rng(4)
    s = ro.sigmoid_f32(rng.standard_normal((200, 256)).astype(np.float32) * 2)
    bias = (rng.standard_normal(256) * 0.1).astype(np.float32)
    ids, w = ro.select_experts(s, bias, 8, 8, 4, 2.5)
    assert ids.shape == (200, 8)
    for t in range(200):
        assert len(set(ids[t].tolist())) == 8
        assert len(set((ids[t] // 32).tolist())) <= 4          # at most topk_group groups
        sel = s[t] + bias
        assert np.all(np.diff(sel[ids[t]]) <= 0)               # listed by decreasing key
    assert np.allclose(w.sum(axis=1), 2.5, atol=1e-5)
    # weights come from the unbiased scores
    chosen = np.take_along_axis(s, ids, axis=1)
    assert np.allclose(w, chosen / chosen.sum(axis=1, keepdims=True) * 2.5, rtol=1e-6)


def test_logits_match_torch_fp64_matmul():
    rng = np.random.default_rng(5)
    x = torch.from_numpy(rng.standard_normal((9, 640)).astype(np.float32)).to(torch.bfloat16)
    wr = torch.from_numpy((0.02 * rng.standard_normal((48, 640))).astype(np.float32)).to(torch.bfloat16)
    got = ro.router_logits(x.view(torch.int16).numpy().view(np.uint16), wr.view(torch.int16).numpy().view(np.uint16))
    ref = (x.double() @ wr.double().T).float().numpy()
    ulps = np.abs(got.view(np.int32).astype(np.int64) - ref.view(np.int32).astype(np.int64))
    assert ulps.max() <= 1


def test_sigmoid_matches_torch():
    x = np.concatenate([np.linspace(-30, 30, 4001, dtype=np.float32), np.array([0.0, -0.0], np.float32)])
    got = ro.sigmoid_f32(x)
    ref = torch.sigmoid(torch.from_numpy(x)).numpy()
    assert got[-2] == 0.5 and got[-1] == 0.5
    assert np.allclose(got, ref, rtol=3e-7, atol=1e-30)


def test_bad_configs_raise():
    s = np.ones((1, 8), np.float32)
    for args in ((3, 3, 1), (3, 4, 5), (9, 4, 2), (2, 8, 1)):
        k, g, tg = args
        with pytest.raises(ValueError):
            ro.select_experts(s, None, k, g, tg)


def test_shared_expert_slot_is_routed_sum_plus_shared():
    """The shared slot (id E, weight 1.0, last) gives bf16(routed fp32 sum + shared rows)."""
    import oracle
    import synth
    w = synth.WORKLOADS["tiny"]
    x = synth.activations(w)
    ids, wts = synth.routing(w)
    wg, wu, wd = synth.weights_host(w)
    rng = np.random.default_rng(11)
    shared = [(0.02 * rng.standard_normal(m.shape[1:])).astype(np.float32)[None] for m in (wg, wu, wd)]
    routed = oracle.prepare_weights(wg, wu, wd)
    both = oracle.prepare_weights(*[np.concatenate([m, s], axis=0) for m, s in zip((wg, wu, wd), shared)])
    ids_s, w_s = ro.append_shared(ids, wts, w.n_experts)
    out = oracle.moe_layer(x, ids_s, w_s, both)
    _, inter = oracle.moe_layer(x, ids, wts, routed, want_intermediates=True)
    t, k = ids.shape
    dest = inter["dest_row"].reshape(t, k)
    acc = np.zeros((t, w.hidden), np.float32)
    for j in range(k):
        acc = (acc + (wts[:, j][:, None] * inter["y"][dest[:, j]]).astype(np.float32)).astype(np.float32)
    sq = oracle.prepare_weights(*shared)
    y_sh = oracle.expert_rows(inter["qx"], inter["sx"], sq[0][0], sq[1][0], sq[2][0], sq[3][0], sq[4][0], sq[5][0])
    assert np.array_equal(out, oracle.f32_to_bf16((acc + y_sh).astype(np.float32)))
