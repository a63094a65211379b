"""CPU oracle of the MoE router (gate).  TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import or run this module; the GPU library never does.

The paper (Background, Mixture-of-Experts) says only that a learned gate
picks a few experts per token by plain or grouped top-k selection, and that
SmallEP evaluates the gate and sorts tokens locally.  It gives no formula,
tie-break or group rule, so this oracle follows one reading, the DeepSeek-V3
gate of the paper's target models:

* logits[t, e] = sum_i x[t, i] * W_r[e, i], x and W_r bf16, the sum taken
  exactly (fp64 holds every bf16 x bf16 product exactly) and rounded once to
  fp32;
* scores s = 1 / (1 + exp(-logits)) in fp32;
* selection keys  sel = s + bias  (fp32; bias is a per-expert correction,
  zero if absent);
* the E experts form n_group contiguous groups of E / n_group; a group's
  score is the sum of its two largest keys; the topk_group groups with the
  largest scores are kept (equal scores: the lower group index first);
* among the kept groups' experts, the k largest keys are chosen (equal keys:
  the lower expert index first), listed in that order;
* weights w_j = s[id_j] / (s[id_0] + ... + s[id_{k-1}]) * scaling, the sum
  in slot order in fp32.

n_group = topk_group = 1 is plain top-k.

Shared expert (Background: DeepSeek's always-active shared experts): with
shared_expert >= 0 the gate appends that id with weight 1.0 as slot k, so
the rest of the layer adds the shared expert's output after the routed
ones, out = bf16(sum_j w_j y_j + y_shared).
"""
from __future__ import annotations

import numpy as np

f32 = np.float32


def _bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def router_logits(x_bf16: np.ndarray, w_bf16: np.ndarray) -> np.ndarray:
    """fp32 logits [T, E]: the exact dot products rounded once to fp32."""
    return (_bf16_to_f64(x_bf16) @ _bf16_to_f64(w_bf16).T).astype(f32)


def sigmoid_f32(logits: np.ndarray) -> np.ndarray:
    """1 / (1 + exp(-l)), every operation in fp32."""
    l = np.asarray(logits, dtype=f32)
    with np.errstate(over="ignore"):
        return (f32(1.0) / (f32(1.0) + np.exp(-l))).astype(f32)


def group_scores(sel: np.ndarray, n_group: int) -> np.ndarray:
    """[T, n_group]: the sum of the two largest keys of each group (fp32)."""
    t, e = sel.shape
    g = sel.reshape(t, n_group, e // n_group)
    top2 = -np.sort(-g, axis=2)[:, :, :2]
    return (top2[:, :, 0] + top2[:, :, 1]).astype(f32)


def select_experts(scores: np.ndarray, bias, k: int, n_group: int, topk_group: int, scaling: float = 1.0):
    """Grouped top-k on fp32 scores [T, E] -> (ids int32 [T, k], weights fp32 [T, k])."""
    s = np.asarray(scores, dtype=f32)
    t, e = s.shape
    check_router_config(e, k, n_group, topk_group)
    b = np.zeros(e, f32) if bias is None else np.asarray(bias, dtype=f32)
    sel = (s + b[None, :]).astype(f32)
    gs = group_scores(sel, n_group)
    # kept groups: order by (-score, group index), first topk_group
    gorder = np.lexsort((np.broadcast_to(np.arange(n_group), gs.shape), -gs), axis=1)[:, :topk_group]
    kept = np.zeros((t, n_group), bool)
    np.put_along_axis(kept, gorder, True, axis=1)
    expert_kept = np.repeat(kept, e // n_group, axis=1)
    keys = np.where(expert_kept, sel, -np.inf)
    order = np.lexsort((np.broadcast_to(np.arange(e), keys.shape), -keys), axis=1)[:, :k]
    ids = order.astype(np.int32)
    chosen = np.take_along_axis(s, order, axis=1)
    total = np.zeros(t, f32)
    for j in range(k):
        total = (total + chosen[:, j]).astype(f32)
    w = (chosen / total[:, None]).astype(f32)
    w = (w * f32(scaling)).astype(f32)
    return ids, w


def check_router_config(e: int, k: int, n_group: int, topk_group: int):
    if n_group < 1 or e % n_group:
        raise ValueError("n_group must divide the expert count")
    if e // n_group < 2 and n_group > 1:
        raise ValueError("a group needs at least two experts (its score is a top-2 sum)")
    if not 1 <= topk_group <= n_group:
        raise ValueError("topk_group must be in [1, n_group]")
    if not 1 <= k <= topk_group * (e // n_group):
        raise ValueError("k must be at most the number of experts in the kept groups")


def append_shared(ids: np.ndarray, w: np.ndarray, shared_expert: int):
    """Slot k := (shared_expert, 1.0)."""
    t = ids.shape[0]
    return (np.concatenate([ids, np.full((t, 1), shared_expert, np.int32)], axis=1),
            np.concatenate([w, np.ones((t, 1), f32)], axis=1))


def router(x_bf16, w_bf16, bias, k: int, n_group: int = 1, topk_group: int = 1, scaling: float = 1.0,
           want_intermediates: bool = False, shared_expert: int = -1):
    """Full gate: bf16 tokens [T, H] and bf16 router weights [E, H] -> ids, weights."""
    logits = router_logits(x_bf16, w_bf16)
    scores = sigmoid_f32(logits)
    ids, w = select_experts(scores, bias, k, n_group, topk_group, scaling)
    if shared_expert >= 0:
        ids, w = append_shared(ids, w, shared_expert)
    if want_intermediates:
        return ids, w, {"logits": logits, "scores": scores}
    return ids, w
