"""Seeded synthetic inputs for the routed-expert FP8 MoE FFN.

This module is shared by the CPU oracle (``oracle/``) and the GPU path
(``paper_2606_10493_amd``).  It only draws numbers: it holds none of the
layer's arithmetic (no FP8 encoding, no block scaling, no GEMM, no SiLU, no
combine).  Expert weights are produced in fp32 and each side quantizes them
to e4m3 with its own code.

The workloads follow the paper's target model (a DeepSeek-V3 routed-expert
layer: hidden 7168, expert intermediate 2048, 256 experts, top-8; System
Design, "Hardware and model target", and the 128-element FP8 scale blocks of
the AVX-512 FP8 GEMV Kernel section).  Real weights, prompts and routing
traces are not available; the recipes below stand in for them:

* activations ~ N(0, 1) drawn in fp32 and rounded to bf16 (round to nearest
  even, done by torch's dtype conversion);
* weights ~ N(0, 0.02) in fp32, layout ``[out, in]`` row-major;
* routing: k distinct expert ids per token, drawn without replacement from
  a uniform or Zipf(s) popularity law (Gumbel-top-k on log p, which is
  successive sampling without replacement), the Zipf rank -> id map being a
  seeded permutation; ids are kept in draw order;
* routing weights: softmax of k N(0,1) logits (tiny config) or sigmoid of
  N(0,1) logits normalised by their sum over the k slots (DeepSeek-V3 shapes).

Every tensor takes its own sub-seed from ``numpy.random.SeedSequence(seed)``
in the fixed order x, routing, w_gate, w_up, w_down.  Full-size expert
weights (11.27 G values per layer) are drawn on the GPU with torch's
device generator, one generator per (layer, expert, matrix), so any single
expert can be re-drawn on its own for the CPU oracle.
"""
from __future__ import annotations

import dataclasses
import hashlib

import numpy as np

BLOCK = 128


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    hidden: int
    inter: int
    n_experts: int
    topk: int
    tokens: int
    routing: str            # "uniform" | "zipf"
    zipf_s: float = 0.0
    weight_rule: str = "sigmoid"  # "softmax" | "sigmoid"
    chunk_tokens: int = 0   # >0: processed in chunks with streamed weights
    seed: int = 0
    layers: int = 1         # >1: a stack of layers streamed through one ring
    ring_slots: int = 0     # streamed: ring size in experts (0: all experts of a layer)
    weight_sets: int = 0    # stacks: distinct weight layers, layer l using set l mod weight_sets (0: one per layer)

    def with_tokens(self, t: int) -> "Workload":
        return dataclasses.replace(self, tokens=t)


# The five workloads: a tiny layer, DeepSeek-V3-shaped decode at 1 and 4
# tokens, batched decode at 64 tokens with skewed routing, an 8192-token
# prefill chunk and a 32768-token prefill streamed in 4096-token chunks.
WORKLOADS = {
    "tiny": Workload("tiny", 256, 128, 8, 2, 16, "uniform", weight_rule="softmax"),
    "decode1": Workload("decode1", 7168, 2048, 256, 8, 1, "uniform"),
    "decode4": Workload("decode4", 7168, 2048, 256, 8, 4, "uniform"),
    "decode64_zipf": Workload("decode64_zipf", 7168, 2048, 256, 8, 64, "zipf", 1.0),
    "prefill8k": Workload("prefill8k", 7168, 2048, 256, 8, 8192, "uniform"),
    "prefill32k_streamed": Workload("prefill32k_streamed", 7168, 2048, 256, 8, 32768,
                                    "zipf", 0.8, chunk_tokens=4096),
    # Four DeepSeek-V3-shaped layers, each with its own weights and routing,
    # streamed one after the other through a ring of 32 expert slots.
    "slp4_ring32": Workload("slp4_ring32", 7168, 2048, 256, 8, 4096, "zipf", 0.8, chunk_tokens=4096,
                            layers=4, ring_slots=32),
    # The same stack through a ping-pong ring of two expert slots.
    "slp4_ring2": Workload("slp4_ring2", 7168, 2048, 256, 8, 4096, "zipf", 0.8, chunk_tokens=4096,
                           layers=4, ring_slots=2),
    # The 58 routed-expert layers of a DeepSeek-V3-class model streamed
    # through one ring of 32 expert slots, each layer with its own routing;
    # the weights cycle over 4 drawn layers (58 distinct layers would need
    # 654 GB of pinned host memory), so every call still copies its whole
    # 11.28 GB over the host link.
    "slp58_ring32": Workload("slp58_ring32", 7168, 2048, 256, 8, 4096, "zipf", 0.8, chunk_tokens=4096,
                             layers=58, ring_slots=32, weight_sets=4),
}


def _seeds(seed: int, layer: int = 0):
    ss = np.random.SeedSequence(seed) if layer == 0 else np.random.SeedSequence([seed, layer])
    kids = ss.spawn(6)
    return dict(zip(("x", "routing", "w_gate", "w_up", "w_down", "router"), kids))


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 (torch's round-to-nearest-even conversion), as uint16 bits."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def activations(w: Workload, tokens: int | None = None) -> np.ndarray:
    """x ~ N(0,1) as bf16 bit patterns, shape [T, H] (uint16)."""
    t = w.tokens if tokens is None else tokens
    rng = np.random.default_rng(_seeds(w.seed)["x"])
    x = rng.standard_normal((t, w.hidden), dtype=np.float32)
    return bf16_bits_from_f32(x)


def routing(w: Workload, tokens: int | None = None, layer: int = 0):
    """(topk_ids int32 [T,k], topk_w fp32 [T,k]) per the workload's law."""
    t = w.tokens if tokens is None else tokens
    e, k = w.n_experts, w.topk
    rng = np.random.default_rng(_seeds(w.seed, layer)["routing"])
    if w.routing == "uniform":
        logp = np.zeros(e)
        rank_to_id = np.arange(e)
    elif w.routing == "zipf":
        logp = -w.zipf_s * np.log(np.arange(1, e + 1, dtype=np.float64))
        rank_to_id = rng.permutation(e)
    else:
        raise ValueError(w.routing)
    ids = np.empty((t, k), dtype=np.int32)
    step = 8192
    for t0 in range(0, t, step):
        t1 = min(t, t0 + step)
        g = rng.gumbel(size=(t1 - t0, e))
        keys = logp[None, :] + g
        top = np.argsort(-keys, axis=1, kind="stable")[:, :k]
        ids[t0:t1] = rank_to_id[top]
    logits = rng.standard_normal((t, k)).astype(np.float32)
    if w.weight_rule == "softmax":
        z = np.exp(logits - logits.max(axis=1, keepdims=True))
        wts = z / z.sum(axis=1, keepdims=True)
    else:
        sg = 1.0 / (1.0 + np.exp(-logits.astype(np.float64)))
        wts = sg / sg.sum(axis=1, keepdims=True)
    return ids, wts.astype(np.float32)


def weights_host(w: Workload, experts=None):
    """fp32 weights on the host: (w_gate [E,I,H], w_up [E,I,H], w_down [E,H,I]).

    Meant for small layers; full DeepSeek-V3 layers use ``expert_weight_device``.
    """
    s = _seeds(w.seed)
    e = w.n_experts
    out = []
    for name, shape in (("w_gate", (e, w.inter, w.hidden)),
                        ("w_up", (e, w.inter, w.hidden)),
                        ("w_down", (e, w.hidden, w.inter))):
        rng = np.random.default_rng(s[name])
        out.append((0.02 * rng.standard_normal(shape, dtype=np.float32)).astype(np.float32))
    if experts is not None:
        out = [m[list(experts)] for m in out]
    return tuple(out)


def _device_seed(seed: int, layer: int, expert: int, which: int) -> int:
    h = hashlib.sha256(f"{seed}/{layer}/{expert}/{which}".encode()).digest()
    return int.from_bytes(h[:8], "little") & ((1 << 63) - 1)


def expert_weight_device(w: Workload, layer: int, expert: int, which: int, device="cuda"):
    """One expert matrix in fp32 drawn with torch's generator on ``device``.

    which: 0 = gate [I,H], 1 = up [I,H], 2 = down [H,I].  The draw depends
    only on (seed, layer, expert, which), so the CPU oracle can re-draw any
    single expert and copy it to the host.
    """
    import torch
    shape = (w.inter, w.hidden) if which < 2 else (w.hidden, w.inter)
    g = torch.Generator(device=device)
    g.manual_seed(_device_seed(w.seed, layer, expert, which))
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32).mul_(0.02)


def router_params(w: Workload, layer: int = 0, bias_std: float = 0.0):
    """Router (gate) weight W_r ~ N(0, 0.02) as bf16 bits [E, H] and a per-expert
    fp32 selection bias ~ N(0, bias_std) (zeros when bias_std is 0)."""
    rng = np.random.default_rng(_seeds(w.seed, layer)["router"])
    wr = bf16_bits_from_f32((0.02 * rng.standard_normal((w.n_experts, w.hidden))).astype(np.float32))
    bias = (bias_std * rng.standard_normal(w.n_experts)).astype(np.float32)
    return wr, bias
