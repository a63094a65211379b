#!/usr/bin/env python3
"""Benchmark of the routed-expert FP8 MoE layer (DeepSeek-V3 shape) on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload prefill32k_streamed] [--also LIST]

A step is one pass of the whole path over one batch already resident in
HBM: quantize -> permute -> expert FFN -> combine.  The default workload is
the largest single-GPU configuration: a 32768-token prefill of one
DeepSeek-V3-shaped routed-expert layer (hidden 7168, expert intermediate
2048, 256 experts, top-8, Zipf(0.8) routing, FP8 e4m3 weights with 128x128
fp32 block scales, synthetic data) in 4096-token chunks, with the layer's
11.27 GB of expert weights in pinned host memory streamed into a device
ring on a copy stream while the expert kernels run (moe_ffn_streamed).
The resident workloads (8192-token prefill chunk, batched decode at 64
tokens, decode at 4 and 1 tokens, ...) are timed in the same run as one
moe_ffn_layer call per step (--unfused: the four calls moe_quant_act,
moe_permute, moe_expert_ffn, moe_combine) and reported under "also", each
with the roofline of its own dominant kernel.  Decode steps rotate over
several independently drawn weight layers so that repeated steps cannot be
served from the 256 MB Infinity Cache.

Prints one JSON line: whole-job tokens/s, the roofline of the dominant
kernel (timed live with HIP events on the stream it runs on) and the CPU
oracle's throughput on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
FP8_PEAK_TFLOPS = 5000.0     # MI355X dense FP8 MFMA
BF16_PEAK_TFLOPS = 2500.0    # MI355X dense bf16 MFMA (the router's logits GEMM)
METRIC = "FP8 MoE expert-FFN tokens/s; decode HBM GB/s; prefill FP8 MFMA TFLOPS"
DEFAULT_WORKLOAD = "prefill32k_streamed"
DEFAULT_ALSO = "prefill8k,decode64_zipf,decode4,decode1,decode1_w8a16,router"

# HBM bytes moved by a kernel, from rocprofv3 FETCH_SIZE and WRITE_SIZE runs
# scaled by a plain 1 GiB copy (FETCH x2.000, WRITE x1.000), recorded in the
# profiles/ summaries of each workload.  Valid only while the kernel's source
# file and the shared device header are the ones measured (sha256 prefix of
# the two files' bytes, source first).  Decode entries are per step (all
# launches of the kernel in a step), prefill entries per launch (the mean
# over the launches of a step), as the rooflines that carry them.
_DEC, _PRE = "paper_2606_10493_amd/csrc/ffn_decode.hip", "paper_2606_10493_amd/csrc/ffn_prefill.hip"
_COMMON = "paper_2606_10493_amd/csrc/common.h"
_DH, _PH = "cb7c22470036695c", "8d7be0b2719ce263"
TRAFFIC = {
    ("decode1", "ffn_decode_gateup"): {"bytes": 235721523, "source": _DEC, "sha256_prefix": _DH},
    ("decode64_zipf", "ffn_decode_gateup"): {"bytes": 4603754906, "source": _DEC, "sha256_prefix": _DH},
    ("decode4", "ffn_decode_gateup"): {"bytes": 942054400, "source": _DEC, "sha256_prefix": _DH},
    ("decode1_w8a16", "ffn_decode_w8a16_gateup"): {"bytes": 235617690, "source": _DEC, "sha256_prefix": _DH},
    ("prefill8k", "ffn_prefill_gateup"): {"bytes": 9711002009, "source": _PRE, "sha256_prefix": _PH},
    ("prefill8k", "ffn_prefill_down"): {"bytes": 6169021849, "source": _PRE, "sha256_prefix": _PH},
    ("prefill32k_streamed", "ffn_prefill_gateup"): {"bytes": 1360592077, "source": _PRE, "sha256_prefix": _PH},
    ("prefill32k_streamed", "ffn_prefill_down"): {"bytes": 1098833100, "source": _PRE, "sha256_prefix": _PH},
}


def source_hash(source):
    import hashlib
    h = hashlib.sha256()
    for f in (source, _COMMON):
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload, kernel):
    t = TRAFFIC.get((workload, kernel))
    if not t or source_hash(t["source"]) != t["sha256_prefix"]:
        return None
    return t["bytes"]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=0, help="timed steps (0: 10 for streamed, 50 for resident)")
    ap.add_argument("--warmup", type=int, default=0, help="warm-up steps (0: 2 for streamed, 10 for resident)")
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--layers", type=int, default=0, help="decode: weight layers to rotate over (0: 4)")
    ap.add_argument("--also", default=DEFAULT_ALSO,
                    help="comma list of extra resident workloads (each with its own roofline); NAME_w8a16 runs "
                         "the W8A16 decode FFN, router times the gate on the main workload's tokens")
    ap.add_argument("--unfused", action="store_true",
                    help="run resident layers as four library calls (quantize, permute, expert FFN, combine) "
                         "instead of one moe_ffn_layer call")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (calibrates HBM byte counters)")
    return ap.parse_args()


def log(msg):
    print(msg, file=sys.stderr, flush=True)


class LayerCache:
    """Device weight layers (packed e4m3 + scales) by layer index.  Weights depend
    only on (seed, layer, expert, matrix), so every DeepSeek-V3-shaped workload
    shares them."""

    def __init__(self, moe, torch, synth):
        self.moe, self.torch, self.synth = moe, torch, synth
        self.layers = {}

    def get(self, w, layer):
        key = (w.hidden, w.inter, w.n_experts, w.seed, layer)
        if key not in self.layers:
            log(f"drawing and quantizing weight layer {layer} on the GPU")
            self.layers[key] = make_layer(self.moe, self.torch, self.synth, w, layer)
        return self.layers[key]


def make_layer(moe, torch, synth, w, layer):
    e, i, h = w.n_experts, w.inter, w.hidden
    mats = []
    tmp = torch.empty((i * h,), dtype=torch.uint8, device="cuda")
    for which, (n, k) in enumerate(((i, h), (i, h), (h, i))):
        q = torch.empty((e, n, k), dtype=torch.uint8, device="cuda")
        s = torch.empty((e, n // 128, k // 128), dtype=torch.float32, device="cuda")
        rowmajor = tmp.view(n, k)
        for x in range(e):
            moe.moe_quant_weight(synth.expert_weight_device(w, layer, x, which), rowmajor, s[x])
            moe.moe_pack_weight(rowmajor, q[x])
        mats += [q, s]
    torch.cuda.synchronize()
    return tuple(mats)


def algorithmic(w, ids):
    """Per-call algorithmic work of the layer and of its kernels (see the design notes)."""
    import numpy as np
    t, k, h, i = w.tokens, w.topk, w.hidden, w.inter
    r = t * k
    n_act = int(np.unique(ids).size)
    sc_gu = 2 * (i // 128) * (h // 128) * 4
    sc_d = (h // 128) * (i // 128) * 4
    # One token (k <= 16, I <= 2048, H <= 8192): the gate/up kernel reads the bf16 row once instead of k qx/sx rows.
    one_token = t == 1 and k <= 16 and i <= 2048 and h <= 8192
    return {
        "active_experts": n_act,
        "rows": r,
        # decode gate/up kernel: touched W_gate + W_up + scales, gathered qx rows + sx (one token: the bf16 row),
        # h written (fp32)
        "gateup_bytes": n_act * (2 * i * h + sc_gu) + (2 * h if one_token else r * (h + (h // 128) * 4)) + r * i * 4,
        # decode down kernel: touched W_down + scales, qh rows + sh, y rows written (fp32)
        "down_bytes": n_act * (h * i + sc_d) + r * (i + (i // 128) * 4) + r * h * 4,
        "layer_weight_bytes": n_act * (3 * h * i + sc_gu + sc_d),
        "gateup_flops": 2 * 2 * r * h * i,
        "down_flops": 2 * r * h * i,
    }


def prefill_gemm_bytes(w, ids, groups):
    """Algorithmic HBM bytes of the prefill GEMM launches of one layer call,
    one launch pair per group [e0, e1) of experts: gate/up reads the group's
    active experts' W_gate, W_up and scales once, each token row (qx + sx)
    with a slot in the group once, and writes qh + sh of the group's routed
    rows; down reads the active experts' W_down and scales and those qh + sh
    rows once, and writes the rows' fp32 outputs."""
    import numpy as np
    h, i = w.hidden, w.inter
    sc_gu = 2 * (i // 128) * (h // 128) * 4
    sc_d = (h // 128) * (i // 128) * 4
    gu = dn = 0
    for e0, e1 in groups:
        m = (ids >= e0) & (ids < e1)
        rows = int(m.sum())
        toks = int(m.any(axis=1).sum())
        act = int(np.unique(ids[m]).size)
        gu += act * (2 * i * h + sc_gu) + toks * (h + (h // 128) * 4) + rows * (i + (i // 128) * 4)
        dn += act * (h * i + sc_d) + rows * (i + (i // 128) * 4) + rows * h * 4
    return gu, dn


def profile_steps(moe, torch, step, n_steps, per_step):
    """Kernel durations of n_steps steps from the library's launch events:
    {name: (launches, total ms)}."""
    moe.moe_profile_begin(per_step * n_steps)
    for i in range(n_steps):
        step(i)
    prof = moe.moe_profile_end()
    torch.cuda.synchronize()
    kern = {}
    for kname, kms in prof:
        n, tot = kern.get(kname, (0, 0.0))
        kern[kname] = (n + 1, tot + kms)
    return kern


def time_resident(moe, torch, synth, cache, name, steps, warmup, layers_n, w8a16=False, fused=True):
    import numpy as np
    w = synth.WORKLOADS[name]
    if w.chunk_tokens:
        raise SystemExit(f"{name}: a streamed workload, not a resident one")
    x = synth.activations(w)
    ids, wts = synth.routing(w)
    dx = torch.from_numpy(x.view(np.int16)).cuda()
    dids = torch.from_numpy(ids).cuda()
    dw = torch.from_numpy(wts).cuda()
    layers = [cache.get(w, l) for l in range(layers_n)]
    buf = moe.MoELayerBuffers(w.hidden, w.inter, w.n_experts, w.topk, w.tokens, with_status=False, w8a16=w8a16,
                              fused=fused and not w8a16)
    stream = torch.cuda.current_stream()

    def step(i):
        moe.run_layer(buf, dx, dids, dw, layers[i % len(layers)], stream)

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for i in range(steps):
        step(i)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    # Per-kernel durations: the same steps again with the library's launch events.
    kern = profile_steps(moe, torch, step, steps, 16)
    out = buf.out.cpu().numpy()
    if not np.all(np.isfinite((out.view(np.uint16).astype(np.uint32) << 16).view(np.float32))):
        raise RuntimeError("non-finite output")
    return w, ids, wts, x, ms, kern


def decode_roofline(alg, kern, steps, workload):
    """Decode gate/up GEMV against HBM (per step: the launches of its row-count classes)."""
    dom = "ffn_decode_gateup"
    n, tot_ms = kern[dom]
    us = 1000.0 * tot_ms / steps
    achieved = alg["gateup_bytes"] / (us * 1e-6) / 1e9
    return {"kernel": dom, "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(workload, dom),
            "per_launch": {"algorithmic_bytes_per_step": alg["gateup_bytes"], "launches_per_step": n // steps,
                           "us_per_step": round(us, 2)}}


def prefill_roofline(flops_total, bytes_total, kern, dom, workload, launches_note=""):
    """A prefill GEMM kernel against its roofline: algorithmic FLOPs and HBM
    bytes per launch over its mean launch duration.  The bound is the larger
    of FLOPs at the dense FP8 MFMA peak and bytes at the HBM peak, i.e. the
    side of the ridge point (5.0 PFLOP/s / 8 TB/s = 625 FLOP/B) the launch's
    arithmetic intensity falls on: an expert with a few hundred rows (8192
    tokens over 256 experts) reads more weight bytes than its MFMAs can hide,
    an expert group with thousands of rows (the 32768-token streamed layer)
    does not.  Both fractions are reported."""
    n, tot_ms = kern[dom]
    avg_us = 1000.0 * tot_ms / n
    flops = flops_total / n
    nbytes = bytes_total / n
    tflops = flops / (avg_us * 1e-6) / 1e12
    gbs = nbytes / (avg_us * 1e-6) / 1e9
    mfma = flops / (FP8_PEAK_TFLOPS * 1e12) >= nbytes / (HBM_PEAK_GBS * 1e9)
    achieved, peak, unit = (tflops, FP8_PEAK_TFLOPS, "TFLOP/s") if mfma else (gbs, HBM_PEAK_GBS, "GB/s")
    return {"kernel": dom, "bound": "mfma" if mfma else "hbm", "achieved": round(achieved, 1), "peak": peak,
            "unit": unit, "frac": round(achieved / peak, 4), "traffic": measured_traffic(workload, dom),
            "per_launch": {"launches": n, "algorithmic_flops": round(flops), "algorithmic_bytes": round(nbytes),
                           "flop_per_byte": round(flops / nbytes, 1), "avg_us": round(avg_us, 2),
                           "TFLOPs": round(tflops, 1), "frac_of_fp8_peak": round(tflops / FP8_PEAK_TFLOPS, 4),
                           "GBps": round(gbs, 1), "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
                           **({"note": launches_note} if launches_note else {})}}


def resident_summary(moe, torch, synth, cache, extra, steps, warmup, layers_n, fused):
    base_name, w8a16 = (extra[:-len("_w8a16")], True) if extra.endswith("_w8a16") else (extra, False)
    w0 = synth.WORKLOADS[base_name]
    decode = w0.tokens <= moe.MOE_DECODE_MAX_TOKENS
    n_layers = layers_n if decode else 1
    w, ids, _, _, ms, kern = time_resident(moe, torch, synth, cache, base_name, steps, warmup, n_layers,
                                           w8a16=w8a16, fused=fused)
    alg = algorithmic(w, ids)
    kern_us = {k: round(1000.0 * tot / steps, 2) for k, (n, tot) in kern.items()}
    res = {"tokens_per_s": round(w.tokens / (ms / 1000.0), 1), "ms_per_step": round(ms, 4),
           "tokens": w.tokens, "routing": w.routing + (f"({w.zipf_s})" if w.routing == "zipf" else ""),
           "active_experts": alg["active_experts"],
           "layer_weight_GBps": round(alg["layer_weight_bytes"] / (ms * 1e-3) / 1e9, 1),
           "weight_layers_rotated": n_layers, "kernel_us_per_step": kern_us}
    if w8a16:
        dom = "ffn_decode_w8a16_gateup"
        n, tot = kern[dom]
        us = 1000.0 * tot / steps
        ach = alg["gateup_bytes"] / (us * 1e-6) / 1e9   # same weight bytes; activations counted as in W8A8
        res["roofline"] = {"kernel": dom, "bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS,
                           "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4),
                           "traffic": measured_traffic(extra, dom)}
    elif decode:
        res["roofline"] = decode_roofline(alg, kern, steps, base_name)
        res["layer_frac_hbm"] = round(alg["layer_weight_bytes"] / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
    else:
        gu_b, dn_b = prefill_gemm_bytes(w, ids, [(0, w.n_experts)])
        res["roofline"] = prefill_roofline(alg["gateup_flops"] * steps, gu_b * steps, kern, "ffn_prefill_gateup",
                                           base_name)
        res["roofline_down"] = prefill_roofline(alg["down_flops"] * steps, dn_b * steps, kern, "ffn_prefill_down",
                                                base_name)
        res["layer_TFLOPs"] = round((alg["gateup_flops"] + alg["down_flops"]) / (ms * 1e-3) / 1e12, 1)
    return res


def time_router(moe, torch, synth, w, steps, warmup):
    """The gate (moe_router) on the workload's tokens: DeepSeek-V3 grouping
    (8 groups, 4 kept), bf16 router weight [E, H], per-expert bias."""
    import numpy as np
    x = synth.activations(w)
    wr, bias = synth.router_params(w, bias_std=0.05)
    dx = torch.from_numpy(x.view(np.int16)).cuda()
    dwr = torch.from_numpy(wr.view(np.int16)).cuda()
    db = torch.from_numpy(bias).cuda()
    ids = torch.empty((w.tokens, w.topk), dtype=torch.int32, device="cuda")
    wts = torch.empty((w.tokens, w.topk), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(1, moe.moe_router_workspace(w.tokens, w.hidden, w.n_experts)), dtype=torch.uint8,
                     device="cuda")
    groups = 8 if w.n_experts % 8 == 0 and w.n_experts >= 16 else 1

    def call(_i=0):
        moe.moe_router(dx, dwr, db, ids, wts, groups, min(4, groups), 1.0, ws)

    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    kern = profile_steps(moe, torch, call, steps, 4)
    return {kk: round(1000.0 * tot / n, 2) for kk, (n, tot) in kern.items()}


def time_streamed(moe, torch, synth, cache, name, steps, warmup):
    """Stream-loaded layers: weights in pinned host memory, streamed through a
    ring of expert slots (all experts of a layer by default).  With several
    layers (stream-loading across a stack, each layer with its own weights and
    routing) every layer's output is the next layer's input and all layers
    share one ring and one stream context."""
    import numpy as np
    w = synth.WORKLOADS[name]
    n_layers = max(1, w.layers)
    n_sets = w.weight_sets or n_layers  # distinct weight layers; layer l uses set l mod n_sets
    x = synth.activations(w)
    routes = [synth.routing(w, layer=l) for l in range(n_layers)]
    host_layers = []
    for l in range(n_sets):
        dev_layer = cache.get(w, l)
        log(f"pinning a host copy of weight layer {l}")
        host = []
        for t in dev_layer:
            h = torch.empty(t.shape, dtype=t.dtype, pin_memory=True)
            h.copy_(t)
            host.append(h)
        host_layers.append(tuple(host))
        if l > 0:   # layer 0 stays resident for the resident workloads of the same run
            del cache.layers[(w.hidden, w.inter, w.n_experts, w.seed, l)]
        del dev_layer
        torch.cuda.empty_cache()
    dims = moe.MoeDims(w.hidden, w.inter, w.n_experts, w.topk)
    slots = w.ring_slots or w.n_experts
    ctx = moe.StreamContext(slots)
    ring = torch.empty(moe.moe_ring_bytes(dims, slots), dtype=torch.uint8, device="cuda")
    ring_s = torch.empty(moe.moe_ring_scale_bytes(dims, slots) // 4, dtype=torch.float32, device="cuda")
    ws = torch.empty(moe.moe_ffn_streamed_workspace(dims, w.tokens, w.chunk_tokens), dtype=torch.uint8,
                     device="cuda")
    outs = [torch.empty((w.tokens, w.hidden), dtype=torch.int16, device="cuda") for _ in range(2)]
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    dx = torch.from_numpy(x.view(np.int16)).cuda()
    dids = [torch.from_numpy(ids).cuda() for ids, _ in routes]
    dws = [torch.from_numpy(wts).cuda() for _, wts in routes]
    compute = torch.cuda.current_stream()
    copy = torch.cuda.Stream()

    def step(_i=0):
        inp = dx
        for l in range(n_layers):
            moe.moe_ffn_streamed(dims, w.chunk_tokens, inp, dids[l], dws[l], host_layers[l % n_sets], ring, ring_s,
                                 ctx, outs[l % 2], status, ws, compute, copy)
            inp = outs[l % 2]

    def timed(fn, n):
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(compute)
        for _ in range(n):
            fn()
        e1.record(compute)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    for _ in range(warmup):
        step()
    ms = timed(step, steps)
    if int(status.item()) != 0:
        raise RuntimeError("device status reported bad routing ids")
    # Copy-only reference: the same bytes host -> device through the same
    # ring (slot-sized pieces, wrapping) on the copy stream, no kernels.
    per_slot = [ring.numel() // 3 // slots, ring_s.numel() // 3 // slots]
    ring_parts = [ring[i * (ring.numel() // 3):(i + 1) * (ring.numel() // 3)] for i in range(3)]
    scale_parts = [ring_s[i * (ring_s.numel() // 3):(i + 1) * (ring_s.numel() // 3)] for i in range(3)]

    def copies():
        with torch.cuda.stream(copy):
            for host in (host_layers[l % n_sets] for l in range(n_layers)):
                for e0 in range(0, w.n_experts, slots):
                    n = min(slots, w.n_experts - e0)
                    for m in range(3):
                        ring_parts[m][: n * per_slot[0]].copy_(host[2 * m][e0:e0 + n].view(-1), non_blocking=True)
                        scale_parts[m][: n * per_slot[1]].copy_(host[2 * m + 1][e0:e0 + n].view(-1),
                                                               non_blocking=True)
        compute.wait_stream(copy)

    copy_ms = [timed(copies, 1) for _ in range(3)]
    # Copy-only time of each layer on its own, and where its pinned host
    # buffers sit (pages per NUMA node).
    per_layer = []
    for li, host in enumerate(host_layers):
        def one_layer(host=host):
            with torch.cuda.stream(copy):
                for e0 in range(0, w.n_experts, slots):
                    n = min(slots, w.n_experts - e0)
                    for m in range(3):
                        ring_parts[m][: n * per_slot[0]].copy_(host[2 * m][e0:e0 + n].view(-1), non_blocking=True)
                        scale_parts[m][: n * per_slot[1]].copy_(host[2 * m + 1][e0:e0 + n].view(-1),
                                                               non_blocking=True)
            compute.wait_stream(copy)
        per_layer.append({"layer": li, "copy_only_ms": [round(timed(one_layer, 1), 3) for _ in range(2)],
                          "host_pages_per_numa_node": numa_pages([t.data_ptr() for t in host])})
    # Kernel durations of the timed number of steps with the library's launch events.
    kern = profile_steps(moe, torch, step, steps, max(4000, 200 * n_layers))
    ctx.close()
    h2d_bytes = sum(t.numel() * t.element_size() for l in range(n_layers) for t in host_layers[l % n_sets])
    ids_all = np.concatenate([ids for ids, _ in routes])
    out0 = outs[(n_layers - 1) % 2].cpu().numpy()
    if not np.all(np.isfinite((out0.view(np.uint16).astype(np.uint32) << 16).view(np.float32))):
        raise RuntimeError("non-finite output")
    return w, ids_all, routes[0][1], x, ms, copy_ms, h2d_bytes, kern, per_layer


def numa_pages(ptrs):
    """Host memory placement: pages per NUMA node of the mappings that hold the
    given host addresses (from /proc/self/maps and /proc/self/numa_maps)."""
    try:
        maps = []
        with open("/proc/self/maps") as f:
            for line in f:
                a, b = line.split()[0].split("-")
                maps.append((int(a, 16), int(b, 16)))
        nodes = {}
        with open("/proc/self/numa_maps") as f:
            for line in f:
                parts = line.split()
                nodes[int(parts[0], 16)] = {p.split("=")[0]: int(p.split("=")[1]) for p in parts[1:]
                                            if p.startswith("N") and "=" in p}
    except OSError:
        return None
    out = {}
    for start, end in maps:
        if any(start <= p < end for p in ptrs):
            for n, c in nodes.get(start, {}).items():
                out[n] = out.get(n, 0) + c
    return out


def cpu_baseline(torch, synth, w, x, ids, wts, budget_s, tokens):
    """The oracle as it stands, on a bounded sample of the workload (the given tokens)."""
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        blas_threads = os.cpu_count() or 1
    k = w.topk
    experts = sorted(set(ids[tokens].reshape(-1).tolist()))
    ow = {}
    for e in experts:   # weight preparation (not timed): re-drawn fp32, quantized by the oracle
        mats = []
        for which in range(3):
            f = synth.expert_weight_device(w, 0, e, which).cpu().numpy()
            mats += list(oracle.quantize_weight(f))
        ow[e] = tuple(mats)
    done = 0
    t0 = time.perf_counter()
    while True:
        qx, sx = oracle.quant_act(x[tokens])
        sub_ids = ids[tokens]
        offsets, src, dest = oracle.permute(sub_ids, w.n_experts)
        y = np.zeros((len(tokens) * k, w.hidden), np.float32)
        for e in experts:
            p0, p1 = int(offsets[e]), int(offsets[e + 1])
            if p1 > p0:
                rows = src[p0:p1] // k
                y[p0:p1] = oracle.expert_rows(qx[rows], sx[rows], *ow[e])
        oracle.combine(y, dest, wts[tokens])
        done += len(tokens)
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    return {"value": done / el, "unit": "tokens/s", "cores": int(blas_threads), "kind": "oracle",
            "host_cpu_count": os.cpu_count(), "blas_threads": int(blas_threads),
            "sample": f"token(s) {tokens[0]}..{tokens[-1]} of the {w.tokens}-token workload ({len(experts)} experts): "
                      f"the full layer path (quantize, permute, expert FFN, combine) repeated "
                      f"{done // len(tokens)} times in {el:.1f} s; weight quantization excluded"}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}); "
              "the multi-GPU expert-parallel path is not built", file=sys.stderr)
        sys.exit(2)
    import synth
    w_main = synth.WORKLOADS[args.workload]
    if w_main.layers > 1 and "HSA_ENABLE_SDMA" not in os.environ:
        # A stack of layers through a small ring waits for a slot before most
        # group copies: shader copies (SDMA off) resolve those waits with
        # shorter gaps between copies than the DMA engines (measured: 803 vs
        # 893 ms per 4-layer step of slp4_ring32); a single layer per step is
        # as fast or faster on the DMA engines, the runtime's default.  Set
        # before the HIP runtime starts.
        os.environ["HSA_ENABLE_SDMA"] = "0"
    import numpy as np  # noqa: F401
    import torch

    import paper_2606_10493_amd as moe

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    torch.cuda.set_device(0)
    if args.copy_calibration:
        n = 1 << 30
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": n, "copy_calibration_bytes_written": n, "launches": 5}))
        return
    cache = LayerCache(moe, torch, synth)
    w0 = synth.WORKLOADS[args.workload]
    layers_n = args.layers or 4
    if w0.chunk_tokens:
        steps, warmup = args.steps or 10, args.warmup or 2
        res, w, x, ids, wts = main_streamed(args, moe, torch, synth, cache, steps, warmup)
    else:
        steps, warmup = args.steps or 50, args.warmup or 10
        res, w, x, ids, wts = main_resident(args, moe, torch, synth, cache, steps, warmup, layers_n)
    also = {}
    r_steps, r_warm = args.steps or 50, args.warmup or 10
    for extra in [a for a in args.also.split(",") if a and a != args.workload]:
        log(f"also: {extra}")
        if extra == "router":
            kus = time_router(moe, torch, synth, w, r_steps, r_warm)
            also["router"] = {"tokens": w.tokens, "kernel_us": kus}
            if kus.get("router_logits"):
                # logits = x W_r^T: 2 T H E FLOPs of bf16 MFMA over the bf16 hidden states and router weight
                # read once and the fp32 logits written once (the selection is latency-bound and small).  The
                # bound is the side of the bf16 ridge point (2.5 PFLOP/s / 8 TB/s = 312.5 FLOP/B) the
                # intensity falls on: about E = 256 FLOP/B, so HBM.
                t, h, e = w.tokens, w.hidden, w.n_experts
                flops = 2.0 * t * h * e
                nbytes = 2.0 * t * h + 2.0 * e * h + 4.0 * t * e
                sec = kus["router_logits"] * 1e-6
                tf, gbs = flops / sec / 1e12, nbytes / sec / 1e9
                mfma = flops / (BF16_PEAK_TFLOPS * 1e12) >= nbytes / (HBM_PEAK_GBS * 1e9)
                ach, peak, unit = (tf, BF16_PEAK_TFLOPS, "TFLOP/s") if mfma else (gbs, HBM_PEAK_GBS, "GB/s")
                also["router"]["roofline"] = {
                    "kernel": "router_logits", "bound": "mfma" if mfma else "hbm", "achieved": round(ach, 1),
                    "peak": peak, "unit": unit, "frac": round(ach / peak, 4), "traffic": None,
                    "per_launch": {"algorithmic_flops": round(flops), "algorithmic_bytes": round(nbytes),
                                   "flop_per_byte": round(flops / nbytes, 1), "us": kus["router_logits"],
                                   "TFLOPs": round(tf, 1), "frac_of_bf16_peak": round(tf / BF16_PEAK_TFLOPS, 4),
                                   "GBps": round(gbs, 1), "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4)}}
            continue
        base = extra[:-len("_w8a16")] if extra.endswith("_w8a16") else extra
        if synth.WORKLOADS[base].chunk_tokens:
            also[extra] = {"skipped": "streamed workloads run as the main --workload"}
            continue
        also[extra] = resident_summary(moe, torch, synth, cache, extra, r_steps, r_warm, layers_n,
                                       fused=not args.unfused)
    res["also"] = also
    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        sample = list(range(w.tokens)) if w.tokens <= 4 else [0]
        cpu = cpu_baseline(torch, synth, w, x, ids, wts, args.cpu_seconds, sample)
    res["cpu_baseline"] = cpu
    print(json.dumps(res), flush=True)


def main_resident(args, moe, torch, synth, cache, steps, warmup, layers_n):
    w0 = synth.WORKLOADS[args.workload]
    decode = w0.tokens <= moe.MOE_DECODE_MAX_TOKENS
    n_layers = layers_n if decode else 1
    w, ids, wts, x, ms, kern = time_resident(moe, torch, synth, cache, args.workload, steps, warmup, n_layers,
                                             fused=not args.unfused)
    alg = algorithmic(w, ids)
    if decode:
        roof = decode_roofline(alg, kern, steps, args.workload)
    else:
        gu_b, _ = prefill_gemm_bytes(w, ids, [(0, w.n_experts)])
        roof = prefill_roofline(alg["gateup_flops"] * steps, gu_b * steps, kern, "ffn_prefill_gateup", args.workload)
    layer_gbs = alg["layer_weight_bytes"] / (ms * 1e-3) / 1e9
    layer_tflops = (alg["gateup_flops"] + alg["down_flops"]) / (ms * 1e-3) / 1e12
    res = {
        "metric": METRIC, "value": round(w.tokens / (ms / 1000.0), 2), "unit": "tokens/s", "n_gpus": 1,
        "steps": steps, "warmup": warmup, "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "fp8_e4m3 (fp32 accumulate)", "data": "synthetic",
        "config": {"workload": args.workload, "hidden": w.hidden, "inter": w.inter, "n_experts": w.n_experts,
                   "topk": w.topk, "tokens": w.tokens, "routing": w.routing,
                   "weight_layers_rotated": n_layers, "active_experts": alg["active_experts"],
                   "entry": "four calls" if args.unfused else "moe_ffn_layer"},
        "layer": {"weight_GBps": round(layer_gbs, 1), "frac_hbm": round(layer_gbs / HBM_PEAK_GBS, 4),
                  "TFLOPs": round(layer_tflops, 2)},
        "roofline": roof,
        "kernel_us_per_step": {k: round(1000.0 * tot / steps, 2) for k, (n, tot) in kern.items()},
    }
    return res, w, x, ids, wts


def streamed_gemm_bytes(moe, w, ids_all, n_layers):
    """prefill_gemm_bytes of every layer call of a streamed step, with the
    expert groups of the call's launches taken from the ring schedule the
    library executes (moe_stream_schedule)."""
    dims = moe.MoeDims(w.hidden, w.inter, w.n_experts, w.topk)
    slots = w.ring_slots or w.n_experts
    ops, _ = moe.moe_stream_schedule(dims, w.tokens, w.chunk_tokens, slots)
    groups = [(a, a + b) for op, a, b, _c in ops if op == moe.MOE_SOP_LAUNCH]
    gu = dn = 0
    for layer in range(n_layers):
        g, d = prefill_gemm_bytes(w, ids_all[layer * w.tokens:(layer + 1) * w.tokens], groups)
        gu += g
        dn += d
    return gu, dn


def main_streamed(args, moe, torch, synth, cache, steps, warmup):
    w, ids, wts, x, ms, copy_ms, h2d_bytes, kern, per_layer = time_streamed(moe, torch, synth, cache, args.workload,
                                                                            steps, warmup)
    n_layers = max(1, w.layers)
    alg = algorithmic(w.with_tokens(w.tokens * n_layers), ids)
    gu_n, gu_ms = kern.get("ffn_prefill_gateup", (0, 0.0))
    dn_n, dn_ms = kern.get("ffn_prefill_down", (0, 0.0))
    copy_best = min(copy_ms)
    h2d_gbs = h2d_bytes / (copy_best * 1e-3) / 1e9
    note = "launches per step: one per expert group (over all 4096-token chunks)"
    if os.environ.get("HSA_ENABLE_SDMA") == "0":
        note += ("; with shader copies the copy kernels share the compute units with the expert kernels, so "
                 "these launch durations include waiting for them")
    gu_b, dn_b = streamed_gemm_bytes(moe, w, ids, n_layers)
    roof = prefill_roofline(alg["gateup_flops"] * steps, gu_b * steps, kern, "ffn_prefill_gateup", args.workload,
                            note)
    roof_dn = prefill_roofline(alg["down_flops"] * steps, dn_b * steps, kern, "ffn_prefill_down", args.workload,
                               note)
    res = {
        "metric": METRIC, "value": round(w.tokens / (ms / 1000.0), 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": steps, "warmup": warmup, "ms_per_step": round(ms, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "fp8_e4m3 (fp32 accumulate)", "data": "synthetic",
        "config": {"workload": args.workload, "hidden": w.hidden, "inter": w.inter, "n_experts": w.n_experts,
                   "topk": w.topk, "tokens": w.tokens, "chunk_tokens": w.chunk_tokens, "routing": w.routing,
                   "zipf_s": w.zipf_s, "layers": n_layers, "ring_slots": w.ring_slots or w.n_experts,
                   "weight_sets": w.weight_sets or n_layers,
                   "entry": "moe_ffn_streamed",
                   "host_to_device": os.environ.get("HSA_ENABLE_SDMA") == "0" and "shader copies (HSA_ENABLE_SDMA=0)"
                   or "runtime default (DMA engines)"},
        "streaming": {"h2d_bytes": h2d_bytes, "copy_only_ms": [round(c, 3) for c in copy_ms],
                      "h2d_GBps_copy_only": round(h2d_gbs, 2),
                      "h2d_GBps_in_layer": round(h2d_bytes / (ms * 1e-3) / 1e9, 2),
                      "frac_of_copy_only": round(copy_best / ms, 4),
                      "layer_tokens_per_s": round(n_layers * w.tokens / (ms / 1000.0), 1),
                      "exposed_compute_ms": round(ms - copy_best, 3),
                      "gemm_kernel_ms_per_step": round((gu_ms + dn_ms) / steps, 3),
                      "gemm_TFLOPs": round((alg["gateup_flops"] + alg["down_flops"]) /
                                           ((gu_ms + dn_ms) / steps * 1e-3) / 1e12, 1),
                      "per_layer": per_layer},
        "roofline": roof,
        "roofline_down": roof_dn,
        "kernel_ms_per_step": {k: round(tot / steps, 3) for k, (n, tot) in kern.items()},
    }
    return res, w, x, ids, wts


if __name__ == "__main__":
    main()
