"""bench.py's roofline arithmetic on the CPU: the algorithmic bytes of the
prefill GEMM launches against a brute-force count, the choice of the bound
from the arithmetic intensity (the side of the ridge point), and the
streamed layer's launch groups taken from the ring schedule the library
executes (a host-only call)."""
import dataclasses

import numpy as np
import pytest

import bench
import synth


def _brute_bytes(w, ids, groups):
    """One launch pair per group, counted row by row and token by token."""
    h, i = w.hidden, w.inter
    sc_gu = 2 * (i // 128) * (h // 128) * 4
    sc_d = (h // 128) * (i // 128) * 4
    gu = dn = 0
    for e0, e1 in groups:
        experts, tokens, rows = set(), set(), 0
        for t in range(ids.shape[0]):
            for j in range(ids.shape[1]):
                e = int(ids[t, j])
                if e0 <= e < e1:
                    experts.add(e)
                    tokens.add(t)
                    rows += 1
        # gate/up: W_gate + W_up + scales per active expert, qx + sx per token, qh + sh per row
        gu += len(experts) * (2 * h * i + sc_gu) + len(tokens) * (h + h // 128 * 4) + rows * (i + i // 128 * 4)
        # down: W_down + scales per active expert, qh + sh per row read, fp32 y per row written
        dn += len(experts) * (h * i + sc_d) + rows * (i + i // 128 * 4) + rows * h * 4
    return gu, dn


@pytest.mark.parametrize("groups", [[(0, 16)], [(0, 4), (4, 8), (8, 12), (12, 16)], [(0, 5), (5, 16)]])
def test_prefill_gemm_bytes_against_brute_force(groups):
    w = synth.Workload("bytes", 512, 256, 16, 4, 300, "zipf", 1.2)
    ids, _ = synth.routing(w)
    assert bench.prefill_gemm_bytes(w, ids, groups) == _brute_bytes(w, ids, groups)


def test_prefill8k_bytes_and_intensity():
    """The 8192-token chunk: 7.717 GB and 5.776 GB, 499 and 333 FLOP/B (the
    figures the design notes and profiles quote), both below the ridge."""
    w = synth.WORKLOADS["prefill8k"]
    ids, _ = synth.routing(w)
    gu, dn = bench.prefill_gemm_bytes(w, ids, [(0, w.n_experts)])
    alg = bench.algorithmic(w, ids)
    assert gu == 7_716_995_072 and dn == 5_776_474_112
    ridge = bench.FP8_PEAK_TFLOPS * 1e12 / (bench.HBM_PEAK_GBS * 1e9)
    assert ridge == pytest.approx(625.0)
    assert alg["gateup_flops"] / gu == pytest.approx(498.7, abs=0.1) and alg["gateup_flops"] / gu < ridge
    assert alg["down_flops"] / dn == pytest.approx(333.1, abs=0.1)


def test_prefill_roofline_takes_the_binding_side():
    """The bound is whichever of FLOPs at the FP8 peak and bytes at the HBM
    peak takes longer; the fraction is in that unit; both are reported."""
    flops, nbytes, n, us = 4.0e12, 8.0e9, 5, 2000.0
    kern = {"k": (n, n * us / 1000.0)}
    r = bench.prefill_roofline(flops * n, nbytes * n, kern, "k", "none")
    assert r["bound"] == "hbm" and r["unit"] == "GB/s"      # 1.0 ms of bytes > 0.8 ms of FLOPs
    assert r["achieved"] == pytest.approx(4000.0) and r["frac"] == pytest.approx(0.5)
    assert r["per_launch"]["frac_of_fp8_peak"] == pytest.approx(0.4)
    r = bench.prefill_roofline(flops * n, nbytes / 4 * n, kern, "k", "none")
    assert r["bound"] == "mfma" and r["unit"] == "TFLOP/s"  # 0.25 ms of bytes < 0.8 ms of FLOPs
    assert r["achieved"] == pytest.approx(2000.0) and r["frac"] == pytest.approx(0.4)
    assert r["per_launch"]["flop_per_byte"] == pytest.approx(2000.0)


def test_streamed_bytes_follow_the_ring_schedule():
    """The streamed layer's launches are the LAUNCH ops of moe_stream_schedule
    (16 groups of 16 experts for the 32768-token workload); summed over them
    the bytes equal the brute-force count over those groups."""
    moe = pytest.importorskip("paper_2606_10493_amd")
    w = dataclasses.replace(synth.WORKLOADS["prefill32k_streamed"], tokens=4096, chunk_tokens=1024)
    ids, _ = synth.routing(w)
    dims = moe.MoeDims(w.hidden, w.inter, w.n_experts, w.topk)
    ops, _ = moe.moe_stream_schedule(dims, w.tokens, w.chunk_tokens, w.ring_slots or w.n_experts)
    groups = [(a, a + b) for op, a, b, _c in ops if op == moe.MOE_SOP_LAUNCH]
    assert groups[0][0] == 0 and groups[-1][1] == w.n_experts
    assert all(g1 == h0 for (_, g1), (h0, _) in zip(groups, groups[1:]))
    assert bench.streamed_gemm_bytes(moe, w, ids, 1) == _brute_bytes(w, ids, groups)
    # One group over all experts moves the weights once; split groups re-read no weight but re-read tokens.
    one_gu, one_dn = bench.prefill_gemm_bytes(w, ids, [(0, w.n_experts)])
    gu, dn = bench.streamed_gemm_bytes(moe, w, ids, 1)
    assert dn == one_dn and gu >= one_gu and np.isclose(gu, one_gu, rtol=0.2)
