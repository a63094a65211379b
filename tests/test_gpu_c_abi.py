"""GPU: the layer through the C ABI from a plain C++ program (no Python, no
torch in that process).

tests/abi_c_layer.cpp (built by __graft_entry__.build() into
tests/_bin/abi_c_layer, linked against the in-tree libmoe.so) reads the
inputs from files, allocates device memory with hipMalloc, quantizes and
packs the weights, and runs the layer on a stream of its own, through
moe_ffn_layer and through the four calls.  Both outputs must equal the
Python binding's output on the same inputs bit for bit, and the oracle's
within 2e-2.
"""
import os
import subprocess

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_cases import bf16_dev, log, quantize_weights_gpu, rel_err, require_gpu, to_dev

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXE = os.path.join(ROOT, "tests", "_bin", "abi_c_layer")
CASES = [
    (256, 128, 8, 2, 16, "uniform", "decode"),    # the tiny layer
    (256, 128, 8, 2, 16, "uniform", "prefill"),
    (512, 256, 16, 4, 300, "zipf", "prefill"),    # several tiles; the multi-chunk sort (T > 256)
]


@pytest.fixture(scope="module")
def moe():
    return require_gpu()


@pytest.mark.skipif(not os.path.exists(EXE), reason="tests/_bin/abi_c_layer is built by __graft_entry__.build()")
@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}x{c[1]}x{c[2]}x{c[3]}x{c[4]}{c[5]}-{c[6]}")
def test_layer_from_plain_cpp_equals_python_binding(moe, case, tmp_path):
    h, i, e, k, t, routing, regime = case
    rule = "softmax" if (h, i, e, k, t) == (256, 128, 8, 2, 16) else "sigmoid"
    w = synth.Workload("c_abi", h, i, e, k, t, routing, 1.0 if routing == "zipf" else 0.0, rule)
    x = synth.activations(w)
    ids, wts = synth.routing(w)
    wg, wu, wd = synth.weights_host(w)
    for name, arr in (("x", x), ("ids", ids), ("wts", wts), ("wg", wg), ("wu", wu), ("wd", wd)):
        np.ascontiguousarray(arr).tofile(tmp_path / f"{name}.bin")
    rg = moe.MOE_REGIME_DECODE if regime == "decode" else moe.MOE_REGIME_PREFILL
    log(f"C ABI program: {case}")
    res = subprocess.run([EXE, str(h), str(i), str(e), str(k), str(t), str(rg), str(tmp_path), str(tmp_path)],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    fused = np.fromfile(tmp_path / "out_fused.bin", dtype=np.uint16).reshape(t, h)
    calls = np.fromfile(tmp_path / "out_calls.bin", dtype=np.uint16).reshape(t, h)
    assert np.array_equal(fused, calls)

    dweights = quantize_weights_gpu(moe, wg, wu, wd)
    buf = moe.MoELayerBuffers(h, i, e, k, t, rg, fused=True)
    moe.run_layer(buf, bf16_dev(x), to_dev(ids), to_dev(wts), dweights)
    torch.cuda.synchronize()
    assert np.array_equal(fused, buf.out.cpu().numpy().view(np.uint16)), "C program and Python binding differ"

    ref = oracle.bf16_to_f32(oracle.moe_layer(x, ids, wts, oracle.prepare_weights(wg, wu, wd)))
    err = rel_err(oracle.bf16_to_f32(fused), ref)
    log(f"C ABI program: {case} vs oracle {err:.3e}")
    assert err <= 2e-2
