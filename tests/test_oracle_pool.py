"""The process-pool helper of the full-size parity tests returns exactly what
the oracle returns when called directly (CPU only)."""
import numpy as np

import oracle
import oracle_pool
import synth


def test_pooled_weight_quantization_equals_direct_calls():
    rng = np.random.default_rng(3)
    mats = [(0.02 * rng.standard_normal((256, 384))).astype(np.float32) for _ in range(5)]
    for (q, s), m in zip(oracle_pool.quantize_weights(mats), mats):
        q_ref, s_ref = oracle.quantize_weight(m)
        assert np.array_equal(q, q_ref) and np.array_equal(s.view(np.uint32), s_ref.view(np.uint32))


def test_pooled_activation_quantization_equals_one_call():
    w = synth.Workload("pool", 512, 256, 8, 2, 700, "uniform")
    x = synth.activations(w)
    q, s = oracle_pool.quant_act_rows(x, rows_per_task=96)
    q_ref, s_ref = oracle.quant_act(x)
    assert np.array_equal(q, q_ref) and np.array_equal(s.view(np.uint32), s_ref.view(np.uint32))
