"""Pins of the oracle's permutation, block-scaled GEMM, expert FFN and combine.

Each check compares the oracle with something it does not compute itself:
brute-force sorting with Python's sorted(), exact integer arithmetic on the
e4m3 grid, an independently written dense FFN (torch fp8 casts + fp64
matmuls), a dense all-experts run masked by routing, and metamorphic
invariants (token permutation, expert relabelling, power-of-two scales).
"""
import numpy as np
import pytest
import torch

import oracle
import synth


# ----------------------------------------------------------------- permute
def _brute_permute(ids, n_exp):
    t, k = ids.shape
    slots = sorted(range(t * k), key=lambda f: (int(ids.reshape(-1)[f]), f))
    offsets = [0]
    for e in range(n_exp):
        offsets.append(offsets[-1] + sum(1 for f in range(t * k) if ids.reshape(-1)[f] == e))
    dest = [0] * (t * k)
    for p, f in enumerate(slots):
        dest[f] = p
    return offsets, slots, dest


@pytest.mark.parametrize("t,k,e,seed", [(1, 1, 1, 0), (5, 2, 8, 1), (16, 2, 8, 2),
                                        (33, 8, 256, 3), (7, 4, 5, 4), (0, 2, 4, 5)])
def test_permute_brute_force(t, k, e, seed):
    rng = np.random.default_rng(seed)
    ids = np.stack([rng.choice(e, k, replace=False) for _ in range(t)]).astype(np.int32) \
        if t else np.zeros((0, k), np.int32)
    off, src, dest = oracle.permute(ids, e)
    b_off, b_src, b_dest = _brute_permute(ids, e)
    assert list(off) == b_off and list(src) == b_src and list(dest) == b_dest
    # invariants
    assert off[-1] == t * k
    assert np.array_equal(dest[src], np.arange(t * k))
    tok_count = np.bincount(src // k, minlength=t) if t else np.zeros(0)
    assert np.all(tok_count == k)
    flat = ids.reshape(-1)
    assert np.all(np.diff(flat[src]) >= 0)


def test_permute_rejects_bad_ids():
    with pytest.raises(ValueError):
        oracle.permute(np.array([[0, 0]], np.int32), 4)
    with pytest.raises(ValueError):
        oracle.permute(np.array([[0, 4]], np.int32), 4)
    with pytest.raises(ValueError):
        oracle.permute(np.array([[-1, 1]], np.int32), 4)


# ----------------------------------------------------- block-scaled GEMM
def test_block_scaled_matmul_exact_on_grid_with_power_of_two_scales():
    """Small-integer e4m3 values and 2^j scales: every step is exact, so the
    oracle must equal the fp64 brute-force double sum exactly.  The scales
    differ per (row, block) and per (n-block, k-block) and the shapes are not
    square, so a swapped scale index or a transposed operand fails."""
    rng = np.random.default_rng(7)
    m, n, k = 5, 256, 384
    ints = np.array([-4, -3, -2, -1, 0, 1, 2, 3, 4], dtype=np.float32)
    a = rng.choice(ints, size=(m, k))
    w = rng.choice(ints, size=(n, k))
    a_q = oracle.e4m3_encode(a)
    w_q = oracle.e4m3_encode(w)
    a_s = np.ldexp(1.0, rng.integers(-3, 4, size=(m, k // 128))).astype(np.float32)
    w_s = np.ldexp(1.0, rng.integers(-3, 4, size=(n // 128, k // 128))).astype(np.float32)
    got = oracle.block_scaled_matmul(a_q, a_s, w_q, w_s)
    ref = np.zeros((m, n))
    for i in range(m):
        for j in range(n):
            tot = 0.0
            for b in range(k // 128):
                d = float(np.dot(a[i, b * 128:(b + 1) * 128].astype(np.float64),
                                 w[j, b * 128:(b + 1) * 128].astype(np.float64)))
                tot += d * float(a_s[i, b]) * float(w_s[j // 128, b])
            ref[i, j] = tot
    assert np.array_equal(got.astype(np.float64), ref)


def test_block_scaled_matmul_close_to_fp64_dequantized_product():
    rng = np.random.default_rng(8)
    x = rng.standard_normal((9, 512)).astype(np.float32)
    w = (0.02 * rng.standard_normal((384, 512))).astype(np.float32)
    a_q, a_s = oracle.quantize_rows(x)
    w_q, w_s = oracle.quantize_weight(w)
    # dequantize independently with torch's fp8 type
    a_deq = torch.from_numpy(a_q).view(torch.float8_e4m3fn).double().numpy() \
        * np.repeat(a_s.astype(np.float64), 128, axis=1)
    w_deq = torch.from_numpy(w_q).view(torch.float8_e4m3fn).double().numpy() \
        * np.kron(w_s.astype(np.float64), np.ones((128, 128)))
    ref = a_deq @ w_deq.T
    got = oracle.block_scaled_matmul(a_q, a_s, w_q, w_s)
    assert np.max(np.abs(got - ref)) / np.max(np.abs(ref)) < 1e-6


# ------------------------------------------------------------ full layer
def _tiny_inputs(seed=0, t=None):
    w = synth.WORKLOADS["tiny"]
    if seed:
        w = synth.Workload(**{**w.__dict__, "seed": seed})
    x = synth.activations(w, t)
    ids, wts = synth.routing(w, t)
    weights = oracle.prepare_weights(*synth.weights_host(w))
    return w, x, ids, wts, weights


def test_dense_masked_equals_moe_layer_bit_for_bit():
    for seed in (0, 1):
        _, x, ids, wts, weights = _tiny_inputs(seed)
        assert np.array_equal(oracle.moe_layer(x, ids, wts, weights),
                              oracle.moe_layer_dense(x, ids, wts, weights))


def _torch_ffn_fp64(x_bits, wg, wu, wd):
    """Independent dense FFN: torch fp8 casts for every quantization, fp64 GEMMs."""
    def q_rows(t32):
        t = t32.reshape(t32.shape[0], -1, 128)
        s = t.abs().amax(dim=2, keepdim=True) / torch.tensor(448.0)
        v = torch.where(s > 0, t / torch.where(s > 0, s, torch.ones_like(s)), t)
        deq = v.clamp(-448, 448).to(torch.float8_e4m3fn).double() * s.double()
        return deq.reshape(t32.shape)

    def q_w(m32):
        n, k = m32.shape
        blk = m32.reshape(n // 128, 128, k // 128, 128)
        s = blk.abs().amax(dim=(1, 3), keepdim=True) / torch.tensor(448.0)
        deq = (blk / s).clamp(-448, 448).to(torch.float8_e4m3fn).double() * s.double()
        return deq.reshape(n, k)

    x = torch.from_numpy(x_bits.view(np.int16)).view(torch.bfloat16).float()
    xq = q_rows(x)
    g = xq @ q_w(torch.from_numpy(wg)).T
    u = xq @ q_w(torch.from_numpy(wu)).T
    h = (g * torch.sigmoid(g) * u).float()
    y = q_rows(h) @ q_w(torch.from_numpy(wd)).T
    return y


def test_single_expert_identity_against_independent_dense_ffn():
    """E = 1, k = 1, w = 1: the layer is bf16(FFN(x))."""
    rng = np.random.default_rng(9)
    t, hdim, idim = 24, 384, 256
    x = synth.bf16_bits_from_f32(rng.standard_normal((t, hdim)).astype(np.float32))
    wg = (0.02 * rng.standard_normal((1, idim, hdim))).astype(np.float32)
    wu = (0.02 * rng.standard_normal((1, idim, hdim))).astype(np.float32)
    wd = (0.02 * rng.standard_normal((1, hdim, idim))).astype(np.float32)
    weights = oracle.prepare_weights(wg, wu, wd)
    ids = np.zeros((t, 1), np.int32)
    wts = np.ones((t, 1), np.float32)
    out = oracle.bf16_to_f32(oracle.moe_layer(x, ids, wts, weights))
    ref = _torch_ffn_fp64(x, wg[0], wu[0], wd[0]).numpy()
    err = np.max(np.abs(out - ref)) / np.max(np.abs(ref))
    assert err < 5e-3, err  # bf16 output rounding (2^-9 relative) dominates


def test_layer_fp64_shadow_bound_on_deepseek_shape():
    """At the real H=7168, I=2048 the oracle's fp32 result stays within the
    independent fp64 statement by far less than the 2e-2 parity bound."""
    rng = np.random.default_rng(10)
    t, hdim, idim = 3, 7168, 2048
    x = synth.bf16_bits_from_f32(rng.standard_normal((t, hdim)).astype(np.float32))
    wg = (0.02 * rng.standard_normal((1, idim, hdim))).astype(np.float32)
    wu = (0.02 * rng.standard_normal((1, idim, hdim))).astype(np.float32)
    wd = (0.02 * rng.standard_normal((1, hdim, idim))).astype(np.float32)
    weights = oracle.prepare_weights(wg, wu, wd)
    ids = np.zeros((t, 1), np.int32)
    wts = np.ones((t, 1), np.float32)
    _, inter = oracle.moe_layer(x, ids, wts, weights, want_intermediates=True)
    ref = _torch_ffn_fp64(x, wg[0], wu[0], wd[0]).numpy()
    err = np.max(np.abs(inter["y"] - ref)) / np.max(np.abs(ref))
    assert err < 2e-3, err


def test_token_permutation_permutes_output_rows():
    w, x, ids, wts, weights = _tiny_inputs()
    out = oracle.moe_layer(x, ids, wts, weights)
    perm = np.random.default_rng(11).permutation(x.shape[0])
    out_p = oracle.moe_layer(x[perm], ids[perm], wts[perm], weights)
    assert np.array_equal(out_p, out[perm])


def test_expert_relabelling_gives_identical_output():
    w, x, ids, wts, weights = _tiny_inputs()
    out = oracle.moe_layer(x, ids, wts, weights)
    relabel = np.random.default_rng(12).permutation(w.n_experts)  # old id -> new id
    inv = np.argsort(relabel)
    weights2 = tuple(m[inv] for m in weights)
    out2 = oracle.moe_layer(x, relabel[ids].astype(np.int32), wts, weights2)
    assert np.array_equal(out, out2)


def test_down_scales_times_power_of_two_scale_outputs_exactly():
    w, x, ids, wts, weights = _tiny_inputs()
    qg, sg, qu, su, qd, sd = weights
    _, i0 = oracle.moe_layer(x, ids, wts, weights, want_intermediates=True)
    for j in (-5, 3):
        w2 = (qg, sg, qu, su, qd, np.ldexp(sd, j).astype(np.float32))
        _, i1 = oracle.moe_layer(x, ids, wts, w2, want_intermediates=True)
        assert np.array_equal(i1["y"], np.ldexp(i0["y"], j).astype(np.float32))


def test_gate_and_up_are_not_swapped():
    """Swapping W_gate and W_up changes SiLU(g)*u into SiLU(u)*g."""
    w, x, ids, wts, weights = _tiny_inputs()
    qg, sg, qu, su, qd, sd = weights
    _, i0 = oracle.moe_layer(x, ids, wts, weights, want_intermediates=True)
    g, u = i0["g"], i0["u"]
    ref_h = (g.astype(np.float64) / (1 + np.exp(-g.astype(np.float64)))) * u
    assert np.max(np.abs(i0["h"] - ref_h)) <= 1e-6 * np.max(np.abs(ref_h))


def test_combine_special_cases():
    rng = np.random.default_rng(13)
    t, k, hdim = 6, 3, 256
    wts = rng.random((t, k)).astype(np.float32)
    ones = np.ones((t * k, hdim), np.float32)
    dest = rng.permutation(t * k).astype(np.int32)
    out = oracle.combine(ones, dest, wts)
    s = (wts[:, 0] + wts[:, 1]).astype(np.float32)
    s = (s + wts[:, 2]).astype(np.float32)
    ref = torch.from_numpy(s).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.all(out == ref[:, None])
    y = rng.standard_normal((t, hdim)).astype(np.float32)
    out1 = oracle.combine(y, np.arange(t, dtype=np.int32), np.ones((t, 1), np.float32))
    ref1 = torch.from_numpy(y).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(out1, ref1)


def test_tiny_config_layer_output_is_finite_and_nontrivial():
    w, x, ids, wts, weights = _tiny_inputs()
    out = oracle.bf16_to_f32(oracle.moe_layer(x, ids, wts, weights))
    assert out.shape == (w.tokens, w.hidden)
    assert np.all(np.isfinite(out)) and np.std(out) > 0


# ------------------------------------------------------------------- W8A16
def test_w8a16_matmul_exact_on_grid_with_power_of_two_scales():
    """bf16 small integers times small-integer e4m3 codes with 2^j block
    scales: exact at every step, equal to the fp64 double sum."""
    rng = np.random.default_rng(17)
    m, n, k = 3, 256, 384
    ints = np.array([-4, -3, -2, -1, 0, 1, 2, 3, 4], dtype=np.float32)
    a = rng.choice(ints, size=(m, k)) * np.float32(1.5)     # bf16-exact
    w = rng.choice(ints, size=(n, k))
    a_bits = synth.bf16_bits_from_f32(a)
    w_q = oracle.e4m3_encode(w)
    w_s = np.ldexp(1.0, rng.integers(-3, 4, size=(n // 128, k // 128))).astype(np.float32)
    got = oracle.block_scaled_matmul_w8a16(a_bits, w_q, w_s)
    ref = np.zeros((m, n))
    for i in range(m):
        for j in range(n):
            ref[i, j] = sum(float(np.dot(a[i, b * 128:(b + 1) * 128].astype(np.float64),
                                         w[j, b * 128:(b + 1) * 128].astype(np.float64))) * float(w_s[j // 128, b])
                            for b in range(k // 128))
    assert np.array_equal(got.astype(np.float64), ref)


def test_w8a16_matmul_close_to_fp64_dequantized_product():
    rng = np.random.default_rng(18)
    x = synth.bf16_bits_from_f32(rng.standard_normal((7, 512)).astype(np.float32))
    w = (0.02 * rng.standard_normal((256, 512))).astype(np.float32)
    w_q, w_s = oracle.quantize_weight(w)
    w_deq = torch.from_numpy(w_q).view(torch.float8_e4m3fn).double().numpy() \
        * np.kron(w_s.astype(np.float64), np.ones((128, 128)))
    xd = torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).double().numpy()
    ref = xd @ w_deq.T
    got = oracle.block_scaled_matmul_w8a16(x, w_q, w_s)
    assert np.max(np.abs(got - ref)) / np.max(np.abs(ref)) < 1e-6


def test_w8a16_single_expert_identity_against_independent_dense_ffn():
    """E = 1, k = 1, w = 1: bf16(FFN(x)) with bf16 activations, torch casts, fp64 GEMMs."""
    rng = np.random.default_rng(19)
    t, hdim, idim = 12, 384, 256
    x = synth.bf16_bits_from_f32(rng.standard_normal((t, hdim)).astype(np.float32))
    mats = [(0.02 * rng.standard_normal(s)).astype(np.float32) for s in ((1, idim, hdim), (1, idim, hdim),
                                                                         (1, hdim, idim))]
    weights = oracle.prepare_weights(*mats)
    out = oracle.bf16_to_f32(oracle.moe_layer_w8a16(x, np.zeros((t, 1), np.int32), np.ones((t, 1), np.float32),
                                                    weights))

    def deq(m32):
        n, k = m32.shape
        blk = torch.from_numpy(m32).reshape(n // 128, 128, k // 128, 128)
        s = blk.abs().amax(dim=(1, 3), keepdim=True) / torch.tensor(448.0)
        return ((blk / s).clamp(-448, 448).to(torch.float8_e4m3fn).double() * s.double()).reshape(n, k)

    xt = torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).double()
    g = xt @ deq(mats[0][0]).T
    u = xt @ deq(mats[1][0]).T
    h = (g * torch.sigmoid(g) * u).to(torch.bfloat16).double()
    ref = (h @ deq(mats[2][0]).T).numpy()
    err = np.max(np.abs(out - ref)) / np.max(np.abs(ref))
    assert err < 5e-3, err


def test_w8a16_and_w8a8_differ_by_the_activation_quantization_only():
    """With activations already on the e4m3 grid of their row scales (block
    amax 448, so qx = x exactly) and h likewise, W8A8 and W8A16 agree within
    fp32 rounding: the modes differ only in where the activations are rounded."""
    rng = np.random.default_rng(20)
    m, k, n = 4, 256, 128
    a = oracle.e4m3_decode(oracle.e4m3_encode((rng.standard_normal((m, k)) * 64).astype(np.float32)))
    a[:, 0] = 448.0
    a[:, 128] = 448.0
    a_bits = synth.bf16_bits_from_f32(a.astype(np.float32))   # e4m3 values are bf16-exact
    a_q, a_s = oracle.quantize_rows(a.astype(np.float32))
    assert np.all(a_s == 1.0)
    w_q, w_s = oracle.quantize_weight((0.02 * rng.standard_normal((n, k))).astype(np.float32))
    r8 = oracle.block_scaled_matmul(a_q, a_s, w_q, w_s)
    r16 = oracle.block_scaled_matmul_w8a16(a_bits, w_q, w_s)
    assert np.array_equal(r8, r16)
