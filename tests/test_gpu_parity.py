"""GPU parity: the HIP library through its C ABI against the CPU oracle.

Bar: bit-exact for quantized activations (codes and scales), weight
quantization, permutation indices and combine given the same expert rows;
max|out - ref| / max|ref| <= 2e-2 for the bf16 layer output (and for the
fp32 expert rows), at sizes the oracle finishes in seconds (several tiles
and a ragged tail) and on sampled tokens of the full DeepSeek-V3 shapes.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_cases import (bf16_dev, bits_to_f32, generated_layer_gpu, log, oracle_expert_weights,
                       oracle_tokens, pack_reference, quantize_weights_gpu, rel_err, require_gpu, to_dev)

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.fixture(scope="module")
def moe():
    return require_gpu()


# ------------------------------------------------------------ quantization
def _crafted_activation_rows():
    """128-wide blocks hitting ties, zeros, signed zeros, subnormals, huge ranges."""
    pos = oracle.E4M3_TABLE[:0x7F]
    mids = ((pos[:-1] + pos[1:]) / 2).astype(np.float32)   # exact in bf16 (<= 5 bits)
    vals = np.concatenate([mids, -mids, pos.astype(np.float32)])
    n = (len(vals) + 126) // 127
    base = np.zeros((n, 128), np.float32)
    base[:, 0] = 448.0                                       # amax 448 -> s = 1 exactly
    flat = np.zeros(n * 127, np.float32)
    flat[: len(vals)] = vals
    base[:, 1:] = flat.reshape(n, 127)
    rows = [base]
    for j in (-30, -7, 9, 60):
        rows.append(np.ldexp(base, j).astype(np.float32))   # same codes, s = 2^j
    rows.append(np.zeros((1, 128), np.float32))
    rows.append(-np.zeros((1, 128), np.float32))
    rows.append(np.ldexp(np.arange(1, 129, dtype=np.float32), -140)[None, :])  # bf16 subnormals
    big = np.full((1, 128), 1.0e-3, np.float32)
    big[0, 0] = 3.0e38
    rows.append(big)
    return np.concatenate(rows).astype(np.float32)


def test_quant_act_crafted_bit_exact(moe):
    x32 = _crafted_activation_rows()
    x32 = np.concatenate([x32, np.random.default_rng(0).standard_normal((x32.shape[0], 128)).astype(np.float32)],
                         axis=1)  # two blocks per row: crafted + random
    bits = synth.bf16_bits_from_f32(x32)
    q_ref, s_ref = oracle.quant_act(bits)
    q = torch.empty(bits.shape, dtype=torch.uint8, device="cuda")
    s = torch.empty((bits.shape[0], bits.shape[1] // 128), dtype=torch.float32, device="cuda")
    moe.moe_quant_act(bf16_dev(bits), q, s)
    torch.cuda.synchronize()
    assert np.array_equal(s.cpu().numpy().view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(q.cpu().numpy(), q_ref)


def test_quant_rows_f32_neighbours_of_ties_bit_exact(moe):
    pos = oracle.E4M3_TABLE[:0x7F]
    mids = ((pos[:-1] + pos[1:]) / 2).astype(np.float32)
    vals = np.concatenate([mids, np.nextafter(mids, np.float32(0)), np.nextafter(mids, np.float32(1e9)),
                           -mids, pos.astype(np.float32)])
    n = (len(vals) + 126) // 127
    x = np.zeros((n, 128), np.float32)
    x[:, 0] = 448.0
    flat = x[:, 1:].reshape(-1)
    flat[: len(vals)] = vals
    x[:, 1:] = flat.reshape(n, 127)
    q_ref, s_ref = oracle.quantize_rows(x)
    q = torch.empty(x.shape, dtype=torch.uint8, device="cuda")
    s = torch.empty((n, 1), dtype=torch.float32, device="cuda")
    moe.moe_quant_rows_f32(to_dev(x), q, s)
    torch.cuda.synchronize()
    assert np.array_equal(s.cpu().numpy(), s_ref)
    assert np.array_equal(q.cpu().numpy(), q_ref)


def _band(lo, hi):
    """Every fp32 value in [lo, hi)."""
    a, b = np.float32(lo).view(np.uint32), np.float32(hi).view(np.uint32)
    return np.arange(a, b, dtype=np.uint32).view(np.float32)


def test_quant_rows_f32_every_value_of_three_bands_bit_exact(moe):
    """Every fp32 value of [2^-8, 2^-5) (across the e4m3 subnormal/normal
    boundary at 2^-6), of [1, 2) and of [256, 448], and the negatives of
    every 16th of them, quantized with scale 1 (each row holds 448): the
    library's codes against the oracle's nearest-value search, value by value
    (40M values)."""
    vals = np.concatenate([_band(2.0 ** -8, 2.0 ** -5), _band(1.0, 2.0), _band(256.0, 448.0), np.float32([448.0])])
    vals = np.concatenate([vals, -vals[::16]])
    n = (len(vals) + 126) // 127
    x = np.zeros((n, 128), np.float32)
    x[:, 0] = 448.0
    flat = np.zeros(n * 127, np.float32)
    flat[: len(vals)] = vals
    x[:, 1:] = flat.reshape(n, 127)
    log(f"quant_rows_f32 on {len(vals)} band values")
    q_ref, s_ref = oracle.quantize_rows(x)
    assert np.all(s_ref == 1.0)
    q = torch.empty(x.shape, dtype=torch.uint8, device="cuda")
    s = torch.empty((n, 1), dtype=torch.float32, device="cuda")
    moe.moe_quant_rows_f32(to_dev(x), q, s)
    torch.cuda.synchronize()
    assert np.array_equal(s.cpu().numpy(), s_ref)
    qc = q.cpu().numpy()
    bad = np.flatnonzero(qc.reshape(-1) != q_ref.reshape(-1))
    assert bad.size == 0, (bad.size, x.reshape(-1)[bad[:8]], qc.reshape(-1)[bad[:8]], q_ref.reshape(-1)[bad[:8]])


def test_quant_rows_f32_tiny_scales_bit_exact(moe):
    """Blocks whose scale amax / 448 lies on either side of 2^-90, where the
    quantizer switches from the reciprocal-and-correction quotient to the
    division, down to subnormal inputs, and an all-zero block: codes and
    scales against the oracle, bit for bit."""
    rng = np.random.default_rng(9)
    amaxes = [448 * 2.0 ** e for e in (-80, -89, -90, -91, -95, -110, -125)] + [1e-38, 3e-42, 0.0]
    rows = []
    for a in amaxes:
        for _ in range(4):
            v = (rng.uniform(-1.0, 1.0, 128) * a).astype(np.float32)
            if a > 0:
                v[rng.integers(0, 128)] = np.float32(a)
            rows.append(v)
    x = np.stack(rows).astype(np.float32)
    q_ref, s_ref = oracle.quantize_rows(x)
    q = torch.empty(x.shape, dtype=torch.uint8, device="cuda")
    s = torch.empty((x.shape[0], 1), dtype=torch.float32, device="cuda")
    moe.moe_quant_rows_f32(to_dev(x), q, s)
    torch.cuda.synchronize()
    assert np.array_equal(s.cpu().numpy().view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(q.cpu().numpy(), q_ref)


@pytest.mark.parametrize("rows,cols", [(1, 128), (37, 1024), (4096, 7168)])
def test_quant_act_random_bit_exact(moe, rows, cols):
    rng = np.random.default_rng(rows)
    bits = synth.bf16_bits_from_f32(rng.standard_normal((rows, cols)).astype(np.float32) * 3)
    q_ref, s_ref = oracle.quant_act(bits)
    q = torch.empty((rows, cols), dtype=torch.uint8, device="cuda")
    s = torch.empty((rows, cols // 128), dtype=torch.float32, device="cuda")
    moe.moe_quant_act(bf16_dev(bits), q, s)
    torch.cuda.synchronize()
    assert np.array_equal(s.cpu().numpy(), s_ref)
    assert np.array_equal(q.cpu().numpy(), q_ref)


def test_quant_weight_bit_exact(moe):
    rng = np.random.default_rng(3)
    w = (0.02 * rng.standard_normal((3, 256, 384))).astype(np.float32)
    w[1, 128:, :128] = 0.0
    w[2, :128, 128:256] *= 1e4
    q = torch.empty(w.shape, dtype=torch.uint8, device="cuda")
    s = torch.empty((3, 2, 3), dtype=torch.float32, device="cuda")
    moe.moe_quant_weight(to_dev(w), q, s)
    torch.cuda.synchronize()
    for m in range(3):
        q_ref, s_ref = oracle.quantize_weight(w[m])
        assert np.array_equal(s.cpu().numpy()[m], s_ref)
        assert np.array_equal(q.cpu().numpy()[m], q_ref)


def test_quant_weight_deepseek_matrix_bit_exact(moe):
    w = synth.WORKLOADS["decode1"]
    f = synth.expert_weight_device(w, 0, 17, 2)          # one W_down [7168, 2048]
    q = torch.empty(f.shape, dtype=torch.uint8, device="cuda")
    s = torch.empty((f.shape[0] // 128, f.shape[1] // 128), dtype=torch.float32, device="cuda")
    moe.moe_quant_weight(f, q, s)
    torch.cuda.synchronize()
    q_ref, s_ref = oracle.quantize_weight(f.cpu().numpy())
    assert np.array_equal(s.cpu().numpy(), s_ref)
    assert np.array_equal(q.cpu().numpy(), q_ref)


@pytest.mark.parametrize("n,rows,cols", [(1, 16, 128), (3, 32, 384), (2, 256, 256), (1, 2048, 7168)])
def test_pack_weight_matches_layout_definition(moe, n, rows, cols):
    """moe_pack_weight is a pure byte permutation; every byte lands where the layout definition puts it."""
    rng = np.random.default_rng(rows + cols)
    q = rng.integers(0, 256, size=(n, rows, cols), dtype=np.uint8)
    dq = to_dev(q)
    packed = torch.full_like(dq, 0xA5)
    moe.moe_pack_weight(dq, packed)
    torch.cuda.synchronize()
    assert np.array_equal(packed.cpu().numpy(), pack_reference(q))


# --------------------------------------------------------------- permute
def _run_permute(moe, ids, n_exp, status=False):
    t, k = ids.shape
    d_ids = to_dev(ids.astype(np.int32))
    off = torch.full((n_exp + 1,), -7, dtype=torch.int32, device="cuda")
    src = torch.full((t * k,), -7, dtype=torch.int32, device="cuda")
    dst = torch.full((t * k,), -7, dtype=torch.int32, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.empty(max(1, moe.moe_permute_workspace(t, k, n_exp)), dtype=torch.uint8, device="cuda")
    moe.moe_permute(d_ids, n_exp, off, src, dst, st, ws)
    torch.cuda.synchronize()
    return off.cpu().numpy(), src.cpu().numpy(), dst.cpu().numpy(), int(st.item())


@pytest.mark.parametrize("name,t", [("tiny", 16), ("decode1", 1), ("decode4", 4), ("decode64_zipf", 64),
                                    ("tiny", 0), ("tiny", 255), ("tiny", 256), ("tiny", 257),
                                    ("prefill8k", 8192), ("prefill32k_streamed", 32768)])
def test_permute_bit_exact(moe, name, t):
    w = synth.WORKLOADS[name]
    ids, _ = synth.routing(w, t) if t else (np.zeros((0, w.topk), np.int32), None)
    log(f"permute {name} T={t}")
    off, src, dst, st = _run_permute(moe, ids, w.n_experts)
    r_off, r_src, r_dst = oracle.permute(ids, w.n_experts)
    assert st == 0
    assert np.array_equal(off, r_off)
    assert np.array_equal(src, r_src)
    assert np.array_equal(dst, r_dst)


def test_permute_wide_topk_and_many_experts(moe):
    rng = np.random.default_rng(4)
    ids = np.stack([rng.choice(1024, 32, replace=False) for _ in range(600)]).astype(np.int32)
    off, src, dst, st = _run_permute(moe, ids, 1024)
    r_off, r_src, r_dst = oracle.permute(ids, 1024)
    assert st == 0 and np.array_equal(off, r_off) and np.array_equal(src, r_src) and np.array_equal(dst, r_dst)


@pytest.mark.parametrize("t,k,e", [(8, 8, 256), (64, 1, 16), (65, 1, 16), (2, 32, 1024), (3, 32, 1024)],
                         ids=lambda v: str(v))
def test_permute_small_batch_boundaries(moe, t, k, e):
    """Around 64 slots, where the one-workgroup sort switches between its
    pairwise-count form (up to 64 slots) and its token-mask form."""
    rng = np.random.default_rng(t * 100 + k)
    ids = np.stack([rng.choice(e, k, replace=False) for _ in range(t)]).astype(np.int32)
    off, src, dst, st = _run_permute(moe, ids, e)
    r_off, r_src, r_dst = oracle.permute(ids, e)
    assert st == 0 and np.array_equal(off, r_off) and np.array_equal(src, r_src) and np.array_equal(dst, r_dst)


@pytest.mark.parametrize("t", [5, 21, 22, 80, 700])
def test_permute_reports_bad_ids_and_stays_a_bijection(moe, t):
    rng = np.random.default_rng(5)
    ids = np.stack([rng.choice(8, 3, replace=False) for _ in range(t)]).astype(np.int32)
    ids[1, 2] = 8          # out of range
    ids[3, 1] = ids[3, 0]  # duplicate
    off, src, dst, st = _run_permute(moe, ids, 8)
    assert st & moe.MOE_DEV_BAD_EXPERT_ID and st & moe.MOE_DEV_DUP_EXPERT_ID
    n = t * 3
    assert sorted(src.tolist()) == list(range(n))
    assert np.array_equal(dst[src], np.arange(n))
    assert off[-1] == n - 2
    # the valid slots keep the oracle order of the valid ids
    valid = np.ones(n, bool)
    valid[1 * 3 + 2] = False
    valid[3 * 3 + 1] = False
    assert np.all(src[off[-1]:] == np.flatnonzero(~valid))
    flat = ids.reshape(-1)
    good = np.flatnonzero(valid)
    assert np.array_equal(src[:off[-1]], good[np.argsort(flat[good], kind="stable")])
    assert np.array_equal(off[:-1], np.searchsorted(np.sort(flat[good]), np.arange(8)))


# --------------------------------------------------------------- combine
@pytest.mark.parametrize("t,k,h", [(1, 8, 7168), (37, 2, 256), (300, 8, 1024), (5, 9, 512), (3, 17, 256), (4, 32, 128)])
def test_combine_bit_exact(moe, t, k, h):
    rng = np.random.default_rng(t)
    y = rng.standard_normal((t * k, h)).astype(np.float32)
    dest = rng.permutation(t * k).astype(np.int32)
    wts = rng.random((t, k)).astype(np.float32)
    out = torch.empty((t, h), dtype=torch.int16, device="cuda")
    moe.moe_combine(to_dev(y), to_dev(dest), to_dev(wts), out)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy().view(np.uint16), oracle.combine(y, dest, wts))


# ----------------------------------------------------------- whole layer
SMALL_CASES = [
    # (hidden, inter, experts, topk, tokens, routing)
    (256, 128, 8, 2, 16, "uniform"),     # the tiny layer
    (1024, 512, 16, 4, 37, "uniform"),   # several tiles, ragged rows
    (512, 256, 8, 2, 300, "zipf"),       # prefill tiles with ragged tails, skewed
    (256, 128, 4, 4, 5, "uniform"),      # k == E
    (768, 384, 32, 8, 64, "zipf"),       # decode limit
]


def _small_layer(case, seed=0):
    h, i, e, k, t, routing = case
    rule = "softmax" if (h, i, e, k, t) == (256, 128, 8, 2, 16) else "sigmoid"
    w = synth.Workload("case", h, i, e, k, t, routing, 1.0 if routing == "zipf" else 0.0, rule, seed=seed)
    x = synth.activations(w)
    ids, wts = synth.routing(w)
    wg, wu, wd = synth.weights_host(w)
    return w, x, ids, wts, (wg, wu, wd)


def _gpu_layer(moe, w, x, ids, wts, dweights, regime):
    buf = moe.MoELayerBuffers(w.hidden, w.inter, w.n_experts, w.topk, w.tokens, regime)
    moe.run_layer(buf, bf16_dev(x), to_dev(ids), to_dev(wts), dweights)
    torch.cuda.synchronize()
    return buf


@pytest.mark.parametrize("case", SMALL_CASES, ids=lambda c: "x".join(map(str, c[:5])) + c[5])
@pytest.mark.parametrize("regime", ["decode", "prefill"])
def test_layer_parity_small(moe, case, regime):
    w, x, ids, wts, (wg, wu, wd) = _small_layer(case)
    rg = moe.MOE_REGIME_DECODE if regime == "decode" else moe.MOE_REGIME_PREFILL
    if rg == moe.MOE_REGIME_DECODE and w.tokens > moe.MOE_DECODE_MAX_TOKENS:
        pytest.skip("decode regime is limited to 64 tokens")
    log(f"layer {case} {regime}")
    ow = oracle.prepare_weights(wg, wu, wd)
    dweights = quantize_weights_gpu(moe, wg, wu, wd)
    for j, (dq, rq) in enumerate(zip(dweights, ow)):
        # codes are packed into operand tiles on the device, scales stay row-major
        assert np.array_equal(dq.cpu().numpy(), pack_reference(rq) if j % 2 == 0 else rq)
    ref, inter = oracle.moe_layer(x, ids, wts, ow, want_intermediates=True)
    buf = _gpu_layer(moe, w, x, ids, wts, dweights, rg)
    assert int(buf.dev_status.item()) == 0
    assert np.array_equal(buf.qx.cpu().numpy(), inter["qx"])
    assert np.array_equal(buf.sx.cpu().numpy(), inter["sx"])
    assert np.array_equal(buf.expert_offsets.cpu().numpy(), inter["offsets"])
    assert np.array_equal(buf.sorted_src.cpu().numpy(), inter["sorted_src"])
    assert np.array_equal(buf.dest_row.cpu().numpy(), inter["dest_row"])
    y_err = rel_err(buf.y_rows.cpu().numpy(), inter["y"])
    out_err = rel_err(bits_to_f32(buf.out), oracle.bf16_to_f32(ref))
    log(f"  y_rows rel err {y_err:.3e}  out rel err {out_err:.3e}")
    assert y_err <= TOL
    assert out_err <= TOL


def test_prefill_tail_tiles_of_every_operand_count(moe):
    """Expert row counts whose 128-row tiles end with 1-32, 33-64, 65-96 and
    97-128 rows, so the prefill K loop runs with 1, 2, 3 and 4 live 32-row
    operands (and full tiles before the tails)."""
    counts = [2, 32, 33, 64, 65, 96, 225, 257]
    k = 2
    t = sum(counts) // k
    w = synth.Workload("tails", 512, 256, len(counts), k, t, "uniform", 0.0, "sigmoid", seed=5)
    x = synth.activations(w)
    _, wts = synth.routing(w)
    # expert e fills counts[e] slots; slot t + j*T goes to token t, choice j
    # (distinct experts per token since every count is at most T)
    slots = np.repeat(np.arange(len(counts), dtype=np.int32), counts)
    ids = np.ascontiguousarray(slots.reshape(k, t).T)
    assert all(len(set(r)) == k for r in ids.tolist())
    wg, wu, wd = synth.weights_host(w)
    ow = oracle.prepare_weights(wg, wu, wd)
    dweights = quantize_weights_gpu(moe, wg, wu, wd)
    ref, inter = oracle.moe_layer(x, ids, wts, ow, want_intermediates=True)
    assert np.diff(inter["offsets"]).tolist() == counts
    buf = _gpu_layer(moe, w, x, ids, wts, dweights, moe.MOE_REGIME_PREFILL)
    assert int(buf.dev_status.item()) == 0
    y_err = rel_err(buf.y_rows.cpu().numpy(), inter["y"])
    out_err = rel_err(bits_to_f32(buf.out), oracle.bf16_to_f32(ref))
    log(f"  tails: y_rows rel err {y_err:.3e}  out rel err {out_err:.3e}")
    assert y_err <= TOL
    assert out_err <= TOL
    # every expert row is checked on its own too, so a skipped operand cannot
    # hide behind the global maximum
    y = buf.y_rows.cpu().numpy().astype(np.float64)
    for e in range(len(counts)):
        o0, o1 = inter["offsets"][e], inter["offsets"][e + 1]
        assert rel_err(y[o0:o1], inter["y"][o0:o1]) <= TOL, e


@pytest.mark.parametrize("w8a16", [False, True])
def test_decode_row_count_classes(moe, w8a16):
    """Decode launches one kernel per expert row-count class (1-16, 17-32,
    33+ rows).  Experts with exactly 1, 16, 17, 32, 33 and 64 rows (and one
    empty expert) must each be computed once, by the right class."""
    counts = [64, 33, 32, 17, 16, 1, 0, 29]  # 192 slots = 64 tokens x 3
    k, t = 3, 64
    w = synth.Workload("classes", 512, 256, len(counts), k, t, "uniform", 0.0, "sigmoid", seed=7)
    x = synth.activations(w)
    _, wts = synth.routing(w)
    slots = np.repeat(np.arange(len(counts), dtype=np.int32), counts)
    ids = np.ascontiguousarray(slots.reshape(k, t).T)  # slot t + j*T -> token t, choice j
    assert all(len(set(r)) == k for r in ids.tolist())
    wg, wu, wd = synth.weights_host(w)
    ow = oracle.prepare_weights(wg, wu, wd)
    dweights = quantize_weights_gpu(moe, wg, wu, wd)
    buf = moe.MoELayerBuffers(w.hidden, w.inter, w.n_experts, w.topk, w.tokens, moe.MOE_REGIME_DECODE, w8a16=w8a16)
    moe.run_layer(buf, bf16_dev(x), to_dev(ids), to_dev(wts), dweights)
    torch.cuda.synchronize()
    assert int(buf.dev_status.item()) == 0
    if w8a16:
        ref, inter = oracle.moe_layer_w8a16(x, ids, wts, ow), None
    else:
        ref, inter = oracle.moe_layer(x, ids, wts, ow, want_intermediates=True)
        assert np.diff(inter["offsets"]).tolist() == counts
        y = buf.y_rows.cpu().numpy().astype(np.float64)
        for e in range(len(counts)):  # every expert's rows on their own
            o0, o1 = inter["offsets"][e], inter["offsets"][e + 1]
            if o1 > o0:
                assert rel_err(y[o0:o1], inter["y"][o0:o1]) <= TOL, e
    err = rel_err(bits_to_f32(buf.out), oracle.bf16_to_f32(ref))
    log(f"  row classes (w8a16={w8a16}): out rel err {err:.3e}")
    assert err <= TOL


@pytest.mark.parametrize("case", SMALL_CASES[:3], ids=lambda c: "x".join(map(str, c[:5])))
def test_decode_and_prefill_kernels_agree(moe, case):
    w, x, ids, wts, (wg, wu, wd) = _small_layer(case, seed=3)
    if w.tokens > moe.MOE_DECODE_MAX_TOKENS:
        w = w.with_tokens(64)
        x, (ids, wts) = x[:64], (ids[:64], wts[:64])
    dweights = quantize_weights_gpu(moe, wg, wu, wd)
    a = _gpu_layer(moe, w, x, ids, wts, dweights, moe.MOE_REGIME_DECODE)
    b = _gpu_layer(moe, w, x, ids, wts, dweights, moe.MOE_REGIME_PREFILL)
    assert rel_err(bits_to_f32(a.out), bits_to_f32(b.out).astype(np.float64)) <= TOL


def test_layer_is_deterministic(moe):
    w, x, ids, wts, (wg, wu, wd) = _small_layer(SMALL_CASES[2], seed=4)
    dweights = quantize_weights_gpu(moe, wg, wu, wd)
    outs = [_gpu_layer(moe, w, x, ids, wts, dweights, moe.MOE_REGIME_PREFILL).out.cpu().numpy()
            for _ in range(2)]
    assert np.array_equal(outs[0], outs[1])


def test_zero_tokens_is_a_no_op(moe):
    w, x, ids, wts, (wg, wu, wd) = _small_layer(SMALL_CASES[0])
    dweights = quantize_weights_gpu(moe, wg, wu, wd)
    w0 = w.with_tokens(0)
    buf = _gpu_layer(moe, w0, x[:0], ids[:0], wts[:0], dweights, moe.MOE_REGIME_AUTO)
    assert buf.expert_offsets.cpu().numpy().tolist() == [0] * (w.n_experts + 1)


# ------------------------------------------------- full DeepSeek-V3 shapes
@pytest.fixture(scope="module")
def deepseek_layer(moe):
    w = synth.WORKLOADS["decode1"]
    log("generating the full DeepSeek-V3 expert layer on the GPU")
    return generated_layer_gpu(moe, w, layer=0)


@pytest.mark.parametrize("name,sample", [("decode1", [0]), ("decode4", [0, 3]), ("decode64_zipf", [5, 63]),
                                         ("prefill8k", [0, 8191])])
def test_deepseek_layer_sampled_tokens(moe, deepseek_layer, name, sample):
    w = synth.WORKLOADS[name]
    log(f"deepseek {name} T={w.tokens}")
    x = synth.activations(w)
    ids, wts = synth.routing(w)
    buf = _gpu_layer(moe, w, x, ids, wts, deepseek_layer, moe.MOE_REGIME_AUTO)
    assert int(buf.dev_status.item()) == 0
    r_off, r_src, r_dst = oracle.permute(ids, w.n_experts)
    assert np.array_equal(buf.expert_offsets.cpu().numpy(), r_off)
    assert np.array_equal(buf.dest_row.cpu().numpy(), r_dst)
    qx_ref, sx_ref = oracle.quant_act(x[sample])
    assert np.array_equal(buf.qx.cpu().numpy()[sample], qx_ref)
    assert np.array_equal(buf.sx.cpu().numpy()[sample], sx_ref)
    experts = sorted(set(ids[sample].reshape(-1).tolist()))
    ow = oracle_expert_weights(w, experts)
    ref = oracle_tokens(x, ids, wts, sample, ow)
    got = bits_to_f32(buf.out)[sample]
    err = rel_err(got, oracle.bf16_to_f32(ref))
    log(f"  sampled tokens {sample}: out rel err {err:.3e}")
    assert err <= TOL
    out_all = bits_to_f32(buf.out)
    assert np.all(np.isfinite(out_all))
