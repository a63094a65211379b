"""Pins of the oracle's FP8 E4M3 decode/encode and block quantizer.

The oracle is checked against things other than itself: torch's
float8_e4m3fn type (an independent implementation of the OCP format), the
OCP landmark values in tests/golden/, exact midpoints and power-of-two
scaling invariants.
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _torch_decode_all():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    return codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()


def test_table_matches_torch_float8_e4m3fn_all_codes():
    ref = _torch_decode_all()
    tab = oracle.E4M3_TABLE
    nan_ref = np.isnan(ref)
    assert np.array_equal(np.isnan(tab), nan_ref)
    assert np.array_equal(tab[~nan_ref], ref[~nan_ref])
    # signs of zero agree as well
    assert np.array_equal(np.signbit(tab[~nan_ref]), np.signbit(ref[~nan_ref]))
    assert nan_ref.sum() == 2  # only S.1111.111


def test_table_golden_landmarks():
    rows = [ln.split() for ln in open(os.path.join(GOLDEN, "e4m3_landmarks.txt"))
            if ln.strip() and not ln.startswith("#")]
    assert len(rows) >= 15
    for code_s, val_s in rows:
        code = int(code_s, 16)
        got = oracle.E4M3_TABLE[code]
        if val_s == "nan":
            assert math.isnan(got), code_s
        else:
            want = float(val_s)
            assert got == want and math.copysign(1, got) == math.copysign(1, want), code_s


def test_encode_round_trips_every_finite_code():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], dtype=np.uint8)
    vals = oracle.e4m3_decode(codes).astype(np.float32)
    assert np.array_equal(oracle.e4m3_encode(vals), codes)


def test_encode_midpoints_go_to_even_and_neighbours_to_nearest():
    pos = oracle.E4M3_TABLE[:0x7F]
    for c in range(0x7E):
        lo, hi = pos[c], pos[c + 1]
        mid = np.float32((lo + hi) / 2)           # exact: midpoints need <= 5 bits
        assert float(mid) == (lo + hi) / 2
        even = c if c % 2 == 0 else c + 1
        assert oracle.e4m3_encode(np.array([mid]))[0] == even, hex(c)
        assert oracle.e4m3_encode(np.array([-mid]))[0] == (even | 0x80)
        below = np.nextafter(mid, np.float32(-np.inf))
        above = np.nextafter(mid, np.float32(np.inf))
        assert oracle.e4m3_encode(np.array([below]))[0] == c
        assert oracle.e4m3_encode(np.array([above]))[0] == c + 1


def test_encode_saturates_and_keeps_sign_of_zero():
    v = np.array([448.0, 449.0, 464.0, 1e6, np.inf, -470.0, 0.0, -0.0, -1e-30, 1e-30],
                 dtype=np.float32)
    got = oracle.e4m3_encode(v)
    assert list(got) == [0x7E, 0x7E, 0x7E, 0x7E, 0x7E, 0xFE, 0x00, 0x80, 0x80, 0x00]


def test_encode_matches_torch_on_random_values():
    rng = np.random.default_rng(1)
    mant = rng.uniform(-1, 1, 200000)
    expo = rng.integers(-14, 10, 200000)
    v = np.ldexp(mant, expo).astype(np.float32)
    v = np.clip(v, -448, 448)
    ref = torch.from_numpy(v).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(oracle.e4m3_encode(v), ref)


def _torch_quantize_rows(x):
    """Independent statement of the activation quantizer using torch's fp8 cast."""
    t = torch.from_numpy(x).reshape(x.shape[0], -1, 128)
    a = t.abs().amax(dim=2, keepdim=True)
    s = a / torch.tensor(448.0, dtype=torch.float32)
    v = torch.where(s > 0, t / torch.where(s > 0, s, torch.ones_like(s)), t)
    q = v.clamp(-448, 448).to(torch.float8_e4m3fn).view(torch.uint8)
    return q.reshape(x.shape).numpy(), s[..., 0].numpy()


def test_quantize_rows_matches_independent_torch_statement():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((64, 1024)).astype(np.float32)
    x[3, 128:256] = 0.0                      # zero block
    x[4, 0:128] = -0.0
    x[5, 256:384] *= 1e-30                   # subnormal-ish block
    q, s = oracle.quantize_rows(x)
    q_ref, s_ref = _torch_quantize_rows(x)
    assert np.array_equal(s, s_ref)
    assert np.array_equal(q, q_ref)
    assert np.all(s[3, 1] == 0) and np.all(q[3, 128:256] == 0x00)
    assert np.all(q[4, 0:128] == 0x80)


def test_quantize_rows_power_of_two_invariance():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((16, 512)).astype(np.float32)
    q0, s0 = oracle.quantize_rows(x)
    for j in (-20, -3, 1, 7, 30):
        q, s = oracle.quantize_rows(np.ldexp(x, j).astype(np.float32))
        assert np.array_equal(q, q0)
        assert np.array_equal(s, np.ldexp(s0, j).astype(np.float32))


def test_quantize_rows_block_with_amax_448_is_lossless():
    rng = np.random.default_rng(4)
    codes = rng.integers(0, 0x7F, size=(8, 256)).astype(np.uint8)
    codes |= (rng.integers(0, 2, size=codes.shape).astype(np.uint8) << 7)
    codes[:, 0] = 0x7E
    codes[:, 128] = 0xFE                     # |-448| is the amax of block 1
    x = oracle.e4m3_decode(codes).astype(np.float32)
    q, s = oracle.quantize_rows(x)
    assert np.all(s == 1.0)
    assert np.array_equal(q, codes)


def test_quant_act_takes_bf16_bits_exactly():
    x = np.array([[1.0, -2.5, 3.0e-3] + [0.0] * 125], dtype=np.float32)
    bits = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    xf = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).float().numpy()
    q1, s1 = oracle.quant_act(bits)
    q2, s2 = oracle.quantize_rows(xf)
    assert np.array_equal(q1, q2) and np.array_equal(s1, s2)


def test_bf16_conversions_match_torch():
    rng = np.random.default_rng(5)
    x = (rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))).astype(np.float32)
    x[:4] = [0.0, -0.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8]   # exact ties
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle.f32_to_bf16(x), ref)
    back = torch.from_numpy(ref.view(np.int16)).view(torch.bfloat16).float().numpy()
    assert np.array_equal(oracle.bf16_to_f32(ref), back)


def test_quantize_weight_blocks_by_brute_force():
    rng = np.random.default_rng(6)
    w = (0.02 * rng.standard_normal((256, 384))).astype(np.float32)
    w[128:256, 0:128] *= 50.0                # one block with a different range
    q, s = oracle.quantize_weight(w)
    assert s.shape == (2, 3)
    for bi in range(2):
        for bj in range(3):
            blk = w[bi * 128:(bi + 1) * 128, bj * 128:(bj + 1) * 128]
            amax = float(np.max(np.abs(blk)))
            assert s[bi, bj] == np.float32(np.float32(amax) / np.float32(448))
            v = torch.from_numpy(blk) / torch.tensor(float(s[bi, bj]), dtype=torch.float32)
            ref = v.clamp(-448, 448).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
            assert np.array_equal(q[bi * 128:(bi + 1) * 128, bj * 128:(bj + 1) * 128], ref)


def test_quantize_rejects_ragged_k():
    with pytest.raises(ValueError):
        oracle.quantize_rows(np.zeros((2, 100), np.float32))
    with pytest.raises(ValueError):
        oracle.quantize_weight(np.zeros((100, 128), np.float32))
