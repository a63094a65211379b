"""GPU: the activation quantizer against the oracle over every fp32 value of
its range at unit scale, and over the rounding boundaries of 62 scales.

* Every fp32 value in [0, 448] (the bit patterns 0 .. 0x43E00000, 1.14e9
  values) and a seeded sample of 2^24 negative values, as rows of 128 whose
  first entry is 448 (so amax / 448 = 1 exactly and x / s = x): the codes
  of moe_quant_rows_f32 against oracle.e4m3_encode, bit for bit.  This
  covers the library's fp32 -> e4m3 conversion (the hardware conversion of
  the value clamped to +-448) on every input it can see at unit scale.
* 62 scales s = fl32(amax / 448) with amax from 2^-21 to 2^19 (41 binades
  with an all-ones mantissa and 21 seeded mantissas): at each scale, the
  values x whose quotient x / s lies on, and 1-3 ulps on both sides of,
  every e4m3 rounding midpoint and every e4m3 value, the quotients from
  2^-13 to 2^-9 around the smallest subnormal, and 2^16 seeded values in
  [-amax, amax]: codes and scales of moe_quant_rows_f32 against
  oracle.quantize_rows, whose quotient is numpy's correctly rounded fp32
  division.  The library forms the quotient from the block's reciprocal
  with one correction step; this checks that it equals the division on the
  values where rounding decides the code.

Cost: about 5 GB of GPU memory traffic and 1.2e9 oracle encodings on the
host (tens of seconds on 16 cores).
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_cases import log, require_gpu, to_dev

pytestmark = pytest.mark.gpu

CHUNK_ROWS = 1 << 19          # 2^19 rows x 127 values per GPU call
LAST = 0x43E00000             # bit pattern of 448.0


@pytest.fixture(scope="module")
def moe():
    return require_gpu()


def _gpu_codes(moe, x_rows):
    n = x_rows.shape[0]
    q = torch.empty((n, 128), dtype=torch.uint8, device="cuda")
    s = torch.empty((n, 1), dtype=torch.float32, device="cuda")
    moe.moe_quant_rows_f32(x_rows, q, s)
    torch.cuda.synchronize()
    return q, s


def test_every_fp32_value_up_to_448_at_unit_scale(moe):
    total = LAST + 1
    per = 127
    n_rows = (total + per - 1) // per
    done = 0
    for r0 in range(0, n_rows, CHUNK_ROWS):
        r1 = min(n_rows, r0 + CHUNK_ROWS)
        b0, b1 = r0 * per, min(total, r1 * per)
        bits = torch.arange(b0, b0 + (r1 - r0) * per, dtype=torch.int64, device="cuda")
        bits = torch.where(bits <= LAST, bits, torch.zeros_like(bits)).to(torch.int32)   # pad with +0
        vals = bits.view(torch.float32).view(r1 - r0, per)
        rows = torch.cat([torch.full((r1 - r0, 1), 448.0, device="cuda"), vals], dim=1).contiguous()
        q, s = _gpu_codes(moe, rows)
        assert bool(torch.all(s == 1.0))
        got = q[:, 1:].reshape(-1)[: b1 - b0].cpu().numpy()
        ref_vals = np.arange(b0, b1, dtype=np.uint32).view(np.float32)
        ref = oracle.e4m3_encode(ref_vals)
        bad = np.nonzero(got != ref)[0]
        assert bad.size == 0, (f"bits {b0 + int(bad[0]):#x}: gpu {got[bad[0]]:#04x} oracle {ref[bad[0]]:#04x}")
        done += b1 - b0
        if (r0 // CHUNK_ROWS) % 4 == 0:
            log(f"  unit scale: {done} of {total} values checked")
    assert done == total


def test_sampled_negative_values_at_unit_scale(moe):
    rng = np.random.default_rng(11)
    bits = rng.integers(0x80000000, 0x80000000 + LAST + 1, size=(1 << 24) // 127 * 127, dtype=np.uint64)
    vals = bits.astype(np.uint32).view(np.float32).reshape(-1, 127)
    rows = np.concatenate([np.full((vals.shape[0], 1), 448.0, np.float32), vals], axis=1)
    q, s = _gpu_codes(moe, to_dev(rows))
    assert bool(torch.all(s == 1.0))
    assert np.array_equal(q[:, 1:].cpu().numpy(), oracle.e4m3_encode(vals))


def _scales():
    """62 block maxima: an all-ones mantissa in each binade 2^-21 .. 2^19, and
    21 seeded mantissas over the same range."""
    ones = [np.float32(np.ldexp(np.float32(2.0) - np.float32(2.0) ** -23, j)) for j in range(-21, 20)]
    rng = np.random.default_rng(12)
    seeded = [np.float32(np.ldexp(1.0 + rng.random(), int(rng.integers(-21, 20)))) for _ in range(21)]
    return ones + seeded


def _probe_values(amax):
    """x whose quotient by s = fl32(amax/448) lies on and around every e4m3
    value and midpoint, near the subnormal boundary, plus seeded values."""
    s = np.float32(amax / np.float32(448.0))
    pos = oracle.E4M3_TABLE[1:0x7F]
    mids = (oracle.E4M3_TABLE[:0x7E] + oracle.E4M3_TABLE[1:0x7F]) / 2
    tiny = np.ldexp(1.0, np.arange(-13, -8)) * np.array([[1.0], [1.25], [1.5], [1.75]])
    targets = np.concatenate([pos, mids, tiny.reshape(-1)]).astype(np.float64)
    base = (targets * np.float64(s)).astype(np.float32)
    cand = [base]
    for k in (1, 2, 3):
        up, dn = base.copy(), base.copy()
        for _ in range(k):
            up = np.nextafter(up, np.float32(np.inf))
            dn = np.nextafter(dn, np.float32(0))
        cand += [up, dn]
    c = np.concatenate(cand)
    c = c[(c > 0) & (c <= amax)]
    rng = np.random.default_rng(int(np.float32(amax).view(np.uint32)))
    rnd = (rng.uniform(-1.0, 1.0, size=1 << 16) * amax).astype(np.float32)
    return np.concatenate([c, -c, rnd]).astype(np.float32)


def test_quotients_at_62_scales(moe):
    scales = _scales()
    assert len(scales) == 62
    for amax in scales:
        v = _probe_values(amax)
        per = 127
        n = (v.size + per - 1) // per
        x = np.zeros((n, per), np.float32)
        x.reshape(-1)[: v.size] = v
        rows = np.concatenate([np.full((n, 1), amax, np.float32), x], axis=1)
        q_ref, s_ref = oracle.quantize_rows(rows)
        q, s = _gpu_codes(moe, to_dev(rows))
        assert np.array_equal(s.cpu().numpy().view(np.uint32), s_ref.view(np.uint32)), amax
        qq = q.cpu().numpy()
        bad = np.argwhere(qq != q_ref)
        assert bad.size == 0, (float(amax), float(rows[tuple(bad[0])]), int(qq[tuple(bad[0])]), int(q_ref[tuple(bad[0])]))
    log(f"  62 scales from {min(scales):.3e} to {max(scales):.3e}: codes and scales equal")
