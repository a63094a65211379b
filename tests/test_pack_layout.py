"""CPU check of the packed weight layout's numpy definition (used by the GPU
test of moe_pack_weight) against a byte-by-byte loop over the layout rule."""
import numpy as np

from gpu_cases import pack_reference


def test_pack_reference_matches_layout_rule_bytewise():
    rng = np.random.default_rng(0)
    q = rng.integers(0, 256, size=(2, 32, 256), dtype=np.uint8)
    p = pack_reference(q).reshape(2, -1)
    n, rows, cols = q.shape
    for m in range(n):
        for g in range(rows // 16):
            for b in range(cols // 128):
                base = (g * (cols // 128) + b) * 2048
                for h in range(2):
                    for kq in range(4):
                        for r in range(16):
                            off = base + 1024 * h + 512 * (kq % 2) + 256 * (kq // 2) + 16 * r
                            got = p[m, off: off + 16]
                            col = 128 * b + 64 * h + 16 * kq
                            want = q[m, 16 * g + r, col: col + 16]
                            assert np.array_equal(got, want)


def test_pack_reference_is_a_permutation():
    q = np.arange(16 * 128, dtype=np.int64).reshape(1, 16, 128) % 251
    p = pack_reference(q.astype(np.uint8))
    assert sorted(p.reshape(-1).tolist()) == sorted(q.astype(np.uint8).reshape(-1).tolist())
