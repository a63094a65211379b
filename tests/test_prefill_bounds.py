"""CPU replay of the prefill GEMM's address arithmetic (no GPU).

For every work item of a launch and every one of its 512 threads, the index
arithmetic of ffn_prefill_kernel (work-item mapping, tile descriptor, the
one unconditional 4-byte load per thread, the packed weight loads of every K
block, the row-scale and expert-row loads with their stand-in rows, and the
output stores) is recomputed here, and each address is checked against the
size of the buffer it points into.  Shapes: the tiny layer, ragged tail
tiles with skewed routing, the DeepSeek-V3 prefill chunk (8192 tokens,
uniform) and the streamed path's launch over one group of G experts in
every chunk (segments of one expert in one chunk, row positions absolute
over the chunks, scales of a ring whose end is the group's last slot).
"""
import numpy as np
import pytest

BM, BN, THREADS, XCD, TILE_BYTES = 128, 256, 512, 8, 2048


def _max_mtiles(R, E):
    return (R + BM - 1) // BM + min(R, E)


def _describe(chunk_offsets, n_units, n_chunks, chunk_rows, max_mtiles):
    """prefill_tiles_kernel: segments seg = u * n_chunks + c (expert u's rows of
    chunk c, absolute rows c * chunk_rows + chunk c's offsets), their m-tile
    scan and the per-m-tile descriptors."""
    segs = []
    for u in range(n_units):
        for c in range(n_chunks):
            oc = chunk_offsets[c]
            segs.append((c * chunk_rows + int(oc[u]), c * chunk_rows + int(oc[u + 1])))
    cnt = [(o1 - o0 + BM - 1) // BM if o1 > o0 else 0 for o0, o1 in segs]
    start = np.concatenate([[0], np.cumsum(cnt)]).astype(np.int64)
    desc = {}
    for seg, (o0, o1) in enumerate(segs):
        for b in range(start[seg], start[seg] + cnt[seg]):
            if b < max_mtiles:
                desc[b] = (seg, int(start[seg]), o0, o1)
    return start, desc


def _tile_of(desc, n_tiles, n_chunks, item):
    seg, s0, o0, o1 = desc[item // n_tiles]
    e, chunk = divmod(seg, n_chunks)
    mcount = (o1 - o0 + BM - 1) // BM
    local = item - s0 * n_tiles
    ntx, mt = divmod(local, mcount)
    q = (o1 - o0 + 31) >> 5
    base, extra = divmod(q, mcount)
    first = o0 + 32 * (mt * base + min(mt, extra))
    groups = base + (1 if mt < extra else 0)
    return e, chunk, first, min(32 * groups, o1 - first), ntx


def _packed_lane_offset(h, kq, r):
    return 1024 * h + 512 * (kq & 1) + 256 * (kq >> 1) + 16 * r


def replay(gateup, E, N, K, topk, a_rows, offsets, sorted_src, R, n_chunks=1, chunk_rows=0, chunk_tokens=0,
           max_mtiles=None):
    """Checks every address one launch computes; returns the number of items run.

    E: experts of the launch (its weight stacks); offsets: [E+1] for one
    chunk, or a list of n_chunks such windows (chunk c's rows start at c *
    chunk_rows, its sorted_src entries are chunk-relative slots); a_rows:
    rows of the activation operand (tokens for gate/up, routed rows for
    down); R: rows of the sorted order (sorted_src and the outputs).
    """
    nb = K // 128
    n_tiles = N // 128 if gateup else N // BN
    chunk_offsets = offsets if n_chunks > 1 else [offsets]
    n_seg = E * n_chunks
    if max_mtiles is None:
        max_mtiles = _max_mtiles(R, E)
    start, desc = _describe(chunk_offsets, E, n_chunks, chunk_rows, max_mtiles)
    total = min(int(start[n_seg]), max_mtiles)
    real = total * n_tiles
    grid = (max_mtiles * n_tiles + XCD - 1) // XCD * XCD
    per = (real + XCD - 1) // XCD
    tid = np.arange(THREADS)
    lane, wave = tid & 63, tid >> 6
    r32, g2 = lane & 31, lane >> 5
    scale_entries = E * (N // 128) * nb
    ran = 0
    for block in range(grid):
        slot = block // XCD
        if slot >= per:
            continue
        item = (block % XCD) * per + slot
        if item >= real:
            continue
        ran += 1
        e, chunk, m0, mc, nt = _tile_of(desc, n_tiles, n_chunks, item)
        assert 0 <= e < E and 0 <= chunk < n_chunks
        assert 0 < mc <= BM and m0 >= 0 and m0 + mc <= R
        # (1) one 4-byte load per thread: a sorted_src entry or a weight scale.
        ti = np.minimum(tid, mc - 1)
        tw = np.where(tid < BM, 0, np.minimum(tid - BM, 2 * nb - 1))
        h, b = tw // nb, tw % nb
        wrow = e * (N // 128) + (nt if gateup else 2 * nt + h)
        sidx = wrow * nb + b
        uses_src = (tid < BM) & gateup
        assert np.all(np.where(uses_src, m0 + ti < R, (sidx >= 0) & (sidx < scale_entries)))
        # (2) packed weights: every K block (the ring loads clamp to nb - 1).
        grp = nt * (128 // 16) + wave if gateup else nt * (BN // 16) + 2 * wave + (r32 >> 4)
        w0 = e * N * K + grp * nb * TILE_BYTES + _packed_lane_offset(0, 2 * g2, r32 & 15)
        assert np.all(w0 >= 0)
        assert np.all(w0 + (nb - 1) * TILE_BYTES + 1536 + 16 <= E * N * K)
        # (3) activation rows and their scales (stand-in rows for invalid or
        # missing ones: the tile's last row, row 0 if that one is invalid).
        rows = np.arange(BM)
        if gateup:
            srow = np.array([sorted_src[m0 + min(t, mc - 1)] // topk + chunk * chunk_tokens for t in rows])
        else:
            srow = m0 + rows
        arow = np.where((rows < mc) & (srow >= 0) & (srow < a_rows), srow, -1)
        a_last = arow[mc - 1] if arow[mc - 1] >= 0 else 0
        ar = np.where(arow >= 0, arow, a_last)
        assert np.all((ar >= 0) & (ar < a_rows))
        assert np.all(ar * nb + (nb - 1) < a_rows * nb)                    # row-scale loads
        c = np.concatenate([tid, tid + THREADS])
        a_off = ar[c >> 3] * K + (c & 7) * 16
        assert np.all(a_off + (nb - 1) * 128 + 16 <= a_rows * K)           # expert-row loads
        # (4) stores of the rows below mc.
        if gateup:
            row = c >> 3
            live = row < mc
            q_off = (m0 + row) * N + nt * 128 + (c & 7) * 16
            assert np.all(q_off[live] + 16 <= R * N)
            assert m0 + mc - 1 < R and (m0 + mc - 1) * (N // 128) + nt < R * (N // 128)
        else:
            for j in range(4):
                t = j * 32 + r32
                live = t < mc
                dst = (m0 + t) * N + nt * BN + wave * 32 + g2 * 4
                assert np.all(dst[live] + 3 * 8 + 4 <= R * N)
    return ran


def _routing(T, E, k, zipf_s, seed):
    rng = np.random.default_rng(seed)
    logp = np.zeros(E) if zipf_s == 0 else -zipf_s * np.log(np.arange(1, E + 1))
    g = rng.gumbel(size=(T, E))
    return np.argsort(-(logp[None, :] + g), axis=1, kind="stable")[:, :k].astype(np.int32)


def _sorted(ids, E):
    flat = ids.reshape(-1)
    order = np.argsort(flat, kind="stable").astype(np.int64)
    offsets = np.concatenate([[0], np.cumsum(np.bincount(flat, minlength=E))]).astype(np.int64)
    return offsets, order


def _run_layer(H, I, E, k, T, zipf_s, seed):
    ids = _routing(T, E, k, zipf_s, seed)
    offsets, src = _sorted(ids, E)
    R = T * k
    n_gu = replay(True, E, I, H, k, T, offsets, src, R)
    n_dn = replay(False, E, H, I, k, R, offsets, None, R)
    return n_gu, n_dn, offsets


@pytest.mark.parametrize("H,I,E,k,T,zipf_s", [
    (256, 128, 8, 2, 16, 0.0),        # the tiny layer
    (512, 256, 16, 4, 300, 1.2),      # ragged tails, skewed routing
    (1024, 384, 4, 4, 700, 0.0),      # k = E, several m-tiles per expert
])
def test_prefill_addresses_small_shapes(H, I, E, k, T, zipf_s):
    n_gu, n_dn, _ = _run_layer(H, I, E, k, T, zipf_s, 0)
    assert n_gu > 0 and n_dn > 0


def test_prefill_addresses_deepseek_prefill_chunk():
    """8192 tokens, uniform top-8 of 256 experts: the last expert has far more
    than 32 rows, so its down tiles on the last n-tile reach the end of the
    scale table."""
    n_gu, n_dn, offsets = _run_layer(7168, 2048, 256, 8, 8192, 0.0, 0)
    assert offsets[256] - offsets[255] > 32
    assert n_gu == 16 * sum(-(-int(m) // 128) for m in np.diff(offsets) if m > 0)
    assert n_dn == 28 * (n_gu // 16)


def test_prefill_addresses_streamed_group_over_chunks():
    """The streamed path's launch pair of one group of G experts over all
    chunks: each chunk sorted on its own (offsets and chunk-relative slots),
    row positions absolute over the chunks (the last chunk partial), the
    weight and scale stacks holding exactly the G experts (a group that ends
    at the ring's last slot)."""
    H, I, E, k, T, G, chunk = 7168, 2048, 256, 8, 1500, 16, 512
    ids = _routing(T, E, k, 0.8, 1)
    n_chunks = -(-T // chunk)
    offs, srcs = [], []
    for c in range(n_chunks):
        o, s = _sorted(ids[c * chunk:(c + 1) * chunk], E)
        offs.append(o)
        srcs.append(s)
    src_all = np.concatenate(srcs)       # chunk c's entries at c * chunk * k (the last chunk partial)
    R = T * k
    assert src_all.size == R
    for e0 in (0, 112, E - G):
        window = [o[e0:e0 + G + 1] for o in offs]
        mm = (R + 127) // 128 + G * n_chunks
        for gateup in (True, False):
            n = replay(gateup, G, I if gateup else H, H if gateup else I, k, T if gateup else R, window,
                       src_all if gateup else None, R, n_chunks=n_chunks, chunk_rows=chunk * k, chunk_tokens=chunk,
                       max_mtiles=mm)
            segs = [(c, u) for u in range(G) for c in range(n_chunks)]
            tiles = sum(-(-int(offs[c][e0 + u + 1] - offs[c][e0 + u]) // 128) for c, u in segs)
            assert n == tiles * (I // 128 if gateup else H // 256)
