"""CPU replay of the prefill GEMM's address arithmetic (no GPU).

For every work item of a launch and every one of its 512 threads, the index
arithmetic of ffn_prefill_kernel (work-item mapping, tile descriptor, the
one unconditional 4-byte load per thread, the packed weight loads of every K
block, the row-scale and expert-row loads with their stand-in rows, and the
output stores) is recomputed here, and each address is checked against the
size of the buffer it points into.  Shapes: the tiny layer, ragged tail
tiles with skewed routing, the DeepSeek-V3 prefill chunk (8192 tokens,
uniform) and the streamed path's launch over one group of G experts in
every chunk (an expert's rows of all chunks numbered as one run of launch
rows mapped to sorted positions and tokens by row tables, scales of a ring
whose end is the group's last slot).
"""
import numpy as np
import pytest

BM, BN, THREADS, XCD, TILE_BYTES, BAND = 128, 256, 512, 8, 2048, 8


def _max_mtiles(R, E):
    return (R + BM - 1) // BM + min(R, E)


def _describe(chunk_offsets, n_units, max_mtiles):
    """prefill_tiles_kernel: per expert u its rows (one chunk: sorted positions
    [off[u], off[u+1]); several chunks: launch rows [vstart[u], vstart[u] +
    M_u), M_u summed over the chunks), the m-tile scan and the descriptors."""
    one = len(chunk_offsets) == 1
    m = [sum(int(oc[u + 1] - oc[u]) for oc in chunk_offsets) for u in range(n_units)]
    vstart = np.concatenate([[0], np.cumsum(m)]).astype(np.int64)
    cnt = [(x + BM - 1) // BM if x > 0 else 0 for x in m]
    start = np.concatenate([[0], np.cumsum(cnt)]).astype(np.int64)
    desc = {}
    for u in range(n_units):
        o0 = int(chunk_offsets[0][u]) if one else int(vstart[u])
        for b in range(start[u], start[u] + cnt[u]):
            if b < max_mtiles:
                desc[b] = (u, int(start[u]), o0, o0 + m[u])
    return start, vstart, desc


def _row_tables(chunk_offsets, n_units, chunk_rows, chunk_tokens, sorted_src, topk, vstart):
    """prefill_rows_kernel: launch row -> (sorted position, token)."""
    n = int(vstart[-1])
    pos = np.full(n, -1, np.int64)
    tok = np.full(n, -1, np.int64)
    for u in range(n_units):
        v = int(vstart[u])
        for c, oc in enumerate(chunk_offsets):
            p0, cnt = int(oc[u]), int(oc[u + 1] - oc[u])
            pp = c * chunk_rows + p0 + np.arange(cnt)
            pos[v:v + cnt] = pp
            tok[v:v + cnt] = np.asarray(sorted_src)[pp] // topk + c * chunk_tokens
            v += cnt
    assert np.all(pos >= 0)
    return pos, tok


def _tile_of(desc, n_tiles, item):
    e, s0, o0, o1 = desc[item // n_tiles]
    mcount = (o1 - o0 + BM - 1) // BM
    local = item - s0 * n_tiles
    band = local // (BAND * n_tiles)
    width = min(BAND, mcount - band * BAND)
    ntx, mt = divmod(local - band * BAND * n_tiles, width)
    mt += band * BAND
    q = (o1 - o0 + 31) >> 5
    base, extra = divmod(q, mcount)
    first = o0 + 32 * (mt * base + min(mt, extra))
    groups = base + (1 if mt < extra else 0)
    return e, first, min(32 * groups, o1 - first), ntx


def _packed_lane_offset(h, kq, r):
    return 1024 * h + 512 * (kq & 1) + 256 * (kq >> 1) + 16 * r


def replay(gateup, E, N, K, topk, a_rows, offsets, sorted_src, R, n_chunks=1, chunk_rows=0, chunk_tokens=0,
           max_mtiles=None):
    """Checks every address one launch computes; returns the number of items run.

    E: experts of the launch (its weight stacks); offsets: [E+1] for one
    chunk, or a list of n_chunks such windows (chunk c's rows start at c *
    chunk_rows, its sorted_src entries are chunk-relative slots); a_rows:
    rows of the activation operand (tokens for gate/up, routed rows for
    down); R: rows of the sorted order (sorted_src, the row tables and the
    outputs).
    """
    nb = K // 128
    n_tiles = N // 128 if gateup else N // BN
    chunk_offsets = offsets if n_chunks > 1 else [offsets]
    if max_mtiles is None:
        max_mtiles = _max_mtiles(R, E)
    start, vstart, desc = _describe(chunk_offsets, E, max_mtiles)
    tables = n_chunks > 1
    if tables:
        row_pos, row_tok = _row_tables(chunk_offsets, E, chunk_rows, chunk_tokens, sorted_src, topk, vstart)
        assert row_pos.size <= R
    total = min(int(start[E]), max_mtiles)
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
        e, m0, mc, nt = _tile_of(desc, n_tiles, item)
        assert 0 <= e < E
        assert 0 < mc <= BM and m0 >= 0 and m0 + mc <= R
        # (1) one 4-byte load per thread: a row index (sorted_src, or a row
        # table) or a weight scale; GATEUP with tables also the row's position.
        ti = np.minimum(tid, mc - 1)
        tw = np.where(tid < BM, 0, np.minimum(tid - BM, 2 * nb - 1))
        h, b = tw // nb, tw % nb
        wrow = e * (N // 128) + (nt if gateup else 2 * nt + h)
        sidx = wrow * nb + b
        has_index = gateup or tables
        uses_src = (tid < BM) & has_index
        table_len = row_pos.size if tables else R
        assert np.all(np.where(uses_src, m0 + ti < table_len, (sidx >= 0) & (sidx < scale_entries)))
        # (2) packed weights: every K block (the ring loads clamp to nb - 1).
        grp = nt * (128 // 16) + wave if gateup else nt * (BN // 16) + 2 * wave + (r32 >> 4)
        w0 = e * N * K + grp * nb * TILE_BYTES + _packed_lane_offset(0, 2 * g2, r32 & 15)
        assert np.all(w0 >= 0)
        assert np.all(w0 + (nb - 1) * TILE_BYTES + 1536 + 16 <= E * N * K)
        # (3) activation rows and their scales (stand-in rows for invalid or
        # missing ones: the tile's last row, row 0 if that one is invalid),
        # and the output rows.
        rows = np.arange(BM)
        vrow = m0 + np.minimum(rows, mc - 1)
        if tables:
            pos = row_pos[vrow]
            srow = row_tok[vrow] if gateup else pos
        else:
            pos = m0 + rows
            srow = np.asarray(sorted_src)[vrow] // topk if gateup else pos
        arow = np.where((rows < mc) & (srow >= 0) & (srow < a_rows), srow, -1)
        a_last = arow[mc - 1] if arow[mc - 1] >= 0 else 0
        ar = np.where(arow >= 0, arow, a_last)
        assert np.all((ar >= 0) & (ar < a_rows))
        assert np.all(ar * nb + (nb - 1) < a_rows * nb)                    # row-scale loads
        c = np.concatenate([tid, tid + THREADS])
        a_off = ar[c >> 3] * K + (c & 7) * 16
        assert np.all(a_off + (nb - 1) * 128 + 16 <= a_rows * K)           # expert-row loads
        orow = pos[:mc]
        assert np.all((orow >= 0) & (orow < R))
        # (4) stores of the rows below mc, at their output rows.
        if gateup:
            row = c >> 3
            live = row < mc
            q_off = orow[np.minimum(row, mc - 1)] * N + nt * 128 + (c & 7) * 16
            assert np.all(q_off[live] + 16 <= R * N)
            assert np.all(orow * (N // 128) + nt < R * (N // 128))
        else:
            for j in range(4):
                t = j * 32 + r32
                live = t < mc
                dst = orow[np.minimum(t, mc - 1)] * N + nt * BN + wave * 32 + g2 * 4
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


def test_work_items_cover_every_tile_once():
    """The work-item order (an expert's m-tiles in bands of 8, each band
    n-tile major) is a bijection onto (m-tile, n-tile) pairs, and an expert's
    m-tiles partition its rows, for experts of 0 to 21 m-tiles (one band, two
    and a partial third) and ragged tails."""
    rng = np.random.default_rng(3)
    m = [0, 1, 31, 128, 129, 1000, 1024, 1025, 2047, 2560] + list(rng.integers(0, 2700, 20))
    offsets = np.concatenate([[0], np.cumsum(m)]).astype(np.int64)
    for n_tiles in (1, 3, 16, 28):
        start, _, desc = _describe([offsets], len(m), 10**9)
        seen = {}
        for item in range(int(start[-1]) * n_tiles):
            e, first, mc, nt = _tile_of(desc, n_tiles, item)
            assert 0 <= nt < n_tiles and 0 < mc <= BM
            assert (e, first, nt) not in seen
            seen[(e, first, nt)] = mc
        for u in range(len(m)):
            for nt in range(n_tiles):
                pos = int(offsets[u])
                for f, c in sorted((f, c) for (e, f, t), c in seen.items() if e == u and t == nt):
                    assert f == pos
                    pos += c
                assert pos == int(offsets[u + 1])


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
    an expert's tiles spanning chunks through the row tables (the last chunk
    partial), the
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
        mm = (R + 127) // 128 + G
        for gateup in (True, False):
            n = replay(gateup, G, I if gateup else H, H if gateup else I, k, T if gateup else R, window,
                       src_all, R, n_chunks=n_chunks, chunk_rows=chunk * k, chunk_tokens=chunk, max_mtiles=mm)
            rows_u = [sum(int(o[e0 + u + 1] - o[e0 + u]) for o in offs) for u in range(G)]
            tiles = sum(-(-m // 128) for m in rows_u)
            assert n == tiles * (I // 128 if gateup else H // 256)
