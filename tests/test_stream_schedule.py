"""The ring schedule of the stream-loaded layer, checked on the host (no GPU).

moe_stream_schedule returns the copy / event / launch sequence that
moe_ffn_streamed enqueues (the same host function builds both).  Here that
sequence is run through a model of the two streams: ops of one stream run in
order, and a wait on an event follows the event's latest record enqueued
before it (HIP's rule; a wait on a never-recorded event does not wait).
From the happens-before order this gives, for every call of a stack of
layers sharing one ring and one context (System Design, Stream-loading
Prefill: the loader fills a slot and sets ON, the model waits for ON, runs
the expert and sets OFF, the slot is reused without copying back):

* every expert is copied once and launched once per call, from slot
  expert mod ring_slots, in groups whose size divides the ring;
* a launch reads each of its slots only after the copy of its own expert
  into that slot has finished, with no later copy into the slot before it;
* a copy overwrites a slot only after every earlier launch that reads the
  slot has finished, in this call or an earlier one;
* with two slot groups or more the copy of the next group does not wait
  for the current group's launch (the copies overlap the kernels).
"""
import pytest

import paper_2606_10493_amd as moe

COPY_OPS = {moe.MOE_SOP_WAIT_OFF, moe.MOE_SOP_COPY, moe.MOE_SOP_RECORD_ON}
COMPUTE_OPS = {moe.MOE_SOP_WAIT_ON, moe.MOE_SOP_LAUNCH, moe.MOE_SOP_RECORD_OFF}


def _happens_before(ops):
    """Vector clocks of the two-stream model: vc[i] = (last copy-stream
    position, last compute-stream position) that happen before op i (i's own
    stream position included).  Returns (stream, position, vc) per op."""
    pos = {"copy": -1, "compute": -1}
    last_vc = {"copy": (-1, -1), "compute": (-1, -1)}
    last_record = {}  # (kind, slot) -> vc of the latest record
    out = []
    for op, a, _, _ in ops:
        s = "copy" if op in COPY_OPS else "compute"
        assert op in COPY_OPS | COMPUTE_OPS
        pos[s] += 1
        vc = list(last_vc[s])
        if op in (moe.MOE_SOP_WAIT_OFF, moe.MOE_SOP_WAIT_ON):
            kind = "off" if op == moe.MOE_SOP_WAIT_OFF else "on"
            rec = last_record.get((kind, a))
            if rec is not None:
                vc = [max(vc[0], rec[0]), max(vc[1], rec[1])]
        vc[0 if s == "copy" else 1] = pos[s]
        vc = tuple(vc)
        last_vc[s] = vc
        if op in (moe.MOE_SOP_RECORD_OFF, moe.MOE_SOP_RECORD_ON):
            last_record[("off" if op == moe.MOE_SOP_RECORD_OFF else "on", a)] = vc
        out.append((s, pos[s], vc))
    return out


def _before(hb, i, j):
    """Op i happens before op j."""
    s, p, _ = hb[i]
    return hb[j][2][0 if s == "copy" else 1] >= p


def _schedule(E, ring, calls):
    """calls: (T, chunk, k) per layer, all on one ring and one context."""
    rec = None
    ops, spans = [], []
    for T, chunk, k in calls:
        d = moe.MoeDims(256, 128, E, k)
        o, rec = moe.moe_stream_schedule(d, T, chunk, ring, rec)
        spans.append((len(ops), len(ops) + len(o), T))
        ops += o
    assert rec == bytes([1] * min(ring, E) + [0] * (ring - min(ring, E)))
    return ops, spans


def _check_stack(E, ring, calls):
    ops, spans = _schedule(E, ring, calls)
    _check(ops, spans, E, ring)


def _check(ops, spans, E, ring):
    hb = _happens_before(ops)

    for lo, hi, T in spans:
        copies = [i for i in range(lo, hi) if ops[i][0] == moe.MOE_SOP_COPY]
        launches = [i for i in range(lo, hi) if ops[i][0] == moe.MOE_SOP_LAUNCH]
        if T == 0:
            assert not copies and not launches
            continue
        groups = [ops[i][1:] for i in copies]
        assert groups == [ops[i][1:] for i in launches]  # each group copied, then launched, in order
        assert [e for a, b, _ in groups for e in range(a, a + b)] == list(range(E))  # each expert once
        for a, b, c in groups:
            assert c == a % ring and c + b <= ring
        if len(groups) > 1:  # the group size G: every group but the last has G experts
            G = groups[0][1]
            assert all(b == G for _, b, _ in groups[:-1]) and groups[-1][1] <= G
            assert ring % G == 0 and (ring == 1 or G <= ring // 2)
        # With two slot groups or more, the next group's copy does not wait for this group's launch.
        if len(groups) > 1 and ring // groups[0][1] >= 2:
            for n in range(len(launches) - 1):
                assert not _before(hb, launches[n], copies[n + 1])

    writes = {}  # slot -> index of the last COPY op writing it
    readers = {}  # slot -> launch op indices since that copy
    for i, (op, a, b, c) in enumerate(ops):
        if op == moe.MOE_SOP_COPY:
            for s in range(c, c + b):
                for r in readers.get(s, []):  # write after read
                    assert _before(hb, r, i), f"copy {i} into slot {s} may overwrite it under launch {r}"
                writes[s] = (i, a + s - c)
                readers[s] = []
        elif op == moe.MOE_SOP_LAUNCH:
            for s in range(c, c + b):
                w, expert = writes[s]  # read after write: the latest copy into s holds this launch's expert
                assert expert == a + s - c
                assert _before(hb, w, i), f"launch {i} may read slot {s} before copy {w} lands"
                readers[s].append(i)


@pytest.mark.parametrize("ring", [1, 2, 3, 4, 6, 16, 32, 256])
def test_one_layer_deepseek_experts(ring):
    _check_stack(256, ring, [(4096, 4096, 8)])


@pytest.mark.parametrize("ring", [1, 2, 4, 32])
def test_layer_stack_shares_the_ring(ring):
    """Four layers on one ring; the group size changes between calls (chunk
    sizes give different rows per expert), so a group of one call waits for
    slots that launches of another grouping read."""
    _check_stack(256, ring, [(4096, 4096, 8), (700, 256, 8), (32768, 4096, 8), (16, 16, 2)])


@pytest.mark.parametrize("E,ring", [(7, 2), (7, 3), (7, 16), (16, 5), (1, 1), (1, 4)])
def test_partial_last_group_and_small_layers(E, ring):
    """E not a multiple of the group (a short last group), a ring larger
    than the layer (slots that are never filled), one expert."""
    k = min(E, 2)
    _check_stack(E, ring, [(300, 128, k), (0, 128, k), (5, 1, k), (300, 128, k)])


@pytest.mark.parametrize("mistake", ["no slot waits", "ON before the copy", "no ON wait", "one slot wait"])
def test_checker_catches_a_broken_schedule(mistake):
    """The checker itself: each edit lets a copy overwrite a slot that a
    launch still reads, or a launch read a slot before its copy lands.  The
    stack regroups the ring (16 experts per group, then 1, then 16 again),
    so a group's slots hold OFF records of different launches."""
    calls = [(4096, 4096, 8), (65536, 65536, 8), (4096, 4096, 8)]
    ops, spans = _schedule(256, 32, calls)
    tagged = [(n, o) for n, (lo, hi, _) in enumerate(spans) for o in ops[lo:hi]]
    if mistake == "no slot waits":
        bad = [(n, o) for n, o in tagged if o[0] != moe.MOE_SOP_WAIT_OFF]
    elif mistake == "ON before the copy":
        bad = []
        for n, o in tagged:
            if o[0] == moe.MOE_SOP_COPY:
                bad += [(n, (moe.MOE_SOP_RECORD_ON, o[3], 0, 0)), (n, o)]
            elif o[0] != moe.MOE_SOP_RECORD_ON:
                bad.append((n, o))
    elif mistake == "no ON wait":
        bad = [(n, o) for n, o in tagged if o[0] != moe.MOE_SOP_WAIT_ON]
    else:  # a group waits for the OFF record of its first slot only
        bad, first = [], True
        for n, o in tagged:
            if o[0] == moe.MOE_SOP_WAIT_OFF:
                if first:
                    bad.append((n, o))
                first = False
            else:
                first = True
                bad.append((n, o))
    assert len(bad) != len(tagged) or mistake == "ON before the copy"
    new_spans, at = [], 0
    for n, (_, _, T) in enumerate(spans):
        cnt = sum(1 for m, _ in bad if m == n)
        new_spans.append((at, at + cnt, T))
        at += cnt
    with pytest.raises(AssertionError):
        _check([o for _, o in bad], new_spans, 256, 32)
    _check(ops, spans, 256, 32)  # the library's own schedule of the same stack passes


def test_schedule_query_errors():
    d = moe.MoeDims(256, 128, 8, 2)
    n = moe.ctypes.c_int32(-1)
    rec = (moe.ctypes.c_uint8 * 4)()
    st = moe.lib.moe_stream_schedule(d, 16, 16, 4, moe.ctypes.cast(rec, moe.ctypes.c_void_p), None, 0,
                                     moe.ctypes.byref(n))
    assert st == moe.MOE_ERR_WORKSPACE and n.value > 0 and bytes(rec) == bytes(4)  # untouched
    for bad in (dict(ring=0), dict(T=-1), dict(chunk=0)):
        args = dict(T=16, chunk=16, ring=4)
        args.update(bad)
        st = moe.lib.moe_stream_schedule(d, args["T"], args["chunk"], args["ring"],
                                         moe.ctypes.cast(rec, moe.ctypes.c_void_p), None, 0, moe.ctypes.byref(n))
        assert st == moe.MOE_ERR_INVALID_ARG, bad
    st = moe.lib.moe_stream_schedule(moe.MoeDims(384, 128, 8, 2), 16, 16, 4,
                                     moe.ctypes.cast(rec, moe.ctypes.c_void_p), None, 0, moe.ctypes.byref(n))
    assert st == moe.MOE_ERR_UNSUPPORTED_SHAPE  # H % 256 != 0, as moe_ffn_streamed
