"""Pins of the oracle's Stage-1 span builder (Sec. 3.2.1: confidence filter,
Eq. 3 time-to-index map, uniform groups, background intervals, Eq. 5 order).

Eq. (3) is checked against exact rational arithmetic; the partition is checked
against the properties the paper states (consecutive groups, uniform sizes,
L_t groups per interval, background tokens preserved one by one)."""
from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth


def _labels(ts, te, conf, tl, t_total, L_a, thr=0.3):
    """Token -> owning segment (or None), from Eq. 3 in exact rationals."""
    segs = []
    for s, e, c, n in zip(ts, te, conf, tl):
        if not c > thr:  # "above" the threshold
            continue
        s, e = max(0, s), min(t_total, e)
        if e <= s:
            continue
        i0 = int(Fraction(L_a) * Fraction(int(s), int(t_total)))  # floor for non-negatives
        i1 = int(Fraction(L_a) * Fraction(int(e), int(t_total)))
        segs.append((i0, i1, len(segs), n))
    segs.sort()  # start, then end, then input order
    owner = [None] * L_a
    cur = 0
    for idx, (i0, i1, _, n) in enumerate(segs):
        i0 = max(i0, cur)
        if i1 <= i0 or n < 1:
            continue
        for t in range(i0, i1):
            owner[t] = (idx, n)
        cur = i1
    return owner


def _check(off, owner, L_a):
    off = np.asarray(off)
    assert off[0] == 0 and off[-1] == L_a and np.all(np.diff(off) > 0)
    groups = {}
    for j in range(len(off) - 1):
        a, b = off[j], off[j + 1]
        own = {owner[t] for t in range(a, b)}
        assert len(own) == 1, "a span mixes intervals"
        o = own.pop()
        if o is None:
            assert b - a == 1, "background tokens stay one per span"
        else:
            groups.setdefault(o, []).append(b - a)
    for (idx, n_text), sizes in groups.items():
        length = sum(sizes)
        assert len(sizes) == min(n_text, length)
        assert max(sizes) - min(sizes) <= 1


@pytest.mark.parametrize("seed", range(60))
def test_random_segment_lists(seed):
    key = synth.stream_key(seed, "offsets")
    r = synth.uniform01(key, 0, 64)
    L_a = 1 + int(r[0] * 16)
    t_total = 1000 + int(r[1] * 5000)
    n_seg = int(r[2] * 5)
    ts = (r[3:3 + n_seg] * t_total).astype(np.int64)
    te = ts + (r[10:10 + n_seg] * t_total * 0.6).astype(np.int64)
    conf = r[20:20 + n_seg].astype(np.float32)
    tl = 1 + (r[30:30 + n_seg] * 6).astype(np.int32)
    off = oracle.build_offsets(ts, te, conf, tl, t_total, L_a)
    _check(off, _labels(ts, te, conf, tl, t_total, L_a), L_a)


def test_confidence_threshold_is_strict():
    off = oracle.build_offsets([0], [1000], np.array([0.3], np.float32), [2], 1000, 8)
    assert off.tolist() == list(range(9))  # conf == 0.3 is dropped: all background
    off = oracle.build_offsets([0], [1000], np.array([0.31], np.float32), [2], 1000, 8)
    assert off.tolist() == [0, 4, 8]


def test_eq3_floor_and_compression_ratio():
    # one 10 s segment of a 40 s clip with 400 audio tokens and 25 text tokens:
    # tokens floor(400*10/40)=100 .. floor(400*20/40)=200 fuse into 25 groups of 4
    off = oracle.build_offsets([10000], [20000], np.array([0.9], np.float32), [25], 40000, 400)
    assert len(off) - 1 == 100 + 25 + 200
    sizes = np.diff(off)
    assert np.all(sizes[:100] == 1) and np.all(sizes[100:125] == 4) and np.all(sizes[125:] == 1)


def test_overlaps_are_clipped_and_text_longer_than_audio():
    # second segment starts inside the first: it starts at the first one's end
    off = oracle.build_offsets([0, 500], [1000, 2000], np.array([0.9, 0.9], np.float32),
                               [50, 1], 2000, 20)
    # first: tokens 0..9 with 50 text tokens -> min(50, 10) = 10 groups of 1; second: 10..19 -> 1 group
    assert off.tolist() == list(range(11)) + [20]


def test_equal_intervals_keep_input_order():
    # two segments mapping to the same token interval: the first one in input
    # order is taken, the second starts at its end and is dropped (empty)
    conf = np.array([0.9, 0.9], np.float32)
    off = oracle.build_offsets([0, 0], [1000, 1000], conf, [2, 5], 1000, 8)
    assert off.tolist() == [0, 4, 8]
    off = oracle.build_offsets([0, 0], [1000, 1000], conf, [5, 2], 1000, 8)
    assert off.tolist() == [0, 1, 3, 4, 6, 8]
