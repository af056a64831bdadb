"""Pins of the oracle's Stage-1 fusion (Sec. 3.2.1, Eq. 4 and Eq. 5).

The fusion is a plain definition (a mean over each group), so the pins are
the library segmented sum, exact identities and conservation laws."""
import numpy as np
import pytest

import oracle
import synth


def _case(seed, L, H, d, lens, dtype):
    lens = np.asarray(lens, dtype=np.int64)
    T = int(lens.sum())
    key = synth.stream_key(seed, "fuse-test")
    x = synth.normal_f32(key, L * H * T * d).reshape(L, H, T, d) * np.float32(3.0)
    return synth.as_storage(x, dtype), synth.offsets_from_lengths(lens)


@pytest.mark.parametrize("dtype", [oracle.F32, oracle.BF16])
def test_matches_numpy_reduceat(dtype):
    lens = synth.span_lengths(synth.workload("tiny"))
    x, off = _case(1, 2, 3, 16, lens, dtype)
    got = oracle.fuse(x, off, dtype)
    xf = synth.storage_to_f64(x, dtype)
    ref = np.add.reduceat(xf, off[:-1], axis=2) / np.diff(off)[None, None, :, None]
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("dtype", [oracle.F32, oracle.BF16])
def test_length_one_spans_are_identity(dtype):
    x, off = _case(2, 1, 2, 8, [1] * 37, dtype)
    got = oracle.fuse(x, off, dtype)
    assert np.array_equal(got, synth.storage_to_f64(x, dtype))


def test_sum_conservation_and_constant_spans():
    lens = [5, 1, 9, 2, 2, 7]
    x, off = _case(3, 1, 1, 4, lens, oracle.F32)
    got = oracle.fuse(x, off, oracle.F32)
    xf = synth.storage_to_f64(x, oracle.F32)
    total = (got[0, 0] * np.asarray(lens)[:, None]).sum(axis=0)
    np.testing.assert_allclose(total, xf[0, 0].sum(axis=0), rtol=1e-12, atol=1e-12)
    # a span whose rows are all equal to c fuses to exactly c
    xc = x.copy()
    xc[0, 0, off[2]:off[3], :] = np.float32(0.625)
    got = oracle.fuse(xc, off, oracle.F32)
    assert np.all(got[0, 0, 2] == 0.625)


def test_anchor_is_added_after_the_mean():
    lens = [4, 3, 1]
    x, off = _case(4, 1, 2, 8, lens, oracle.F32)
    a = synth.normal_f32(synth.stream_key(4, "a"), 1 * 2 * 3 * 8).reshape(1, 2, 3, 8)
    plain = oracle.fuse(x, off, oracle.F32)
    anch = oracle.fuse(x, off, oracle.F32, anchor=a)
    np.testing.assert_allclose(anch - plain, a.astype(np.float64), rtol=0, atol=1e-12)


def test_layers_and_heads_are_independent():
    lens = [2, 6, 3]
    x, off = _case(5, 2, 2, 4, lens, oracle.F32)
    whole = oracle.fuse(x, off, oracle.F32)
    part = oracle.fuse(np.ascontiguousarray(x[1:2, 1:2]), off, oracle.F32)
    assert np.array_equal(whole[1:2, 1:2], part)


@pytest.mark.parametrize("bad", [[1, 3, 5], [0, 3, 3, 5], [0, 4, 2, 5], [0, 2, 6]])
def test_bad_offsets_rejected(bad):
    x, _ = _case(6, 1, 1, 4, [5], oracle.F32)
    with pytest.raises(ValueError):
        oracle.fuse(x, np.array(bad, dtype=np.int32), oracle.F32)
