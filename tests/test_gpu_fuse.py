"""GPU parity of Stage-1 fusion (voxzip_fuse_spans) against the fp64 oracle."""
import numpy as np
import pytest

import oracle
import synth
from vzt import RTOL, GpuCache, bf16_ulp, check_close, from_dev, to_dev, widen

pytestmark = pytest.mark.gpu


def _run(k_in, v_in, off, dtype, cap, anchor=None, Hq=None):
    L, H, T, d = k_in.shape
    g = GpuCache(L, Hq or H, H, d, cap, dtype)
    sentinel = 7.0
    g.k.fill_(sentinel)
    g.v.fill_(sentinel)
    g.score.fill_(-1.0)
    g.pos.fill_(-5)
    ak = av = None
    if anchor is not None:
        ak, av = to_dev(anchor[0]), to_dev(anchor[1])
    g.fuse(to_dev(k_in), to_dev(v_in), to_dev(off), ak, av)
    k, v, s, p = g.snapshot()
    return g, k, v, s, p, sentinel


def _verify(k_in, v_in, off, dtype, k, v, s, p, sentinel, anchor=None):
    n = len(off) - 1
    for name, x_in, got, a in (("K", k_in, k, None if anchor is None else anchor[0]),
                               ("V", v_in, v, None if anchor is None else anchor[1])):
        ref = oracle.fuse(x_in, off, dtype, anchor=a)
        g = widen(got[:, :, :n], dtype)
        check_close(g, ref, RTOL[dtype], f"fused {name}")
        if dtype == synth.DT_BF16:  # one rounding of a float32 result: within one bf16 ulp
            assert np.all(np.abs(g - ref) <= bf16_ulp(ref) + 1e-6 * np.abs(ref))
        if anchor is None:  # length-1 spans are copies, bit for bit
            one = np.nonzero(np.diff(off) == 1)[0]
            assert np.array_equal(got[:, :, one], x_in[:, :, off[one]])
        assert np.all(widen(got[:, :, n:], dtype) == sentinel)  # slots past n_spans untouched
    assert np.array_equal(p[:, :n], np.broadcast_to(np.arange(n, dtype=np.int32), (p.shape[0], n)))
    assert np.all(s[:, :n] == 0.0) and np.all(p[:, n:] == -5) and np.all(s[:, n:] == -1.0)


@pytest.mark.parametrize("name", ["tiny", "layer"])
def test_fuse_workload_shapes(name):
    w = synth.workload(name)
    off = synth.offsets_from_lengths(synth.span_lengths(w))
    k_in, v_in = synth.prefill_kv(w, "k"), synth.prefill_kv(w, "v")
    n = len(off) - 1
    _, k, v, s, p, sen = _run(k_in, v_in, off, w.dtype, n + 40)
    _verify(k_in, v_in, off, w.dtype, k, v, s, p, sen)


@pytest.mark.parametrize("dtype,d", [(synth.DT_BF16, 64), (synth.DT_BF16, 128), (synth.DT_F32, 64),
                                     (synth.DT_F32, 128)])
def test_fuse_ragged_spans_with_anchor(dtype, d):
    L, H = 3, 2
    key = synth.stream_key(11, "fuse-ragged", dtype, d)
    lens = synth.uniform_int(key, 0, 97, 1, 41)          # tails of the 4-row unroll, long spans
    lens[::7] = 1
    off = synth.offsets_from_lengths(lens)
    T, n = int(off[-1]), len(lens)
    mk = lambda tag, shape: synth.as_storage(
        synth.normal_f32(synth.stream_key(key, tag), int(np.prod(shape))).reshape(shape) * np.float32(2.5), dtype)
    k_in, v_in = mk("k", (L, H, T, d)), mk("v", (L, H, T, d))
    anchor = (mk("ak", (L, H, n, d)), mk("av", (L, H, n, d)))
    _, k, v, s, p, sen = _run(k_in, v_in, off, dtype, n + 3, anchor=anchor)
    _verify(k_in, v_in, off, dtype, k, v, s, p, sen, anchor=anchor)
    _, k, v, s, p, sen = _run(k_in, v_in, off, dtype, n)      # cap exactly n_spans
    _verify(k_in, v_in, off, dtype, k, v, s, p, sen)


def test_fuse_single_span_and_all_identity():
    dtype, d = synth.DT_BF16, 128
    x = synth.as_storage(synth.normal_f32(synth.stream_key(5, "one"), 2 * 1 * 300 * d).reshape(2, 1, 300, d), dtype)
    y = synth.as_storage(synth.normal_f32(synth.stream_key(6, "one"), 2 * 1 * 300 * d).reshape(2, 1, 300, d), dtype)
    off = np.array([0, 300], dtype=np.int32)                 # one span over everything
    _, k, v, s, p, sen = _run(x, y, off, dtype, 4)
    _verify(x, y, off, dtype, k, v, s, p, sen)
    off = np.arange(301, dtype=np.int32)                     # every token its own span
    _, k, v, s, p, sen = _run(x, y, off, dtype, 300)
    assert np.array_equal(k, x) and np.array_equal(v, y)


def test_fuse_full_size_sampled_layers():
    """32k-token, 48-layer cache fused in one launch; layers 0, 23, 47 checked in full."""
    w = synth.workload("long32k")
    off = synth.offsets_from_lengths(synth.span_lengths(w))
    n = len(off) - 1
    k_in, v_in = synth.prefill_kv(w, "k"), synth.prefill_kv(w, "v")
    g, k, v, s, p, sen = _run(k_in, v_in, off, w.dtype, n + 300, Hq=w.n_q_heads)
    for l in (0, 23, 47):
        _verify(k_in[l:l + 1], v_in[l:l + 1], off, w.dtype, k[l:l + 1], v[l:l + 1], s[l:l + 1], p[l:l + 1], sen)
    assert np.all(p[:, :n] == np.arange(n)) and np.all(s[:, :n] == 0)


def test_fuse_with_offsets_from_the_span_builder():
    """End to end Stage 1: ASR segments -> voxzip_build_span_offsets (host) ->
    voxzip_fuse_spans (GPU), against the oracle's fusion of the oracle's offsets."""
    import paper_2608_08569_amd as vz
    key = synth.stream_key(5, "stage1-e2e")
    r = synth.uniform01(key, 0, 256)
    t_total, L_a, n = 120000, 1500, 30
    starts = np.sort((r[:n] * (t_total - 5000)).astype(np.int64))
    ends = starts + 800 + (r[n:2 * n] * 4000).astype(np.int64)
    conf = (0.1 + 0.9 * r[2 * n:3 * n]).astype(np.float32)
    tl = 1 + (r[3 * n:4 * n] * 12).astype(np.int32)
    off = vz.voxzip_build_span_offsets(starts, ends, conf, tl, t_total, L_a)
    assert np.array_equal(off, oracle.build_offsets(starts, ends, conf, tl, t_total, L_a))
    dtype, L, H, d = synth.DT_BF16, 2, 4, 128
    x = synth.as_storage(synth.normal_f32(synth.stream_key(key, "k"), L * H * L_a * d).reshape(L, H, L_a, d), dtype)
    y = synth.as_storage(synth.normal_f32(synth.stream_key(key, "v"), L * H * L_a * d).reshape(L, H, L_a, d), dtype)
    _, k, v, s, p, sen = _run(x, y, off, dtype, len(off) + 7)
    _verify(x, y, off, dtype, k, v, s, p, sen)
