"""The seeded input generator: SplitMix64 values, rounding, span recipes."""
import math

import numpy as np
import pytest
import torch

import synth

MASK = (1 << 64) - 1


def _splitmix_scalar(state, n):
    """Sequential SplitMix64 written out with Python integers (a second,
    independent implementation of the published generator)."""
    out = []
    for _ in range(n):
        state = (state + 0x9E3779B97F4A7C15) & MASK
        z = state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK
        out.append(z ^ (z >> 31))
    return out


def test_splitmix_published_first_value():
    # SplitMix64 seeded with 0: first output of the reference generator.
    assert int(synth.splitmix_u64(0, 0, 1)[0]) == 0xE220A8397B1DCDAF


@pytest.mark.parametrize("key", [0, 1, 0xDEADBEEF, (1 << 64) - 5])
def test_splitmix_vector_matches_sequential(key):
    ref = _splitmix_scalar(key, 64)
    got = [int(x) for x in synth.splitmix_u64(key, 0, 64)]
    assert got == ref
    # counter-based: an offset window equals the matching slice
    got_off = [int(x) for x in synth.splitmix_u64(key, 17, 10)]
    assert got_off == ref[17:27]


def test_normals_box_muller_values_and_moments():
    key = synth.stream_key(3, "t")
    u = synth.splitmix_u64(key, 0, 8)
    z = synth.normal_f32(key, 8)
    for i in range(4):
        u1 = ((int(u[2 * i]) >> 11) + 1) * 2.0 ** -53
        u2 = (int(u[2 * i + 1]) >> 11) * 2.0 ** -53
        r = math.sqrt(-2 * math.log(u1))
        assert z[2 * i] == np.float32(r * math.cos(2 * math.pi * u2))
        assert z[2 * i + 1] == np.float32(r * math.sin(2 * math.pi * u2))
    big = synth.normal_f32(key, 1 << 20).astype(np.float64)
    assert abs(big.mean()) < 5e-3
    assert abs(big.var() - 1.0) < 5e-3


def test_threaded_generation_is_deterministic():
    key = synth.stream_key(9, "x")
    a = synth.normal_f32(key, (1 << 23) + 3)
    b = synth.normal_f32(key, (1 << 23) + 3)
    assert np.array_equal(a, b)
    # the tail of a longer draw equals a shorter draw (counter-based)
    c = synth.normal_f32(key, 1000)
    assert np.array_equal(a[:1000], c)


def test_bf16_rounding_matches_torch():
    key = synth.stream_key(1, "bf")
    x = synth.normal_f32(key, 100000) * np.float32(37.0)
    edge = np.array([0.0, -0.0, 1.0, 1.00390625, 1.0039063, 1.01171875, 3.0e38, -3.0e38, 1e-40,
                     np.float32(1.0) + np.float32(2 ** -8), np.float32(1.0) + np.float32(3 * 2 ** -8)],
                    dtype=np.float32)
    x = np.concatenate([x, edge])
    ours = synth.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = synth.bf16_bits_to_f32(ours)
    assert np.array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_span_recipes():
    w = synth.workload("tiny")
    lens = synth.span_lengths(w)
    assert len(lens) == 64 and lens.sum() == 512 and lens.min() >= 1 and lens.max() <= 16

    w = synth.workload("layer")
    lens = synth.span_lengths(w)
    audio = lens[: len(lens) - 256]
    assert lens.sum() == 4096 + 256 and np.all(lens[-256:] == 1)
    assert audio.max() <= 32 and 3.5 < audio.mean() < 4.5

    w = synth.workload("long32k")
    lens = synth.span_lengths(w)
    assert lens.sum() == 32768 and lens.max() <= 32
    assert 7600 < len(lens) < 8800  # about 0.25x of the audio tokens

    w = synth.workload("aggr64k")
    lens = synth.span_lengths(w)
    assert lens.sum() == 65536 and lens.max() <= 64
    assert 4.6 < lens.mean() < 5.4
    assert 0.07 < np.mean(lens == 1) < 0.14


def test_offsets_and_state_helpers():
    off = synth.offsets_from_lengths(np.array([3, 1, 2]))
    assert off.tolist() == [0, 3, 4, 6]
    k, v, s, p = synth.random_state(0, 2, 2, 8, 40, 30, synth.DT_BF16, next_pos=100)
    assert k.dtype == np.uint16 and k.shape == (2, 2, 40, 8)
    for l in range(2):
        pl = p[l, :30]
        assert len(set(pl.tolist())) == 30
        assert set(range(4)) <= set(pl.tolist())
        assert set(range(90, 100)) <= set(pl.tolist())
        assert np.all(s[l, :30] >= 0)


def test_decode_inputs_shapes_and_bias():
    w = synth.workload("aggr64k")
    w.n_layers = 2
    b = synth.q_bias(w)
    assert b.shape == (2, 32, 128)
    norms = np.linalg.norm(b, axis=-1)
    assert np.allclose(norms, norms[0, 0])
    q, k, v = synth.decode_inputs(w, 0, bias=b)
    assert q.shape == (2, 32, 128) and k.shape == (2, 4, 128) and q.dtype == np.uint16


def test_batch_workload():
    lens = synth.batch_lengths()
    assert lens.shape == (synth.BATCH,) and lens.min() >= 2048 and lens.max() <= 32768
    assert np.array_equal(lens, synth.batch_lengths())            # seeded
    assert not np.array_equal(lens, synth.batch_lengths(seed=1))
    ws = synth.batch_workloads()
    assert [w.budget for w in ws] == [int(n) // 4 for n in lens]
    assert all(w.interval == 16 and w.n_layers == 48 and w.steps == 128 for w in ws)
    # each sequence draws its own spans
    a, b = synth.span_lengths(ws[0], seq=0), synth.span_lengths(ws[1], seq=1)
    assert a.sum() == lens[0] and b.sum() == lens[1] and not np.array_equal(a[:50], b[:50])
