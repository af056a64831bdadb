"""GPU parity of the whole-range decode path: single-sequence bf16 calls with at
least 128 (layer, KV head) items, where one workgroup streams every key of a
(layer, KV head), or of one part of at most 8192 keys when the cache holds
more than 8224.  State-synced against the fp64 oracle (every layer for short
caches, sampled layers for long ones); the cases cover caches shorter than one
chunk per wave, ragged tails, the 8224-key maximum of one part (8 chunks per
wave and one 32-key tile), caches of 2 and 3 parts, 1 to 8 query heads per KV
head."""
import numpy as np
import pytest

import synth
from test_gpu_decode import synced_step
from vzt import GpuCache, from_dev, to_dev

pytestmark = pytest.mark.gpu


def layered_state(seed, L, Hkv, d, cap, length, dtype, next_pos):
    """A resident cache whose layers differ without drawing L layers of
    normals: a 4-layer random state, each layer rolled along its resident
    slots by a layer-dependent shift."""
    base_L = 4
    k0, v0, s0, p0 = synth.random_state(seed, base_L, Hkv, d, cap, length, dtype, next_pos=next_pos)
    k = np.zeros((L, Hkv, cap, d), dtype=k0.dtype)
    v = np.zeros_like(k)
    s = np.zeros((L, cap), dtype=s0.dtype)
    p = np.zeros((L, cap), dtype=p0.dtype)
    for l in range(L):
        b, sh = l % base_L, (37 * l) % max(length, 1)
        k[l, :, :length] = np.roll(k0[b, :, :length], sh, axis=1)
        v[l, :, :length] = np.roll(v0[b, :, :length], sh, axis=1)
        s[l, :length] = np.roll(s0[b, :length], sh)
        p[l, :length] = np.roll(p0[b, :length], sh)
    return k, v, s, p


def step_inputs(key, t, L, Hq, Hkv, d, dtype):
    mk = lambda tag, shape: synth.as_storage(
        synth.normal_f32(synth.stream_key(key, tag, t), int(np.prod(shape))).reshape(shape) * np.float32(1.7), dtype)
    return mk("q", (L, Hq, d)), mk("k", (L, Hkv, d)), mk("v", (L, Hkv, d))


def run_case(Hq, Hkv, L, length, steps=1, layers=None, seed=5):
    dtype, d = synth.DT_BF16, 128
    cap = length + steps + 1
    k, v, s, p = layered_state(seed, L, Hkv, d, cap, length, dtype, length + 11)
    g = GpuCache(L, Hq, Hkv, d, cap, dtype)
    g.load(k, v, s, p, length, length + 11)
    key = synth.stream_key(seed, "range", Hq, Hkv, L, length)
    for t in range(steps):
        q, kn, vn = step_inputs(key, t, L, Hq, Hkv, d, dtype)
        synced_step(g, q, kn, vn, 0.95, layers)
    return g


@pytest.mark.parametrize("length", [0, 1, 127, 128, 1000, 1023, 1024])
def test_whole_range_short_all_layers(length):
    """Fewer chunks than waves, exact chunk multiples and ragged tails; every
    one of the 32 layers against the oracle, two steps."""
    run_case(32, 4, 32, length, steps=2)


@pytest.mark.parametrize("length", [4095, 8191, 8192, 8222, 8223])
def test_whole_range_long_sampled_layers(length):
    """8 full chunks per wave (8191 -> 8192 keys), one more key or tile on
    the last wave (up to 8223 -> 8224 keys, the one-part maximum); layers 0,
    13 and 31."""
    run_case(32, 4, 32, length, steps=1, layers=[0, 13, 31])


@pytest.mark.parametrize("length", [7827, 7907, 8163])
def test_whole_range_alternating_order(length):
    """Two steps each (the new positions of consecutive steps differ in
    parity, so both read orders run): 7828 keys (61 full chunks and a 20-key
    partial one: on the odd step the waves' ranges are exchanged and wave 0
    holds 8 full chunks and the partial one in its last slot), 7908 and 8164
    (61 and 63 full chunks with a 100-key partial chunk: reversed without
    the exchange); layers 0, 13 and 31."""
    run_case(32, 4, 32, length, steps=2, layers=[0, 13, 31])


@pytest.mark.parametrize("length", [8224, 9215, 12000, 16384, 20000])
def test_whole_range_parts_sampled_layers(length):
    """Caches in parts: 8225 keys (the first past one part: 2 parts of 4352
    and 3873 keys), 12001, 16385 and 20001 (2 to 6 parts: at least
    ceil(T / 8192), more when they fill the last round of workgroups on the
    device's CUs), two steps (the second one key longer); layers 0, 13 and
    31."""
    run_case(32, 4, 32, length, steps=2, layers=[0, 13, 31])


@pytest.mark.parametrize("Hq,Hkv,L,length", [(16, 4, 32, 3000), (64, 8, 16, 5000), (8, 1, 128, 2000),
                                             (12, 2, 64, 777), (24, 4, 32, 8192), (64, 8, 16, 9000),
                                             (8, 1, 128, 8500), (12, 2, 64, 10000)])
def test_whole_range_head_groups(Hq, Hkv, L, length):
    """4, 8, 6 and 3 query heads per KV head, and 1, 2 or 8 KV heads; one
    part, or two parts for the longer caches."""
    run_case(Hq, Hkv, L, length, steps=1, layers=[0, L // 2, L - 1])


def test_whole_range_headline_shape_deterministic():
    """48 layers, 32Q/4KV, 8192 resident keys: two runs of the same step from
    the same state give identical bits, and every layer's output and scores
    are finite with each layer's score mass growing by 32 (Eq. 6 with the
    probabilities of 32 heads summing to one each)."""
    dtype, d, L, Hq, Hkv, length = synth.DT_BF16, 128, 48, 32, 4, 8192
    k, v, s, p = layered_state(9, L, Hkv, d, length + 2, length, dtype, length + 3)
    q, kn, vn = step_inputs(synth.stream_key(9, "headline"), 0, L, Hq, Hkv, d, dtype)
    runs = []
    for _ in range(2):
        g = GpuCache(L, Hq, Hkv, d, length + 2, dtype)
        g.load(k, v, s, p, length, length + 3)
        g.step(to_dev(q), to_dev(kn), to_dev(vn), 0.95)
        runs.append((from_dev(g.out), *g.snapshot()))
    for a, b in zip(*runs):
        assert np.array_equal(a, b)
    S = runs[0][3][:, : length + 1].astype(np.float64)
    mass = S.sum(axis=1) - 0.95 * s[:, :length].astype(np.float64).sum(axis=1)
    assert np.all(np.abs(mass - Hq) <= 1e-3 * Hq)
