"""GPU parity of Stage-2 eviction (voxzip_evict_compact) on oracle-supplied
float32 scores: the kept position set is bit-exact, and the compacted rows of
K, V, score and position are bit-exact once keyed by position."""
import numpy as np
import pytest

import oracle
import synth
from vzt import GpuCache, from_dev, to_dev

pytestmark = pytest.mark.gpu


def _check_evict(L, Hkv, d, cap, length, budget, dtype, next_pos, n_sink=4, n_recent=-1, tie_levels=0,
                 seed=0, want_kept=True):
    import torch
    k, v, s, p = synth.random_state(seed, L, Hkv, d, cap, length, dtype, next_pos=next_pos, tie_levels=tie_levels)
    g = GpuCache(L, 8, Hkv, d, cap, dtype) if Hkv <= 8 else GpuCache(L, Hkv, Hkv, d, cap, dtype)
    g.load(k, v, s, p, length, next_pos)
    keep, nl = oracle.evict_select(s.astype(np.float64), p, length, budget, n_sink, n_recent, next_pos)
    kept = torch.full((L, budget), -1, dtype=torch.int32, device="cuda") if want_kept else None
    new_len = g.evict(budget, n_sink=n_sink, n_recent=n_recent, kept=kept)
    assert new_len == nl == min(length, budget)
    K, V, S, P = g.snapshot()
    for l in range(L):
        ref_pos = p[l][keep[l]]
        if want_kept:
            kk = from_dev(kept)[l]
            assert np.array_equal(kk[:nl], ref_pos)
        order = np.argsort(P[l, :nl], kind="stable")
        assert np.array_equal(P[l, :nl][order], ref_pos)
        assert np.array_equal(K[l][:, :nl][:, order], k[l][:, keep[l]])
        assert np.array_equal(V[l][:, :nl][:, order], v[l][:, keep[l]])
        assert np.array_equal(S[l, :nl][order], s[l][keep[l]])
        # kept rows already below the budget did not move
        stay = np.nonzero(np.isin(np.arange(min(budget, length)), keep[l]))[0]
        assert np.array_equal(P[l, stay], p[l, stay])
    return g


@pytest.mark.parametrize("evicted", [1, 2, 5, 8, 9, 16, 100, 700])
@pytest.mark.parametrize("dtype", [synth.DT_BF16, synth.DT_F32])
def test_small_and_radix_paths(evicted, dtype):
    budget = 1000
    _check_evict(3, 4, 128 if dtype == synth.DT_BF16 else 64, 1800, budget + evicted, budget, dtype,
                 next_pos=budget + evicted + 300, seed=evicted)


@pytest.mark.parametrize("tie_levels", [2, 7, 64])
@pytest.mark.parametrize("evicted", [3, 40])
def test_ties_go_to_the_smaller_position(tie_levels, evicted):
    _check_evict(2, 4, 128, 700, 500 + evicted, 500, synth.DT_BF16, next_pos=900, tie_levels=tie_levels,
                 seed=100 + tie_levels)


def test_first_eviction_large():
    """A 64k-token-like first eviction: 13.1k resident tokens down to B = 3277 (20x)."""
    _check_evict(2, 4, 128, 13200, 13107, 3277, synth.DT_BF16, next_pos=13107, seed=7)


@pytest.mark.parametrize("n_sink,n_recent", [(0, -1), (4, 0), (0, 0), (10, 30), (4, 196)])
def test_window_variants(n_sink, n_recent):
    _check_evict(2, 2, 64, 400, 330, 200, synth.DT_BF16, next_pos=600, n_sink=n_sink, n_recent=n_recent,
                 seed=n_sink + 3 * max(n_recent, 0))


def test_no_eviction_reports_positions_and_moves_nothing():
    g = _check_evict(2, 4, 128, 300, 250, 256, synth.DT_BF16, next_pos=400)
    assert g.len == 250


def test_without_kept_output():
    _check_evict(2, 4, 128, 1100, 1050, 1000, synth.DT_BF16, next_pos=1200, want_kept=False)


def test_deterministic_bits():
    a = _check_evict(2, 4, 128, 1800, 1500, 1000, synth.DT_BF16, next_pos=1600, seed=9).snapshot()
    b = _check_evict(2, 4, 128, 1800, 1500, 1000, synth.DT_BF16, next_pos=1600, seed=9).snapshot()
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_worked_selection_from_the_golden_file():
    """The library's eviction on the hand-worked case of
    tests/golden/stage2_select_worked.json (fp32 cache, d = 64, one layer):
    the kept positions and the rows that stay, keyed by position."""
    import json
    import os
    import torch
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "stage2_select_worked.json")))
    x = g["input"]
    n, B = len(x["positions"]), x["budget"]
    k = (np.arange(n * 64, dtype=np.float32).reshape(1, 1, n, 64) + 1.0)
    v = -k
    s = np.array([x["scores"]], dtype=np.float32)
    p = np.array([x["positions"]], dtype=np.int32)
    gc = GpuCache(1, 8, 1, 64, n, synth.DT_F32)
    gc.load(k, v, s, p, n, x["next_pos"])
    kept = torch.full((1, B), -1, dtype=torch.int32, device="cuda")
    assert gc.evict(B, kept=kept) == B
    assert from_dev(kept)[0].tolist() == g["kept_positions"]
    K, V, S, P = gc.snapshot()
    order = np.argsort(P[0, :B], kind="stable")
    assert P[0, :B][order].tolist() == g["kept_positions"]
    want = np.array(g["kept_positions"])
    assert np.array_equal(K[0, 0, :B][order], k[0, 0, want]) and np.array_equal(V[0, 0, :B][order], v[0, 0, want])
    assert np.array_equal(S[0, :B][order], s[0, want])


def _layered(seed, L, Hkv, d, cap, length, next_pos, grid=None):
    """A 48-layer-sized state without drawing every layer (the rolled 4-layer
    state of the whole-range tests); scores optionally put on a grid of
    `grid` levels in [0, 0.5) (many exact ties when grid is small)."""
    from test_gpu_range import layered_state
    k, v, s, p = layered_state(seed, L, Hkv, d, cap, length, synth.DT_BF16, next_pos)
    if grid is not None:
        s = (np.floor(s.astype(np.float64) * 2 * grid) / (2 * grid)).astype(np.float32)
    return k, v, s, p


def _check_kept_rows(l, keep, kept_dev, K, V, S, P, k, v, s_ref, p, nl):
    ref_pos = p[l][keep[l]]
    assert np.array_equal(kept_dev[l, :nl], ref_pos), f"layer {l}: kept position set"
    order = np.argsort(P[l, :nl], kind="stable")
    assert np.array_equal(P[l, :nl][order], ref_pos), f"layer {l}: resident positions"
    assert np.array_equal(K[l][:, :nl][:, order], k[l][:, keep[l]]), f"layer {l}: K rows"
    assert np.array_equal(V[l][:, :nl][:, order], v[l][:, keep[l]]), f"layer {l}: V rows"
    if s_ref is not None:
        assert np.array_equal(S[l, :nl][order], s_ref[l][keep[l]]), f"layer {l}: scores"


@pytest.mark.parametrize("length,budget,grid", [
    (8193, 8192, None),    # E = 1 at the benchmark's length: 16 LDS keys per thread
    (8195, 8192, 64),      # E = 3 with many exact ties
    (8200, 8192, None),    # E = 8: the last block-minimum case
    (12000, 11999, None),  # E = 1 in a 12k-slot layer
    (12000, 11997, 256),   # E = 3, ties
    (12000, 11992, None),  # E = 8
    (16384, 16370, None),  # E = 14: radix select over the largest LDS key array
    (16384, 16000, None),  # E = 384: keys re-read from memory, grid-wide copy
])
def test_headline_size_eviction_against_oracle(length, budget, grid):
    """voxzip_evict_compact at the benchmark's shape (48 layers, 4 KV heads,
    d = 128, bf16) and above it, on the oracle's float32 scores: the kept
    position set of every layer is bit-exact and the compacted rows are
    bit-exact once keyed by position (Sec. 3.2.2, Eq. 7-9)."""
    import torch
    L, Hkv, d = 48, 4, 128
    next_pos = length + 37
    cap = length + 3
    k, v, s, p = _layered(71 + length - budget, L, Hkv, d, cap, length, next_pos, grid)
    g = GpuCache(L, 32, Hkv, d, cap, synth.DT_BF16)
    g.load(k, v, s, p, length, next_pos)
    keep, nl = oracle.evict_select(s.astype(np.float64), p, length, budget, 4, -1, next_pos)
    kept = torch.full((L, budget), -1, dtype=torch.int32, device="cuda")
    assert g.evict(budget, kept=kept) == nl == budget
    K, V, S, P = g.snapshot()
    kd = from_dev(kept)
    for l in range(L):
        _check_kept_rows(l, keep, kd, K, V, S, P, k, v, s, p, nl)


@pytest.mark.parametrize("length,budget,grid", [
    (8192, 8192, None),    # T = 8193, E = 1: the generation step bench.py times
    (8194, 8192, 512),     # E = 3 with exact ties
    (8199, 8192, None),    # E = 8
    (8223, 8215, None),    # T = 8224, the longest single-part cache, E = 9: several minimum rounds + radix
])
def test_generation_step_eviction_against_oracle(length, budget, grid):
    """voxzip_decode_evict (decode, fused score fold and selection) at the
    benchmark's shape, against the oracle's decode step followed by its
    selection.  With q = 0 every query head's softmax is uniform (p = 1/T for
    every key: Eq. 2's closed form), so each key's score grows by the same
    amount; with gamma = 1/2 and old scores on a grid of multiples of 2^-15,
    the fold (one rounding of A/2 + c) keeps the order and the ties of the
    scores exactly, on the GPU as in fp64.  The kept position sets and the
    compacted rows must then equal the oracle's bit for bit, the new scores
    agree within float32 rounding and the outputs are the mean of V."""
    import torch
    import paper_2608_08569_amd as vz
    from vzt import check_close, check_rel, widen
    L, Hq, Hkv, d, dt = 48, 32, 4, 128, synth.DT_BF16
    next_pos = length + 41
    cap = length + 2
    gamma = 0.5
    k, v, s, p = _layered(91 + length - budget, L, Hkv, d, cap, length, next_pos,
                          grid if grid is not None else 1 << 14)
    key = synth.stream_key(93, "gen-step", length, budget)
    q = np.zeros((L, Hq, d), dtype=np.uint16)
    kn = synth.as_storage(synth.normal_f32(synth.stream_key(key, "k"), L * Hkv * d).reshape(L, Hkv, d), dt)
    vn = synth.as_storage(synth.normal_f32(synth.stream_key(key, "v"), L * Hkv * d).reshape(L, Hkv, d), dt)
    # the oracle: decode step (append, attention, fold), then the selection
    ro, rs, rp, _ = oracle.decode_step(q, kn, vn, k, v, s.astype(np.float64), p, length, next_pos, gamma, dt)
    T = length + 1
    keep, nl = oracle.evict_select(rs, rp, T, budget, 4, -1, next_pos + 1)
    k1, v1 = k.copy(), v.copy()
    k1[:, :, length], v1[:, :, length] = kn, vn
    # the library, one call
    g = GpuCache(L, Hq, Hkv, d, cap, dt)
    g.load(k, v, s, p, length, next_pos)
    ws = vz.workspace(vz.VZ_OP_DECODE_EVICT, L, Hq, Hkv, d, cap)
    kept = torch.full((L, budget), -1, dtype=torch.int32, device="cuda")
    new_len = vz.voxzip_decode_evict(to_dev(q), to_dev(kn), to_dev(vn), g.k, g.v, g.score, g.pos, g.out, length,
                                     next_pos, gamma, budget, kept_pos_out=kept, workspace=ws)
    assert new_len == nl == budget
    K, V, S, P = g.snapshot()
    kd = from_dev(kept)
    check_close(widen(from_dev(g.out), dt), ro, 2e-2, "outputs (mean of V)")
    for l in range(L):
        _check_kept_rows(l, keep, kd, K, V, S, P, k1, v1, None, rp, nl)
        order = np.argsort(P[l, :nl], kind="stable")
        check_rel(S[l, :nl][order], rs[l][keep[l]], 1e-5, f"layer {l}: new scores")


def test_empty_cache_with_kept_output():
    """len = 0 with a kept-position output, in a single call and for the first
    sequence of a ragged batch (slot 0 of the planes): nothing is kept, every
    key load stays inside the slots (they are clamped to slot 0), and the
    other sequence is served as usual."""
    import torch
    import paper_2608_08569_amd as vz
    L, Hkv, d, budget = 2, 4, 128, 3
    g = GpuCache(L, 8, Hkv, d, 1, synth.DT_BF16)
    g.pos.fill_(-7)
    kept = torch.full((L, budget), -1, dtype=torch.int32, device="cuda")
    assert vz.voxzip_evict_compact(g.k, g.v, g.score, g.pos, 0, budget, 0, n_sink=1, n_recent=1,
                                   kept_pos_out=kept, workspace=g.ws_ev) == 0
    torch.cuda.synchronize()
    assert (from_dev(kept) == -1).all() and (from_dev(g.pos) == -7).all()
    # ragged: sequence 0 empty at slot 0, sequence 1 with 6 slots and budget 3
    total = 8
    k = torch.zeros(L, Hkv, total, d, dtype=torch.bfloat16, device="cuda")
    v = torch.zeros_like(k)
    s = torch.zeros(L, total, dtype=torch.float32, device="cuda")
    p = torch.full((L, total), -7, dtype=torch.int32, device="cuda")
    p[:, 2:8] = torch.tensor([5, 0, 4, 1, 3, 2], dtype=torch.int32, device="cuda")
    s[:, 2:8] = torch.tensor([0.1, 0.2, 0.3, 0.4, 0.6, 0.5], device="cuda")
    i32 = lambda x: torch.tensor(x, dtype=torch.int32, device="cuda")
    base = torch.tensor([0, 2], dtype=torch.int64, device="cuda")
    kept_r = torch.full((L, total), -1, dtype=torch.int32, device="cuda")
    new_len = i32([9, 9])
    status = i32([9, 9])
    ws = vz.workspace_ragged(vz.VZ_OP_EVICT, L, 8, Hkv, d, total, 2)
    vz.voxzip_evict_compact_ragged(k, v, s, p, base, i32([2, 6]), i32([0, 6]), i32([budget, budget]),
                                   i32([0, 6]), n_sink=1, n_recent=1, kept_pos_out=kept_r, new_len_out=new_len,
                                   status=status, workspace=ws)
    torch.cuda.synchronize()
    assert from_dev(status).tolist() == [0, 0] and from_dev(new_len).tolist() == [0, 3]
    kr = from_dev(kept_r)
    # sequence 1: sink {0}, recent {5}, middle {4, 1, 3, 2} by score: pos 3 (0.6) kept
    assert (kr[:, :2] == -1).all() and (kr[:, 2:5] == [0, 3, 5]).all()
    assert (from_dev(p)[:, :2] == -7).all()
