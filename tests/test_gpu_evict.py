"""GPU parity of Stage-2 eviction (voxzip_evict_compact) on oracle-supplied
float32 scores: the kept position set is bit-exact, and the compacted rows of
K, V, score and position are bit-exact once keyed by position."""
import numpy as np
import pytest

import oracle
import synth
from vzt import GpuCache, from_dev

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
