"""Pins of the oracle's Stage-2 eviction (Sec. 3.2.2, Eq. 7-9): brute force on
tiny inputs, the no-op and StreamingLLM special cases, and invariants."""
import itertools

import numpy as np
import pytest

import oracle
import synth


def _brute_keep(score, pos, length, budget, n_sink, M, next_pos):
    """Enumerate every subset of the middle of the right size; keep the one
    with the largest score sum, ties to the lexicographically smallest sorted
    position list (smaller positions win)."""
    slots = list(range(length))
    sink = [j for j in slots if pos[j] < n_sink]
    recent = [j for j in slots if pos[j] >= next_pos - M and pos[j] >= n_sink]
    mid = [j for j in slots if j not in sink and j not in recent]
    n_top = budget - len(sink) - len(recent)
    best = None
    for sub in itertools.combinations(mid, n_top):
        total = sum(score[j] for j in sub)
        key = (-total, sorted(pos[j] for j in sub))
        if best is None or key < best[0]:
            best = (key, sub)
    kept = sink + list(best[1]) + recent
    return sorted(kept, key=lambda j: pos[j])


@pytest.mark.parametrize("seed", range(12))
def test_brute_force_tiny(seed):
    length = 8 + seed % 7            # 8 .. 14
    budget = 5 + seed % 4            # M = 1
    next_pos = length + 3 * (seed % 3)
    _, _, score, pos = synth.random_state(seed, 1, 1, 4, 16, length, 0, next_pos=next_pos,
                                          tie_levels=(4 if seed % 2 else 0))
    M = budget // 5
    # use exact binary fractions so the brute-force sums are exact
    sc = np.round(score.astype(np.float64) * 64) / 64
    keep, nl = oracle.evict_select(sc, pos, length, budget, 4, -1, next_pos)
    ref = _brute_keep(sc[0], pos[0], length, budget, 4, M, next_pos)
    assert nl == budget
    assert keep[0].tolist() == ref


def test_budget_at_or_above_length_keeps_everything():
    _, _, score, pos = synth.random_state(1, 2, 1, 4, 64, 50, 0, next_pos=80)
    for budget in (50, 51, 64):
        keep, nl = oracle.evict_select(score, pos, 50, budget, 4, -1, 80)
        assert nl == 50
        for l in range(2):
            assert sorted(keep[l].tolist()) == list(range(50))
            assert np.all(np.diff(pos[l][keep[l]]) > 0)


def test_no_history_budget_is_streaming_sinks_plus_recent():
    # N = B - T - M = 0: only the sink and recent windows survive
    length, next_pos, budget, M = 60, 200, 24, 20
    _, _, score, pos = synth.random_state(2, 1, 1, 4, 64, length, 0, next_pos=next_pos)
    keep, nl = oracle.evict_select(score, pos, length, budget, 4, M, next_pos)
    kept_pos = pos[0][keep[0]].tolist()
    assert kept_pos == [0, 1, 2, 3] + list(range(next_pos - M, next_pos))


@pytest.mark.parametrize("tie_levels", [0, 3, 50])
def test_invariants_and_sorted_order(tie_levels):
    length, next_pos, budget = 300, 1000, 100
    _, _, score, pos = synth.random_state(3, 3, 1, 4, 320, length, 0, next_pos=next_pos,
                                          tie_levels=tie_levels)
    keep, nl = oracle.evict_select(score, pos, length, budget, 4, -1, next_pos)
    M = budget // 5
    assert nl == budget
    for l in range(3):
        kp = pos[l][keep[l]]
        assert np.all(np.diff(kp) > 0)                      # ascending positions
        assert set(range(4)) <= set(kp.tolist())            # sinks
        assert set(range(next_pos - M, next_pos)) <= set(kp.tolist())  # recent
        mid_kept = [j for j in keep[l] if 4 <= pos[l][j] < next_pos - M]
        mid_all = [j for j in range(length) if 4 <= pos[l][j] < next_pos - M]
        dropped = sorted(set(mid_all) - set(mid_kept))
        # every kept middle slot outranks every dropped one under (score desc, pos asc)
        worst_kept = max(((-score[l][j], pos[l][j]) for j in mid_kept))
        best_dropped = min(((-score[l][j], pos[l][j]) for j in dropped))
        assert worst_kept < best_dropped


def test_rejects_windows_larger_than_budget():
    _, _, score, pos = synth.random_state(4, 1, 1, 4, 64, 50, 0, next_pos=50)
    with pytest.raises(ValueError):
        oracle.evict_select(score, pos, 50, 20, 4, 17, 50)


def _golden_select():
    import json
    import os
    return json.load(open(os.path.join(os.path.dirname(__file__), "golden", "stage2_select_worked.json")))


def test_worked_selection_from_the_golden_file():
    """The kept set worked out by hand in tests/golden/stage2_select_worked.json
    (three scores tie for the last two places: the smaller positions win)."""
    g = _golden_select()
    x = g["input"]
    score = np.array([x["scores"]], dtype=np.float32).astype(np.float64)
    pos = np.array([x["positions"]], dtype=np.int32)
    keep, nl = oracle.evict_select(score, pos, len(x["positions"]), x["budget"], 4, -1, x["next_pos"])
    assert nl == x["budget"]
    assert pos[0][keep[0]].tolist() == g["kept_positions"]
