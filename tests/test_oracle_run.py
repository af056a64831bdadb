"""Pins of the oracle's end-to-end driver (``oracle.Run``: Stage-1 fusion, then
decode steps, with the Stage-2 eviction after the score update every
`interval` steps when the cache is over budget; Sec. 3.2.1 Eq. 4, Sec. 3.1
Eq. 1-2, Sec. 3.2.2 Eq. 6-9 in that order), of its row gather (the Eq. 7-8
concatenation) and of its storage rounding.

The driver is checked against a model of the method kept by POSITION rather
than by slot: every token ever seen is a dict entry (its K and V rows and its
decayed score), attention is a numpy softmax over the resident positions, and
the eviction sorts the middle positions by (score descending, position
ascending).  The two share nothing but the inputs, so a wrong gather (rows of
one array moved without another), a wrong trigger step or an eviction taken
before the score update makes them disagree."""
import numpy as np
import pytest

import oracle
import synth


class PositionModel:
    """Sec. 3.1-3.2 written per position: tokens[pos] = (K [Hkv][d], V), score[pos]."""

    def __init__(self, k_rows, v_rows, Hq, gamma, budget, n_sink=4, n_recent=None, interval=1):
        n = k_rows.shape[1]
        self.K = {j: k_rows[:, j].astype(np.float64) for j in range(n)}
        self.V = {j: v_rows[:, j].astype(np.float64) for j in range(n)}
        self.A = {j: 0.0 for j in range(n)}
        self.resident = list(range(n))
        self.next_pos = n
        self.Hq, self.gamma, self.budget = Hq, gamma, budget
        self.n_sink = n_sink
        self.M = budget // 5 if n_recent is None else n_recent
        self.interval = interval
        self.t = 0
        self.evictions = []

    def step(self, q, kn, vn):
        """q [Hq][d], kn/vn [Hkv][d] (float64)."""
        p_new = self.next_pos
        self.K[p_new], self.V[p_new], self.A[p_new] = kn, vn, 0.0
        self.resident.append(p_new)
        self.next_pos += 1
        Hkv, d = kn.shape
        G = self.Hq // Hkv
        Ks = np.stack([self.K[j] for j in self.resident], axis=1)   # [Hkv][T][d]
        Vs = np.stack([self.V[j] for j in self.resident], axis=1)
        out = np.zeros((self.Hq, d))
        mass = np.zeros(len(self.resident))
        for h in range(self.Hq):
            s = Ks[h // G] @ q[h] / np.sqrt(d)
            e = np.exp(s - s.max())
            p = e / e.sum()
            out[h] = p @ Vs[h // G]
            mass += p
        for i, j in enumerate(self.resident):
            self.A[j] = self.gamma * self.A[j] + mass[i]
        self.t += 1
        if self.t % self.interval == 0 and len(self.resident) > self.budget:
            sinks = [j for j in self.resident if j < self.n_sink]
            recent = [j for j in self.resident if j >= self.next_pos - self.M and j >= self.n_sink]
            middle = [j for j in self.resident if j not in sinks and j not in recent]
            n_top = self.budget - len(sinks) - len(recent)
            top = sorted(middle, key=lambda j: (-self.A[j], j))[:n_top]
            gone = sorted(set(self.resident) - set(sinks) - set(recent) - set(top))
            self.evictions.append((self.t - 1, gone))
            self.resident = sorted(sinks + top + recent)
        return out


def _run_pair(seed, n, steps, budget, gamma, interval, Hq=4, Hkv=2, d=16):
    """The oracle's driver and the position model over the same fp32 inputs
    (length-1 spans, so the fused cache is the prefill cache itself)."""
    key = synth.stream_key(seed, "run-pin", n, steps, budget, interval)
    nrm = lambda tag, shape: synth.normal_f32(synth.stream_key(key, tag), int(np.prod(shape))).reshape(shape)
    k_in, v_in = nrm("k", (1, Hkv, n, d)), nrm("v", (1, Hkv, n, d))
    off = np.arange(n + 1, dtype=np.int32)
    run = oracle.Run(k_in, v_in, off, oracle.F32, Hq, n + steps + 1, gamma, budget, interval=interval)
    model = PositionModel(k_in[0], v_in[0], Hq, gamma, budget, interval=interval)
    for t in range(steps):
        q, kn, vn = nrm(f"q{t}", (1, Hq, d)), nrm(f"kn{t}", (1, Hkv, d)), nrm(f"vn{t}", (1, Hkv, d))
        o_run = run.step(q, kn, vn)
        o_mod = model.step(q[0].astype(np.float64), kn[0].astype(np.float64), vn[0].astype(np.float64))
        yield t, run, model, o_run[0], o_mod


def _check_state(t, run, model):
    assert run.len == len(model.resident), f"step {t}: resident count"
    assert run.next_pos == model.next_pos
    P = run.pos[0, : run.len]
    assert sorted(P.tolist()) == model.resident, f"step {t}: resident positions"
    for i, j in enumerate(P):
        assert np.array_equal(run.k[0][:, i], model.K[j].astype(np.float32)), f"step {t}: K row of position {j}"
        assert np.array_equal(run.v[0][:, i], model.V[j].astype(np.float32)), f"step {t}: V row of position {j}"
        assert abs(run.score[0, i] - model.A[j]) <= 1e-12 * max(1.0, abs(model.A[j])), f"step {t}: score of {j}"


@pytest.mark.parametrize("gamma", [0.0, 0.9])
def test_run_matches_position_model_every_step(gamma):
    """Interval 1: one eviction per step once over budget.  With gamma = 0 the
    kept middle is the top-N of the current step's attention alone, so taking
    the eviction before the score update would keep other positions."""
    n, budget = 40, 36
    for t, run, model, o_run, o_mod in _run_pair(1, n, 14, budget, gamma, interval=1):
        np.testing.assert_allclose(o_run, o_mod, rtol=1e-10, atol=1e-12)
        _check_state(t, run, model)
    assert len(model.evictions) == 14
    assert model.evictions[0] == (0, model.evictions[0][1]) and len(model.evictions[0][1]) == n + 1 - budget


@pytest.mark.parametrize("interval", [3, 5])
def test_run_interval_rule(interval):
    """Eviction fires exactly after the steps t with (t + 1) % interval == 0
    and len > B, down to B, and never in between (reading C13)."""
    n, budget, steps = 30, 31, 17
    lens = []
    for t, run, model, o_run, o_mod in _run_pair(2, n, steps, budget, 0.8, interval=interval):
        _check_state(t, run, model)
        lens.append(run.len)
    want, length = [], n
    for t in range(steps):
        length += 1
        if (t + 1) % interval == 0 and length > budget:
            length = budget
        want.append(length)
    assert lens == want
    fired = [t for t, _ in model.evictions]
    assert fired == [t for t in range(steps) if (t + 1) % interval == 0 and t >= 1]


def test_run_fuses_with_the_pinned_fusion_and_rounds_to_storage():
    """With real spans in bfloat16, the driver's initial cache is the fused
    rows of oracle.fuse rounded to bfloat16 (nearest-even through float32),
    scores 0, positions 0..n-1, and its first step equals oracle.decode_step
    from that state."""
    import torch
    Hq, Hkv, d = 4, 1, 64
    key = synth.stream_key(3, "run-fuse")
    lens = synth.spans_geometric(key, 300, p=0.25, max_len=16)
    off = synth.offsets_from_lengths(lens)
    n = len(lens)
    k_in = synth.as_storage(synth.normal_f32(synth.stream_key(key, "k"), 300 * d).reshape(1, Hkv, 300, d), 1)
    v_in = synth.as_storage(synth.normal_f32(synth.stream_key(key, "v"), 300 * d).reshape(1, Hkv, 300, d), 1)
    run = oracle.Run(k_in, v_in, off, oracle.BF16, Hq, n + 4, 0.95, n + 10)
    to_bf16 = lambda x: torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy() \
        .view(np.uint16)
    assert np.array_equal(run.k[:, :, :n], to_bf16(oracle.fuse(k_in, off, oracle.BF16)))
    assert np.array_equal(run.v[:, :, :n], to_bf16(oracle.fuse(v_in, off, oracle.BF16)))
    assert not run.score.any() and run.pos[0, :n].tolist() == list(range(n)) and run.len == n
    q = synth.as_storage(synth.normal_f32(synth.stream_key(key, "q"), Hq * d).reshape(1, Hq, d), 1)
    kn = synth.as_storage(synth.normal_f32(synth.stream_key(key, "kn"), Hkv * d).reshape(1, Hkv, d), 1)
    vn = synth.as_storage(synth.normal_f32(synth.stream_key(key, "vn"), Hkv * d).reshape(1, Hkv, d), 1)
    ref_o, ref_s, ref_p, _ = oracle.decode_step(q, kn, vn, run.k.copy(), run.v.copy(), run.score.copy(),
                                                run.pos.copy(), n, n, 0.95, oracle.BF16)
    o = run.step(q, kn, vn)
    assert np.array_equal(o, ref_o) and np.array_equal(run.score[:, : n + 1], ref_s)
    assert np.array_equal(run.pos[:, : n + 1], ref_p)


def test_gather_rows_concatenates_by_keep_list():
    """Eq. 7-8: row i of the result is row keep[i] of the input, per layer,
    for K/V planes [L][H][cap][d] and for per-slot arrays [L][cap]."""
    x = np.arange(2 * 3 * 6 * 2).reshape(2, 3, 6, 2)
    keep = np.array([[5, 0, 2], [1, 3, 4]])
    g = oracle.gather_rows(x, keep)
    assert g.shape == (2, 3, 3, 2)
    for l in range(2):
        for h in range(3):
            for i in range(3):
                assert np.array_equal(g[l, h, i], x[l, h, keep[l, i]])
    y = np.arange(12).reshape(2, 6) * 10
    assert oracle.gather_rows(y, keep).tolist() == [[50, 0, 20], [70, 90, 100]]


def test_round_store_nearest_even():
    """float64 -> float32 -> bfloat16, each step to nearest, ties to even:
    crafted halfway cases, and torch's own float32 -> bfloat16 conversion
    (round to nearest even) on random values."""
    import torch
    one = 1.0
    cases = {
        one + 2.0 ** -8: 0x3F80,                 # halfway between 1 and 1 + 2^-7: to 1 (even)
        one + 3 * 2.0 ** -8: 0x3F82,             # halfway between 1 + 2^-7 and 1 + 2^-6: to the even one
        one + 2.0 ** -8 + 2.0 ** -20: 0x3F81,    # just above halfway: up
        -(one + 2.0 ** -8): 0xBF80,
        -(one + 3 * 2.0 ** -8): 0xBF82,
        2.0 ** -130: 0x0000 | (1 << 3),          # a float32 subnormal survives as a bf16 subnormal
        0.0: 0x0000,
    }
    x = np.array(list(cases), dtype=np.float64)
    got = oracle._round_store(x, oracle.BF16)
    assert got.dtype == np.uint16
    assert [int(b) for b in got] == list(cases.values())
    # the float32 step alone: 1 + 2^-24 is halfway between float32 1 and 1 + 2^-23
    assert oracle._round_store(np.array([one + 2.0 ** -24, one + 3 * 2.0 ** -24]), oracle.F32).tolist() == \
        [1.0, float(np.float32(one + 2.0 ** -22))]
    r = synth.normal_f32(synth.stream_key(4, "round"), 4096).astype(np.float64) * 3.7
    r += synth.normal_f32(synth.stream_key(5, "round"), 4096).astype(np.float64) * 1e-9
    ref = torch.from_numpy(r.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(oracle._round_store(r, oracle.BF16), ref)
