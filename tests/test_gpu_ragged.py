"""GPU parity of the ragged twins (voxzip_*_ragged).  Every sequence of a
packed batch is checked against the fp64 oracle and, bit for bit, against the
single-sequence entry point run on a copy of the same data; slots outside
every sequence stay untouched; a sequence with out-of-range values is skipped
and its status says why."""
import numpy as np
import pytest

import oracle
import synth
from vzt import RTOL, GpuCache, check_close, check_rel, from_dev, to_dev, widen

pytestmark = pytest.mark.gpu


def torch():
    import torch as t
    return t


class Packed:
    """Placement of a ragged batch: sequence s owns slots base[s] .. base[s] +
    cap[s] - 1 of planes of `total` slots; sequences sit in a shuffled order
    with `gap` unused slots around each."""

    def __init__(self, caps, gap, seed):
        n = len(caps)
        order = np.argsort(synth.uniform01(synth.stream_key(seed, "pack-order", n), 0, n), kind="stable")
        self.base = np.zeros(n, dtype=np.int64)
        at = gap
        for s in order:
            self.base[s] = at
            at += int(caps[s]) + gap
        self.caps = np.asarray(caps, dtype=np.int32)
        self.total = at
        self.owned = np.zeros(self.total, dtype=bool)
        for s in range(n):
            self.owned[self.base[s]: self.base[s] + self.caps[s]] = True

    def sl(self, s):
        return slice(int(self.base[s]), int(self.base[s] + self.caps[s]))

    def dev(self):
        t = torch()
        return (t.from_numpy(self.base.copy()).cuda(), t.from_numpy(self.caps.copy()).cuda())


def _storage_noise(seed, shape, dtype):
    x = synth.normal_f32(synth.stream_key(seed, "noise", *shape), int(np.prod(shape))).reshape(shape)
    return synth.as_storage(x, dtype)


def _packed_state(pk, L, Hkv, d, dtype, lens, next_pos, seed):
    """Packed K, V, scores, positions: every sequence a random resident state,
    the gaps noise (K/V) and sentinels (score -7, position -5)."""
    n = len(lens)
    K = _storage_noise(seed, (L, Hkv, pk.total, d), dtype)
    V = _storage_noise(seed + 1, (L, Hkv, pk.total, d), dtype)
    S = np.full((L, pk.total), -7.0, dtype=np.float32)
    P = np.full((L, pk.total), -5, dtype=np.int32)
    for s in range(n):
        k, v, sc, p = synth.random_state(seed * 1000 + s, L, Hkv, d, int(pk.caps[s]), int(lens[s]), dtype,
                                         next_pos=int(next_pos[s]))
        K[:, :, pk.sl(s)], V[:, :, pk.sl(s)], S[:, pk.sl(s)], P[:, pk.sl(s)] = k, v, sc, p
    return K, V, S, P


def _i32(a):
    return torch().tensor(np.asarray(a, dtype=np.int32), device="cuda")


def _run_decode_case(dtype, d, Hq, Hkv, lens, L=2, steps=2, seed=0, gamma=0.95):
    t = torch()
    import paper_2608_08569_amd as vz
    n = len(lens)
    lens = np.asarray(lens, dtype=np.int64)
    next_pos = lens + 3 * np.arange(n)
    caps = lens + steps + 1 + (np.arange(n) * 7) % 5
    pk = Packed(caps, gap=5, seed=seed)
    K, V, S, P = _packed_state(pk, L, Hkv, d, dtype, lens, next_pos, seed)
    Kd, Vd = to_dev(K), to_dev(V)
    Sd, Pd = to_dev(S), to_dev(P)
    base_d, cap_d = pk.dev()
    len_d, next_d = _i32(lens), _i32(next_pos)
    status = _i32(np.full(n, -99))
    tdt = t.float32 if dtype == synth.DT_F32 else t.bfloat16
    out_d = t.zeros(n, L, Hq, d, dtype=tdt, device="cuda")
    ws = vz.workspace_ragged(vz.VZ_OP_DECODE, L, Hq, Hkv, d, pk.total, n)
    for step in range(steps):
        key = synth.stream_key(seed, "ragged-decode", step)
        q = _storage_noise(key, (n, L, Hq, d), dtype)
        kn = _storage_noise(key + 1, (n, L, Hkv, d), dtype)
        vn = _storage_noise(key + 2, (n, L, Hkv, d), dtype)
        t.cuda.synchronize()
        K0, V0, S0, P0 = from_dev(Kd), from_dev(Vd), from_dev(Sd), from_dev(Pd)
        vz.voxzip_decode_attend_score_ragged(to_dev(q), to_dev(kn), to_dev(vn), Kd, Vd, Sd, Pd, out_d, base_d,
                                             cap_d, len_d, next_d, gamma, status=status, workspace=ws)
        t.cuda.synchronize()
        K1, V1, S1, P1, out = from_dev(Kd), from_dev(Vd), from_dev(Sd), from_dev(Pd), from_dev(out_d)
        assert np.all(from_dev(status) == vz.VZ_OK)
        for s in range(n):
            sl, ln, npos = pk.sl(s), int(lens[s]), int(next_pos[s])
            ref_o, ref_s, ref_p, _ = oracle.decode_step(q[s], kn[s], vn[s], K0[:, :, sl], V0[:, :, sl],
                                                        S0[:, sl].astype(np.float64), P0[:, sl], ln, npos,
                                                        gamma, dtype)
            check_close(widen(out[s], dtype), ref_o, RTOL[dtype], f"seq {s} output")
            check_rel(S1[:, sl][:, : ln + 1], ref_s, RTOL[dtype], f"seq {s} score")
            assert np.array_equal(P1[:, sl][:, : ln + 1], ref_p)
            # the single-sequence entry point on the same data gives the same bits
            g = GpuCache(L, Hq, Hkv, d, int(pk.caps[s]), dtype)
            g.load(K0[:, :, sl], V0[:, :, sl], S0[:, sl], P0[:, sl], ln, npos)
            g.step(to_dev(q[s]), to_dev(kn[s]), to_dev(vn[s]), gamma)
            Kg, Vg, Sg, Pg = g.snapshot()
            assert np.array_equal(from_dev(g.out), out[s]), f"seq {s} output differs from the single call"
            assert np.array_equal(Sg, S1[:, sl]) and np.array_equal(Pg, P1[:, sl])
            assert np.array_equal(Kg, K1[:, :, sl]) and np.array_equal(Vg, V1[:, :, sl])
        gap = ~pk.owned
        assert np.array_equal(K1[:, :, gap], K0[:, :, gap]) and np.array_equal(V1[:, :, gap], V0[:, :, gap])
        assert np.array_equal(S1[:, gap], S0[:, gap]) and np.array_equal(P1[:, gap], P0[:, gap])
        len_d += 1
        next_d += 1
        lens += 1
        next_pos += 1


LENS = [0, 1, 5, 127, 128, 129, 255, 256, 700, 1500]


@pytest.mark.parametrize("Hq,Hkv", [(32, 4), (8, 8), (16, 2)])
def test_ragged_decode_fused_path(Hq, Hkv):
    _run_decode_case(synth.DT_BF16, 128, Hq, Hkv, LENS, seed=Hq + Hkv)


@pytest.mark.parametrize("dtype,d,Hq,Hkv", [(synth.DT_F32, 64, 8, 2), (synth.DT_BF16, 128, 64, 4),
                                            (synth.DT_BF16, 64, 8, 1), (synth.DT_F32, 128, 4, 4)])
def test_ragged_decode_generic_path(dtype, d, Hq, Hkv):
    _run_decode_case(dtype, d, Hq, Hkv, LENS[::2] + [300], seed=7 + Hq)


def test_ragged_decode_finishing_launches_agree():
    """Planes of more than 128 chunks take the output and fold kernels, smaller
    ones one finishing kernel that forms the layer statistics itself: the
    300-key sequence's ragged call (a 17,300-slot plane, two launches) gives
    the bits of its single call (one launch), and so does the long one."""
    _run_decode_case(synth.DT_BF16, 128, 32, 4, [300, 17000], steps=1, seed=12)


def test_ragged_decode_new_row_at_every_tile_row():
    """Lengths 224..255 put the new K/V row of Eq. (1) in each of the 32 rows
    of a wave's tile on the chunked path (2 layers x 4 KV heads): the wave
    holding it takes it into its tile registers after its loads and writes
    it to the cache from there; every sequence against the oracle and, bit
    for bit, against its single-sequence call."""
    _run_decode_case(synth.DT_BF16, 128, 32, 4, list(range(224, 256)), steps=1, seed=21)


def test_ragged_decode_one_sequence_and_gamma_edges():
    _run_decode_case(synth.DT_BF16, 128, 32, 4, [2000], steps=1, gamma=1.0, seed=3)
    _run_decode_case(synth.DT_BF16, 128, 32, 4, [9, 300], steps=1, gamma=0.0, seed=4)


def test_ragged_decode_skips_invalid_sequences():
    """Sequences 1-5 carry out-of-range values and sequence 6 is an idle slot
    (capacity 0); they are reported and nothing of them is touched, while
    sequence 0 is served normally."""
    t = torch()
    import paper_2608_08569_amd as vz
    L, Hq, Hkv, d, dtype = 2, 32, 4, 128, synth.DT_BF16
    lens = np.array([100, 200, 50, 300, 40, 60, 80], dtype=np.int64)
    next_pos = lens + 1
    caps = lens + 8
    pk = Packed(caps, gap=4, seed=5)
    K, V, S, P = _packed_state(pk, L, Hkv, d, dtype, lens, next_pos, 5)
    Kd, Vd, Sd, Pd = to_dev(K), to_dev(V), to_dev(S), to_dev(P)
    base_d, cap_d = pk.dev()
    len_d, next_d = _i32(lens), _i32(next_pos)
    cap_d[1] = 200                       # no free slot: len == cap
    base_d[2] = pk.total - 10            # runs past the planes
    next_d[3] = -1                       # negative position
    len_d[4] = 2 ** 31 - 1               # len + 1 would overflow
    len_d[5] = -1
    cap_d[6] = 0                         # an idle batch slot
    expect = [vz.VZ_OK, vz.VZ_ERR_CAPACITY, vz.VZ_ERR_INVALID, vz.VZ_ERR_INVALID, vz.VZ_ERR_CAPACITY,
              vz.VZ_ERR_INVALID, vz.VZ_IDLE]
    n = len(lens)
    key = synth.stream_key(5, "ragged-invalid")
    q = _storage_noise(key, (n, L, Hq, d), dtype)
    kn = _storage_noise(key + 1, (n, L, Hkv, d), dtype)
    vn = _storage_noise(key + 2, (n, L, Hkv, d), dtype)
    out_d = t.full((n, L, Hq, d), 3.0, dtype=t.bfloat16, device="cuda")
    status = _i32(np.full(n, -99))
    ws = vz.workspace_ragged(vz.VZ_OP_DECODE, L, Hq, Hkv, d, pk.total, n)
    vz.voxzip_decode_attend_score_ragged(to_dev(q), to_dev(kn), to_dev(vn), Kd, Vd, Sd, Pd, out_d, base_d, cap_d,
                                         len_d, next_d, 0.95, status=status, workspace=ws)
    t.cuda.synchronize()
    assert from_dev(status).tolist() == expect
    out = from_dev(out_d)
    K1, V1, S1, P1 = from_dev(Kd), from_dev(Vd), from_dev(Sd), from_dev(Pd)
    for s in range(1, n):
        assert np.all(widen(out[s], dtype) == 3.0), f"seq {s} output written"
        sl = pk.sl(s)
        assert np.array_equal(K1[:, :, sl], K[:, :, sl]) and np.array_equal(V1[:, :, sl], V[:, :, sl])
        assert np.array_equal(S1[:, sl], S[:, sl]) and np.array_equal(P1[:, sl], P[:, sl])
    sl, ln = pk.sl(0), int(lens[0])
    ref_o, ref_s, ref_p, _ = oracle.decode_step(q[0], kn[0], vn[0], K[:, :, sl], V[:, :, sl],
                                                S[:, sl].astype(np.float64), P[:, sl], ln, int(next_pos[0]), 0.95,
                                                dtype)
    check_close(widen(out[0], dtype), ref_o, RTOL[dtype], "valid sequence output")
    check_rel(S1[:, sl][:, : ln + 1], ref_s, RTOL[dtype], "valid sequence score")


def _run_evict_case(dtype, d, Hkv, cases, L=2, seed=0, n_sink=4, n_recent=-1, want_kept=True):
    """cases: (length, budget, next_pos) per sequence."""
    t = torch()
    import paper_2608_08569_amd as vz
    n = len(cases)
    lens = np.array([c[0] for c in cases], dtype=np.int64)
    budgets = np.array([c[1] for c in cases], dtype=np.int64)
    next_pos = np.array([c[2] for c in cases], dtype=np.int64)
    caps = np.maximum(lens, 1) + 3
    pk = Packed(caps, gap=3, seed=seed)
    K, V, S, P = _packed_state(pk, L, Hkv, d, dtype, lens, next_pos, seed)
    Kd, Vd, Sd, Pd = to_dev(K), to_dev(V), to_dev(S), to_dev(P)
    base_d, cap_d = pk.dev()
    kept_d = t.full((L, pk.total), -1, dtype=t.int32, device="cuda") if want_kept else None
    new_len_d = _i32(np.full(n, -9))
    status = _i32(np.full(n, -99))
    ws = vz.workspace_ragged(vz.VZ_OP_EVICT, L, 8, Hkv, d, pk.total, n)
    vz.voxzip_evict_compact_ragged(Kd, Vd, Sd, Pd, base_d, cap_d, _i32(lens), _i32(budgets), _i32(next_pos),
                                   n_sink=n_sink, n_recent=n_recent, kept_pos_out=kept_d, new_len_out=new_len_d,
                                   status=status, workspace=ws)
    t.cuda.synchronize()
    assert np.all(from_dev(status) == vz.VZ_OK)
    K1, V1, S1, P1 = from_dev(Kd), from_dev(Vd), from_dev(Sd), from_dev(Pd)
    kept_all = from_dev(kept_d) if want_kept else None
    new_len = from_dev(new_len_d)
    for s in range(n):
        sl, ln, B, npos = pk.sl(s), int(lens[s]), int(budgets[s]), int(next_pos[s])
        keep, nl = oracle.evict_select(S[:, sl].astype(np.float64), P[:, sl], ln, B, n_sink, n_recent, npos)
        assert new_len[s] == nl == min(ln, B)
        for l in range(L):
            ref_pos = P[l, sl][keep[l]]
            if want_kept:
                assert np.array_equal(kept_all[l, sl][:nl], ref_pos), f"seq {s} kept positions"
            order = np.argsort(P1[l, sl][:nl], kind="stable")
            assert np.array_equal(P1[l, sl][:nl][order], ref_pos)
            assert np.array_equal(K1[l][:, sl][:, :nl][:, order], K[l][:, sl][:, keep[l]])
            assert np.array_equal(V1[l][:, sl][:, :nl][:, order], V[l][:, sl][:, keep[l]])
            assert np.array_equal(S1[l, sl][:nl][order], S[l, sl][keep[l]])
        # the single-sequence entry point on the same data gives the same bits
        g = GpuCache(L, 8, Hkv, d, int(pk.caps[s]), dtype)
        g.load(K[:, :, sl], V[:, :, sl], S[:, sl], P[:, sl], ln, npos)
        kg = t.full((L, B), -1, dtype=t.int32, device="cuda") if want_kept else None
        assert g.evict(B, n_sink=n_sink, n_recent=n_recent, kept=kg) == nl
        Kg, Vg, Sg, Pg = g.snapshot()
        assert np.array_equal(Kg, K1[:, :, sl]) and np.array_equal(Vg, V1[:, :, sl])
        assert np.array_equal(Sg, S1[:, sl]) and np.array_equal(Pg, P1[:, sl])
        if want_kept:
            assert np.array_equal(from_dev(kg)[:, :nl], kept_all[:, sl][:, :nl])
    gap = ~pk.owned
    assert np.array_equal(K1[:, :, gap], K[:, :, gap]) and np.array_equal(S1[:, gap], S[:, gap])
    assert np.array_equal(P1[:, gap], P[:, gap])
    if want_kept:
        assert np.all(kept_all[:, gap] == -1)


def test_ragged_evict_paths():
    """One batch covering no eviction, the block-minimum rounds (1 and 8
    evictions), the radix select (9), a copy-kernel compaction (300 moved
    rows) and a sequence whose keys do not fit in LDS (17000 slots)."""
    cases = [(500, 600, 520), (1001, 1000, 1200), (1008, 1000, 1100), (1009, 1000, 1300), (1300, 1000, 1400),
             (17000, 16990, 17050), (40, 40, 40)]
    _run_evict_case(synth.DT_BF16, 128, 4, cases, seed=1)


@pytest.mark.parametrize("dtype,d", [(synth.DT_F32, 64), (synth.DT_BF16, 64)])
def test_ragged_evict_dtypes_and_windows(dtype, d):
    cases = [(300, 200, 400), (64, 60, 64), (900, 100, 950)]
    _run_evict_case(dtype, d, 2, cases, seed=2, n_sink=2, n_recent=10)
    _run_evict_case(dtype, d, 2, cases, seed=3, want_kept=False)


def test_ragged_evict_skips_invalid_sequences():
    t = torch()
    import paper_2608_08569_amd as vz
    L, Hkv, d, dtype = 2, 4, 128, synth.DT_BF16
    lens = np.array([300, 300, 300, 300, 300, 300], dtype=np.int64)
    next_pos = lens + 10
    pk = Packed(lens + 2, gap=2, seed=9)
    K, V, S, P = _packed_state(pk, L, Hkv, d, dtype, lens, next_pos, 9)
    Kd, Vd, Sd, Pd = to_dev(K), to_dev(V), to_dev(S), to_dev(P)
    base_d, cap_d = pk.dev()
    budget = _i32([200, 0, 200, 200, 200, 200])  # seq 1: budget < 1
    len_d = _i32(lens)
    len_d[2] = 303                              # len > cap
    nxt = _i32(next_pos)
    nxt[3] = 100                                # next_pos < len
    base_d[4] = -1
    cap_d[5] = 0                                # an idle batch slot
    status = _i32(np.full(6, -99))
    new_len = _i32(np.full(6, -9))
    ws = vz.workspace_ragged(vz.VZ_OP_EVICT, L, 8, Hkv, d, pk.total, 6)
    vz.voxzip_evict_compact_ragged(Kd, Vd, Sd, Pd, base_d, cap_d, len_d, budget, nxt, new_len_out=new_len,
                                   status=status, workspace=ws)
    t.cuda.synchronize()
    assert from_dev(status).tolist() == [vz.VZ_OK, vz.VZ_ERR_INVALID, vz.VZ_ERR_CAPACITY, vz.VZ_ERR_INVALID,
                                         vz.VZ_ERR_INVALID, vz.VZ_IDLE]
    assert from_dev(new_len).tolist() == [200, 300, 303, 300, 300, 300]
    K1, S1, P1 = from_dev(Kd), from_dev(Sd), from_dev(Pd)
    for s in range(1, 6):
        sl = pk.sl(s)
        assert np.array_equal(K1[:, :, sl], K[:, :, sl]) and np.array_equal(S1[:, sl], S[:, sl])
        assert np.array_equal(P1[:, sl], P[:, sl])
    sl = pk.sl(0)
    keep, nl = oracle.evict_select(S[:, sl].astype(np.float64), P[:, sl], 300, 200, 4, -1, int(next_pos[0]))
    for l in range(L):
        assert np.array_equal(np.sort(P1[l, sl][:nl]), P[l, sl][keep[l]])


def _run_fuse_case(dtype, d, T_ins, L=2, H=2, seed=0, anchor=False, max_spans=None):
    t = torch()
    import paper_2608_08569_amd as vz
    n = len(T_ins)
    offs = []
    for s, T in enumerate(T_ins):
        lens = synth.spans_geometric(synth.stream_key(seed, "ragged-fuse", s), T, 0.25, 32) if T > 0 else \
            np.zeros(0, dtype=np.int64)
        offs.append(synth.offsets_from_lengths(lens))
    n_spans = np.array([len(o) - 1 for o in offs], dtype=np.int64)
    pin = Packed(np.maximum(T_ins, 1), gap=3, seed=seed + 1)
    k_in = _storage_noise(seed + 2, (L, H, pin.total, d), dtype)
    v_in = _storage_noise(seed + 3, (L, H, pin.total, d), dtype)
    # offsets of all sequences in one array, with a gap before each
    off_base = np.zeros(n, dtype=np.int64)
    flat = []
    at = 0
    for s in range(n):
        flat.append(np.full(2, -3, dtype=np.int32))
        at += 2
        off_base[s] = at
        flat.append(offs[s].astype(np.int32))
        at += len(offs[s])
    flat = np.concatenate(flat)
    caps = n_spans + 1 + np.arange(n) % 3
    pk = Packed(caps, gap=2, seed=seed + 4)
    ak = av = None
    if anchor:
        ak = _storage_noise(seed + 5, (L, H, pk.total, d), dtype)
        av = _storage_noise(seed + 6, (L, H, pk.total, d), dtype)
    sentinel = 5.0
    tdt = t.float32 if dtype == synth.DT_F32 else t.bfloat16
    ko = t.full((L, H, pk.total, d), sentinel, dtype=tdt, device="cuda")
    vo = t.full((L, H, pk.total, d), sentinel, dtype=tdt, device="cuda")
    so = t.full((L, pk.total), -1.0, dtype=t.float32, device="cuda")
    po = t.full((L, pk.total), -5, dtype=t.int32, device="cuda")
    base_d, cap_d = pk.dev()
    status = _i32(np.full(n, -99))
    vz.voxzip_fuse_spans_ragged(to_dev(k_in), to_dev(v_in), t.from_numpy(pin.base.copy()).cuda(), _i32(T_ins),
                                to_dev(flat), t.from_numpy(off_base).cuda(), _i32(n_spans),
                                int(n_spans.max()) if max_spans is None else max_spans, ko, vo, so, po, base_d,
                                cap_d, status=status, anchor_k=None if ak is None else to_dev(ak),
                                anchor_v=None if av is None else to_dev(av))
    t.cuda.synchronize()
    K, V, S, P = from_dev(ko), from_dev(vo), from_dev(so), from_dev(po)
    return dict(pk=pk, pin=pin, offs=offs, n_spans=n_spans, k_in=k_in, v_in=v_in, ak=ak, av=av, K=K, V=V, S=S,
                P=P, status=from_dev(status), sentinel=sentinel)


@pytest.mark.parametrize("dtype,d", [(synth.DT_BF16, 128), (synth.DT_F32, 64)])
@pytest.mark.parametrize("anchor", [False, True])
def test_ragged_fuse_matches_oracle_and_single_calls(dtype, d, anchor):
    t = torch()
    import paper_2608_08569_amd as vz
    T_ins = np.array([1, 40, 300, 129, 1000, 7], dtype=np.int64)
    r = _run_fuse_case(dtype, d, T_ins, seed=11 + d, anchor=anchor)
    assert np.all(r["status"] == vz.VZ_OK)
    pk, pin = r["pk"], r["pin"]
    L, H = r["K"].shape[:2]
    for s in range(len(T_ins)):
        n, off = int(r["n_spans"][s]), r["offs"][s]
        x_sl = slice(int(pin.base[s]), int(pin.base[s] + T_ins[s]))
        o_sl = slice(int(pk.base[s]), int(pk.base[s] + n))
        for name, x_in, got, a in (("K", r["k_in"], r["K"], r["ak"]), ("V", r["v_in"], r["V"], r["av"])):
            ref = oracle.fuse(x_in[:, :, x_sl], off, dtype, anchor=None if a is None else a[:, :, o_sl])
            check_close(widen(got[:, :, o_sl], dtype), ref, RTOL[dtype], f"seq {s} fused {name}")
        assert np.array_equal(r["P"][:, o_sl], np.broadcast_to(np.arange(n, dtype=np.int32), (L, n)))
        assert np.all(r["S"][:, o_sl] == 0.0)
        # single-sequence call on the same input: same bits
        g = GpuCache(L, H, H, d, int(pk.caps[s]), dtype)
        g.k.fill_(r["sentinel"])
        g.v.fill_(r["sentinel"])
        g.fuse(to_dev(np.ascontiguousarray(r["k_in"][:, :, x_sl])), to_dev(np.ascontiguousarray(r["v_in"][:, :, x_sl])),
               to_dev(off), None if r["ak"] is None else to_dev(np.ascontiguousarray(r["ak"][:, :, o_sl])),
               None if r["av"] is None else to_dev(np.ascontiguousarray(r["av"][:, :, o_sl])))
        Kg, Vg, _, _ = g.snapshot()
        assert np.array_equal(Kg[:, :, :n], r["K"][:, :, o_sl]) and np.array_equal(Vg[:, :, :n], r["V"][:, :, o_sl])
    # every slot no sequence wrote keeps its sentinel
    written = np.zeros(pk.total, dtype=bool)
    for s in range(len(T_ins)):
        written[int(pk.base[s]): int(pk.base[s] + r["n_spans"][s])] = True
    assert np.all(widen(r["K"][:, :, ~written], dtype) == r["sentinel"])
    assert np.all(r["P"][:, ~written] == -5) and np.all(r["S"][:, ~written] == -1.0)


def test_ragged_fuse_reports_sequences_over_the_span_bound():
    import paper_2608_08569_amd as vz
    T_ins = np.array([64, 400, 32], dtype=np.int64)
    r = _run_fuse_case(synth.DT_BF16, 128, T_ins, seed=21, max_spans=40)
    n = r["n_spans"]
    expect = [vz.VZ_OK if n[s] <= 40 else vz.VZ_ERR_CAPACITY for s in range(3)]
    assert r["status"].tolist() == expect and expect.count(vz.VZ_ERR_CAPACITY) >= 1
    pk = r["pk"]
    for s in range(3):
        if expect[s] != vz.VZ_OK:
            o_sl = pk.sl(s)
            assert np.all(widen(r["K"][:, :, o_sl], synth.DT_BF16) == r["sentinel"])


def test_batch16_ragged_calls():
    """The batched workload through the ragged twins: the 16 sequences (2k-32k
    audio tokens, budget len/4, eviction every 16 steps) in one packed cache
    at the real head shape, on the first 2 of the 48 layers; one fusion call,
    then 32 decode steps of one call each (two evictions), every sequence
    checked against the oracle every step, state-synced."""
    t = torch()
    import paper_2608_08569_amd as vz
    layers = range(2)
    L = len(layers)
    ws_list = synth.batch_workloads()
    w0 = ws_list[0]
    n = len(ws_list)
    offs = [synth.offsets_from_lengths(synth.span_lengths(w, seq=i)) for i, w in enumerate(ws_list)]
    n_spans = np.array([len(o) - 1 for o in offs], dtype=np.int64)
    budgets = np.array([w.budget for w in ws_list], dtype=np.int64)
    T_ins = np.array([w.n_audio + w.n_text for w in ws_list], dtype=np.int64)
    caps = np.maximum(n_spans, budgets) + w0.interval + 1
    pk = Packed(caps, gap=0, seed=0)
    pin = Packed(T_ins, gap=0, seed=1)
    Hq, Hkv, d = w0.n_q_heads, w0.kv_heads, w0.d
    k_in = np.zeros((L, Hkv, pin.total, d), dtype=np.uint16)
    v_in = np.zeros_like(k_in)
    for i, w in enumerate(ws_list):
        k_in[:, :, pin.sl(i)] = synth.prefill_kv(w, "k", seq=i, layers=layers)
        v_in[:, :, pin.sl(i)] = synth.prefill_kv(w, "v", seq=i, layers=layers)
    off_base = np.concatenate([[0], np.cumsum(n_spans + 1)[:-1]]).astype(np.int64)
    flat = np.concatenate(offs).astype(np.int32)
    Kd = t.zeros(L, Hkv, pk.total, d, dtype=t.bfloat16, device="cuda")
    Vd = t.zeros_like(Kd)
    Sd = t.zeros(L, pk.total, dtype=t.float32, device="cuda")
    Pd = t.zeros(L, pk.total, dtype=t.int32, device="cuda")
    base_d, cap_d = pk.dev()
    status = _i32(np.full(n, -99))
    vz.voxzip_fuse_spans_ragged(to_dev(k_in), to_dev(v_in), t.from_numpy(pin.base.copy()).cuda(), _i32(T_ins),
                                to_dev(flat), t.from_numpy(off_base).cuda(), _i32(n_spans), int(n_spans.max()),
                                Kd, Vd, Sd, Pd, base_d, cap_d, status=status)
    t.cuda.synchronize()
    assert np.all(from_dev(status) == vz.VZ_OK)
    del k_in, v_in
    lens, next_pos = n_spans.copy(), n_spans.copy()
    len_d, next_d, bud_d = _i32(lens), _i32(next_pos), _i32(budgets)
    new_len_d = _i32(np.zeros(n))
    out_d = t.zeros(n, L, Hq, d, dtype=t.bfloat16, device="cuda")
    ws_dec = vz.workspace_ragged(vz.VZ_OP_DECODE, L, Hq, Hkv, d, pk.total, n)
    ws_ev = vz.workspace_ragged(vz.VZ_OP_EVICT, L, Hq, Hkv, d, pk.total, n)
    for step in range(32):
        ins = [synth.decode_inputs(w, step, seq=i) for i, w in enumerate(ws_list)]
        q = np.stack([x[0][:L] for x in ins])
        kn = np.stack([x[1][:L] for x in ins])
        vn = np.stack([x[2][:L] for x in ins])
        t.cuda.synchronize()
        K0, V0, S0, P0 = from_dev(Kd), from_dev(Vd), from_dev(Sd), from_dev(Pd)
        vz.voxzip_decode_attend_score_ragged(to_dev(q), to_dev(kn), to_dev(vn), Kd, Vd, Sd, Pd, out_d, base_d,
                                             cap_d, len_d, next_d, w0.gamma, status=status, workspace=ws_dec)
        t.cuda.synchronize()
        assert np.all(from_dev(status) == vz.VZ_OK)
        out, S1, P1 = from_dev(out_d), from_dev(Sd), from_dev(Pd)
        ref_scores = []
        for i in range(n):
            sl, ln = pk.sl(i), int(lens[i])
            ref_o, ref_s, ref_p, _ = oracle.decode_step(q[i], kn[i], vn[i], K0[:, :, sl], V0[:, :, sl],
                                                        S0[:, sl].astype(np.float64), P0[:, sl], ln,
                                                        int(next_pos[i]), w0.gamma, w0.dtype)
            check_close(widen(out[i], w0.dtype), ref_o, RTOL[w0.dtype], f"seq {i} step {step} output")
            check_rel(S1[:, sl][:, : ln + 1], ref_s, RTOL[w0.dtype], f"seq {i} step {step} score")
            assert np.array_equal(P1[:, sl][:, : ln + 1], ref_p)
            ref_scores.append(ref_s)
        len_d += 1
        next_d += 1
        lens += 1
        next_pos += 1
        if (step + 1) % w0.interval == 0:
            # select on the oracle's float32 scores so that a near tie cannot flip the kept set
            sc = S1.copy()
            for i in range(n):
                sc[:, int(pk.base[i]): int(pk.base[i] + lens[i])] = ref_scores[i].astype(np.float32)
            Sd.copy_(t.from_numpy(sc))
            K2, V2, P2 = from_dev(Kd), from_dev(Vd), from_dev(Pd)
            vz.voxzip_evict_compact_ragged(Kd, Vd, Sd, Pd, base_d, cap_d, len_d, bud_d, next_d,
                                           new_len_out=new_len_d, status=status, workspace=ws_ev)
            t.cuda.synchronize()
            assert np.all(from_dev(status) == vz.VZ_OK)
            K3, V3, S3, P3 = from_dev(Kd), from_dev(Vd), from_dev(Sd), from_dev(Pd)
            for i in range(n):
                sl, ln, B = pk.sl(i), int(lens[i]), int(budgets[i])
                keep, nl = oracle.evict_select(sc[:, sl].astype(np.float64), P2[:, sl], ln, B, 4, -1,
                                               int(next_pos[i]))
                for l in range(L):
                    order = np.argsort(P3[l, sl][:nl], kind="stable")
                    assert np.array_equal(P3[l, sl][:nl][order], P2[l, sl][keep[l]])
                    assert np.array_equal(K3[l][:, sl][:, :nl][:, order], K2[l][:, sl][:, keep[l]])
                    assert np.array_equal(V3[l][:, sl][:, :nl][:, order], V2[l][:, sl][:, keep[l]])
                    assert np.array_equal(S3[l, sl][:nl][order], sc[l, sl][keep[l]])
                lens[i] = nl
            assert np.array_equal(from_dev(new_len_d), lens)
            len_d.copy_(new_len_d)
    assert np.array_equal(lens, np.minimum(n_spans + 32, budgets))


def test_ragged_many_sequences():
    """150 short sequences (the lookup scans 64 sequences per round, so three
    rounds), lengths 0..300 including 0, 127 and 128: decode against the oracle
    and the single call, then eviction against the oracle, every sequence."""
    key = synth.stream_key(41, "many")
    n = 150
    lens = synth.uniform_int(key, 0, n, 0, 300).astype(np.int64)
    lens[:4] = [0, 127, 128, 1]
    _run_decode_case(synth.DT_BF16, 128, 32, 4, lens.tolist(), L=1, steps=1, seed=41)
    budgets = np.maximum(lens // 2, 8)
    cases = [(int(x), int(b), int(x) + 3) for x, b in zip(lens, budgets)]
    _run_evict_case(synth.DT_BF16, 128, 4, cases, L=1, seed=42)
