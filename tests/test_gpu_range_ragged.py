"""GPU parity of the ragged decode call on the whole-range path (bf16, d = 128,
at least 128 (layer, KV head) items): one order
launch ranks the sequences' parts longest first (up to 1024 sequences; in
sequence order beyond), one workgroup per (part, layer, KV head), then the
merge of sequences in parts and the fold.  Every
sequence is checked against the fp64 oracle on sampled layers and, bit for
bit on every layer, against the single-sequence call on a copy of its data;
slots outside every sequence stay untouched; the workspace starts filled
with garbage (it needs no initialisation)."""
import numpy as np
import pytest

import oracle
import synth
from test_gpu_range import layered_state
from test_gpu_ragged import Packed, _i32
from vzt import RTOL, GpuCache, check_close, check_rel, from_dev, to_dev, widen

pytestmark = pytest.mark.gpu

DT, D = synth.DT_BF16, 128


def torch():
    import torch as t
    return t


def _packed(pk, L, Hkv, lens, next_pos, seed):
    """Every sequence a layered random state; the gaps a sentinel pattern
    (K 0x4040, V 0xC040, score -7, position -5)."""
    K = np.full((L, Hkv, pk.total, D), 0x4040, dtype=np.uint16)
    V = np.full_like(K, 0xC040)
    S = np.full((L, pk.total), -7.0, dtype=np.float32)
    P = np.full((L, pk.total), -5, dtype=np.int32)
    for s in range(len(lens)):
        k, v, sc, p = layered_state(seed * 1000 + s, L, Hkv, D, int(pk.caps[s]), int(lens[s]), DT,
                                    int(next_pos[s]))
        K[:, :, pk.sl(s)], V[:, :, pk.sl(s)], S[:, pk.sl(s)], P[:, pk.sl(s)] = k, v, sc, p
    return K, V, S, P


def _inputs(seed, step, n, L, Hq, Hkv):
    key = synth.stream_key(seed, "ragged-range", step)
    mk = lambda tag, shape: synth.as_storage(
        synth.normal_f32(synth.stream_key(key, tag), int(np.prod(shape))).reshape(shape) * np.float32(1.7), DT)
    return mk("q", (n, L, Hq, D)), mk("k", (n, L, Hkv, D)), mk("v", (n, L, Hkv, D))


def run_ragged(Hq, Hkv, L, lens, layers, steps=1, seed=0, gap=3, gamma=0.95, single_check=None):
    """Decode steps of a packed batch through the ragged call; every sequence
    against the oracle on `layers` and (those in `single_check`, default all)
    bit for bit against the single-sequence call."""
    t = torch()
    import paper_2608_08569_amd as vz
    n = len(lens)
    lens = np.asarray(lens, dtype=np.int64)
    next_pos = lens + 2 * np.arange(n) + 1
    caps = lens + steps + 1 + (np.arange(n) * 5) % 3
    pk = Packed(caps, gap=gap, seed=seed)
    K, V, S, P = _packed(pk, L, Hkv, lens, next_pos, seed)
    Kd, Vd, Sd, Pd = to_dev(K), to_dev(V), to_dev(S), to_dev(P)
    del K, V
    base_d, cap_d = pk.dev()
    len_d, next_d = _i32(lens), _i32(next_pos)
    status = _i32(np.full(n, -99))
    out_d = t.zeros(n, L, Hq, D, dtype=t.bfloat16, device="cuda")
    ws = vz.workspace_ragged(vz.VZ_OP_DECODE, L, Hq, Hkv, D, pk.total, n)
    ws.fill_(0x7F)
    checked = range(n) if single_check is None else single_check
    for step in range(steps):
        q, kn, vn = _inputs(seed, step, n, L, Hq, Hkv)
        t.cuda.synchronize()
        K0, V0, S0, P0 = from_dev(Kd), from_dev(Vd), from_dev(Sd), from_dev(Pd)
        vz.voxzip_decode_attend_score_ragged(to_dev(q), to_dev(kn), to_dev(vn), Kd, Vd, Sd, Pd, out_d, base_d,
                                             cap_d, len_d, next_d, gamma, status=status, workspace=ws)
        t.cuda.synchronize()
        K1, V1, S1, P1, out = from_dev(Kd), from_dev(Vd), from_dev(Sd), from_dev(Pd), from_dev(out_d)
        assert np.all(from_dev(status) == vz.VZ_OK)
        for s in range(n):
            sl, ln, npos = pk.sl(s), int(lens[s]), int(next_pos[s])
            ref_o, ref_s, ref_p, _ = oracle.decode_step(q[s][layers], kn[s][layers], vn[s][layers],
                                                        K0[layers][:, :, sl], V0[layers][:, :, sl],
                                                        S0[layers][:, sl].astype(np.float64), P0[layers][:, sl],
                                                        ln, npos, gamma, DT)
            check_close(widen(out[s][layers], DT), ref_o, RTOL[DT], f"seq {s} (len {ln}) output")
            check_rel(S1[layers][:, sl][:, : ln + 1], ref_s, RTOL[DT], f"seq {s} (len {ln}) score")
            assert np.array_equal(P1[layers][:, sl][:, : ln + 1], ref_p)
            assert np.array_equal(K1[:, :, sl][:, :, ln], kn[s]) and np.array_equal(V1[:, :, sl][:, :, ln], vn[s])
            if s in checked:
                g = GpuCache(L, Hq, Hkv, D, int(pk.caps[s]), DT)
                g.load(K0[:, :, sl], V0[:, :, sl], S0[:, sl], P0[:, sl], ln, npos)
                g.step(to_dev(q[s]), to_dev(kn[s]), to_dev(vn[s]), gamma)
                Kg, Vg, Sg, Pg = g.snapshot()
                assert np.array_equal(from_dev(g.out), out[s]), f"seq {s} output differs from the single call"
                assert np.array_equal(Sg, S1[:, sl]) and np.array_equal(Pg, P1[:, sl])
                assert np.array_equal(Kg, K1[:, :, sl]) and np.array_equal(Vg, V1[:, :, sl])
                del g, Kg, Vg
        gap_m = ~pk.owned
        assert np.array_equal(K1[:, :, gap_m], K0[:, :, gap_m]) and np.array_equal(V1[:, :, gap_m], V0[:, :, gap_m])
        assert np.array_equal(S1[:, gap_m], S0[:, gap_m]) and np.array_equal(P1[:, gap_m], P0[:, gap_m])
        del K0, V0, K1, V1
        len_d += 1
        next_d += 1
        lens += 1
        next_pos += 1


def test_ragged_range_mixed_lengths():
    """Empty to 12000 resident keys in one batch: one-part sequences (up to
    the 8224-key maximum) next to sequences in 2 parts; two steps, so the
    8223-key sequence moves into parts on the second; layers 0, 13, 31."""
    run_ragged(32, 4, 32, [0, 1, 127, 1000, 8223, 8224, 12000, 300], layers=[0, 13, 31], steps=2, seed=1)


@pytest.mark.parametrize("Hq,Hkv,L,lens", [
    (64, 8, 16, [3, 2500, 9000, 128]),
    (8, 1, 128, [700, 8300, 40]),
    (12, 2, 64, [5000, 1, 129]),
])
def test_ragged_range_head_groups(Hq, Hkv, L, lens):
    """8, 8 and 6 query heads per KV head over 8, 1 and 2 KV heads."""
    run_ragged(Hq, Hkv, L, lens, layers=[0, L // 2, L - 1], seed=Hq + Hkv)


def test_ragged_range_many_sequences():
    """150 sequences of 0 to 300 keys (many ties in the order, the fold
    table spread over the whole block); layers 0 and 31; the single-call
    comparison on every tenth sequence."""
    key = synth.stream_key(43, "many-range")
    n = 150
    lens = synth.uniform_int(key, 0, n, 0, 300).astype(np.int64)
    lens[:5] = [0, 127, 128, 1, 255]
    run_ragged(32, 4, 32, lens.tolist(), layers=[0, 31], seed=43, single_check=set(range(0, n, 10)))


def test_ragged_range_more_sequences_than_one_order_block():
    """1100 sequences of 0 to 40 keys (more than the 1024 the order kernel
    ranks: sequence order, a block scan over runs of two sequences); layers
    0 and 31; the single-call comparison on every fiftieth sequence."""
    key = synth.stream_key(47, "more-seqs")
    n = 1100
    lens = synth.uniform_int(key, 0, n, 0, 40).astype(np.int64)
    lens[:3] = [0, 40, 1]
    run_ragged(32, 4, 32, lens.tolist(), layers=[0, 31], seed=47, gap=1, single_check=set(range(0, n, 50)))


def test_ragged_range_gamma_edges():
    run_ragged(32, 4, 32, [2000, 9000], layers=[0, 31], gamma=1.0, seed=5)
    run_ragged(32, 4, 32, [9, 300], layers=[0, 31], gamma=0.0, seed=6)


def test_ragged_range_skips_invalid_and_overflowing_sequences():
    """A sequence with no free slot, one outside the planes and an idle slot
    are skipped (status says why, nothing of theirs written); two sequences over the
    same 20000 slots need more fold blocks than the table holds (the tables
    are sized for sequences that do not overlap): the first in the order
    (the smaller index, as the parts are alike) is served, the other
    reported."""
    t = torch()
    import paper_2608_08569_amd as vz
    L, Hq, Hkv = 32, 32, 4
    # sequence 0: full (len = cap); 1: fine; 2: base past the planes; 3: an idle slot (cap 0)
    caps = np.array([50, 400, 60, 70])
    pk = Packed(caps, gap=2, seed=3)
    lens = np.array([50, 399, 10, 20])
    next_pos = lens + 4
    K, V, S, P = _packed(pk, L, Hkv, np.minimum(lens, caps - 1), next_pos, 3)
    Kd, Vd, Sd, Pd = to_dev(K), to_dev(V), to_dev(S), to_dev(P)
    base = pk.base.copy()
    base[2] = pk.total - 5
    base_d = t.from_numpy(base).cuda()
    cap_d = t.from_numpy(pk.caps.copy()).cuda()
    cap_d[3] = 0
    status = _i32(np.full(4, -99))
    q, kn, vn = _inputs(3, 0, 4, L, Hq, Hkv)
    out_d = t.zeros(4, L, Hq, D, dtype=t.bfloat16, device="cuda")
    ws = vz.workspace_ragged(vz.VZ_OP_DECODE, L, Hq, Hkv, D, pk.total, 4)
    ws.fill_(0x55)
    vz.voxzip_decode_attend_score_ragged(to_dev(q), to_dev(kn), to_dev(vn), Kd, Vd, Sd, Pd, out_d, base_d, cap_d,
                                         _i32(lens), _i32(next_pos), 0.95, status=status, workspace=ws)
    t.cuda.synchronize()
    st = from_dev(status)
    assert st.tolist() == [vz.VZ_ERR_CAPACITY, vz.VZ_OK, vz.VZ_ERR_INVALID, vz.VZ_IDLE]
    assert not from_dev(out_d)[3].any()
    K1, S1, P1 = from_dev(Kd), from_dev(Sd), from_dev(Pd)
    for s in (0, 2, 3):
        sl = pk.sl(s)
        assert np.array_equal(K1[:, :, sl], K[:, :, sl]) and np.array_equal(S1[:, sl], S[:, sl])
        assert np.array_equal(P1[:, sl], P[:, sl])
    sl = pk.sl(1)
    ref_o, ref_s, ref_p, _ = oracle.decode_step(q[1][[0, 31]], kn[1][[0, 31]], vn[1][[0, 31]], K[[0, 31]][:, :, sl],
                                                V[[0, 31]][:, :, sl], S[[0, 31]][:, sl].astype(np.float64),
                                                P[[0, 31]][:, sl], 399, int(next_pos[1]), 0.95, DT)
    check_close(widen(from_dev(out_d)[1][[0, 31]], DT), ref_o, RTOL[DT], "output")
    check_rel(S1[[0, 31]][:, sl][:, :400], ref_s, RTOL[DT], "score")
    del K, V, Kd, Vd

    # two sequences over the same slots: 20001 keys each
    total = 20010
    cap = 20005
    lens = np.array([20000, 20000])
    k, v, sc, p = layered_state(8, L, Hkv, D, cap, 20000, DT, 20003)
    Kd = t.zeros(L, Hkv, total, D, dtype=t.bfloat16, device="cuda")
    Vd = t.zeros_like(Kd)
    Sd = t.zeros(L, total, dtype=t.float32, device="cuda")
    Pd = t.zeros(L, total, dtype=t.int32, device="cuda")
    Kd[:, :, :cap].copy_(to_dev(k))
    Vd[:, :, :cap].copy_(to_dev(v))
    Sd[:, :cap].copy_(t.from_numpy(sc))
    Pd[:, :cap].copy_(t.from_numpy(p))
    base_d = t.zeros(2, dtype=t.int64, device="cuda")
    cap_d = _i32([cap, cap])
    status = _i32(np.full(2, -99))
    q, kn, vn = _inputs(8, 0, 2, L, Hq, Hkv)
    out_d = t.zeros(2, L, Hq, D, dtype=t.bfloat16, device="cuda")
    ws = vz.workspace_ragged(vz.VZ_OP_DECODE, L, Hq, Hkv, D, total, 2)
    ws.fill_(0x33)
    vz.voxzip_decode_attend_score_ragged(to_dev(q), to_dev(kn), to_dev(vn), Kd, Vd, Sd, Pd, out_d, base_d, cap_d,
                                         _i32(lens), _i32([20003, 20003]), 0.95, status=status, workspace=ws)
    t.cuda.synchronize()
    st = from_dev(status)
    assert st[0] == vz.VZ_OK and st[1] == vz.VZ_ERR_CAPACITY
    ls = [0, 31]
    ref_o, ref_s, ref_p, _ = oracle.decode_step(q[0][ls], kn[0][ls], vn[0][ls], k[ls], v[ls],
                                                sc[ls].astype(np.float64), p[ls], 20000, 20003, 0.95, DT)
    check_close(widen(from_dev(out_d)[0][ls], DT), ref_o, RTOL[DT], "output")
    check_rel(from_dev(Sd)[ls][:, :20001], ref_s, RTOL[DT], "score")
    assert np.array_equal(from_dev(Pd)[ls][:, :20001], ref_p)
    assert not from_dev(out_d)[1].any()


def test_batch16_full_size_sampled_layers():
    """The batched workload at full size, in the launch configuration bench.py
    times: its 16 sequences' span counts (1,280 to 8,077 resident keys), 48
    layers, 32Q/4KV, one ragged call per step on the whole-range path (3,072
    range workgroups); two steps; every sequence against the oracle on layers
    0, 23 and 47, three sequences bit for bit on every layer against their
    single calls.  The device state is written sequence by sequence, so the
    host holds one sequence's layers at a time."""
    t = torch()
    import paper_2608_08569_amd as vz
    ws_list = synth.batch_workloads()
    w0 = ws_list[0]
    L, Hq, Hkv = w0.n_layers, w0.n_q_heads, w0.kv_heads
    n = len(ws_list)
    lens = np.array([len(synth.offsets_from_lengths(synth.span_lengths(w, seq=i))) - 1
                     for i, w in enumerate(ws_list)], dtype=np.int64)
    caps = np.maximum(lens, [w.budget for w in ws_list]) + w0.interval + 1
    next_pos = lens.copy()
    pk = Packed(caps, gap=0, seed=0)
    Kd = t.empty(L, Hkv, pk.total, D, dtype=t.bfloat16, device="cuda")
    Vd = t.empty_like(Kd)
    Sd = t.empty(L, pk.total, dtype=t.float32, device="cuda")
    Pd = t.empty(L, pk.total, dtype=t.int32, device="cuda")
    for s in range(n):
        k, v, sc, p = layered_state(60 + s, L, Hkv, D, int(caps[s]), int(lens[s]), DT, int(next_pos[s]))
        sl = pk.sl(s)
        Kd[:, :, sl].copy_(to_dev(k))
        Vd[:, :, sl].copy_(to_dev(v))
        Sd[:, sl].copy_(t.from_numpy(sc))
        Pd[:, sl].copy_(t.from_numpy(p))
        del k, v
    base_d, cap_d = pk.dev()
    len_d, next_d = _i32(lens), _i32(next_pos)
    status = _i32(np.full(n, -99))
    out_d = t.zeros(n, L, Hq, D, dtype=t.bfloat16, device="cuda")
    ws = vz.workspace_ragged(vz.VZ_OP_DECODE, L, Hq, Hkv, D, pk.total, n)
    ls = [0, 23, 47]
    whole = [2, 9, 15]  # shortest, a middle one, longest
    for step in range(2):
        q, kn, vn = _inputs(61, step, n, L, Hq, Hkv)
        t.cuda.synchronize()
        K0, V0 = from_dev(Kd[ls]), from_dev(Vd[ls])
        S0, P0 = from_dev(Sd), from_dev(Pd)
        before = {s: (from_dev(Kd[:, :, pk.sl(s)]), from_dev(Vd[:, :, pk.sl(s)])) for s in whole}
        vz.voxzip_decode_attend_score_ragged(to_dev(q), to_dev(kn), to_dev(vn), Kd, Vd, Sd, Pd, out_d, base_d,
                                             cap_d, len_d, next_d, w0.gamma, status=status, workspace=ws)
        t.cuda.synchronize()
        assert np.all(from_dev(status) == vz.VZ_OK)
        out, S1, P1 = from_dev(out_d), from_dev(Sd), from_dev(Pd)
        for s in range(n):
            sl, ln, npos = pk.sl(s), int(lens[s]), int(next_pos[s])
            ref_o, ref_s, ref_p, _ = oracle.decode_step(q[s][ls], kn[s][ls], vn[s][ls], K0[:, :, sl], V0[:, :, sl],
                                                        S0[ls][:, sl].astype(np.float64), P0[ls][:, sl], ln, npos,
                                                        w0.gamma, DT)
            check_close(widen(out[s][ls], DT), ref_o, RTOL[DT], f"step {step} seq {s} output")
            check_rel(S1[ls][:, sl][:, : ln + 1], ref_s, RTOL[DT], f"step {step} seq {s} score")
            assert np.array_equal(P1[ls][:, sl][:, : ln + 1], ref_p)
        for s in whole:
            sl, ln, npos = pk.sl(s), int(lens[s]), int(next_pos[s])
            g = GpuCache(L, Hq, Hkv, D, int(caps[s]), DT)
            g.load(before[s][0], before[s][1], S0[:, sl], P0[:, sl], ln, npos)
            g.step(to_dev(q[s]), to_dev(kn[s]), to_dev(vn[s]), w0.gamma)
            Kg, Vg, Sg, Pg = g.snapshot()
            assert np.array_equal(from_dev(g.out), out[s]), f"step {step} seq {s}: output differs from the single call"
            assert np.array_equal(Sg, S1[:, sl]) and np.array_equal(Pg, P1[:, sl])
            assert np.array_equal(Kg, from_dev(Kd[:, :, sl])) and np.array_equal(Vg, from_dev(Vd[:, :, sl]))
            del g, Kg, Vg
        del before, K0, V0
        len_d += 1
        next_d += 1
        lens += 1
        next_pos += 1


def test_ragged_range_calls_on_two_streams():
    """Two packed batches decoded at the same time on two streams, each with
    its own workspace, give the bits of the same calls run one after the
    other: the path keeps all of its state in the workspace, and no
    workgroup waits for another."""
    t = torch()
    import paper_2608_08569_amd as vz
    L, Hq, Hkv = 32, 32, 4
    batches = []
    for seed, lens in ((71, [300, 5000, 9000, 17]), (72, [8000, 64, 2500])):
        lens = np.asarray(lens, dtype=np.int64)
        n = len(lens)
        next_pos = lens + 5
        caps = lens + 3
        pk = Packed(caps, gap=2, seed=seed)
        K, V, S, P = _packed(pk, L, Hkv, lens, next_pos, seed)
        q, kn, vn = _inputs(seed, 0, n, L, Hq, Hkv)
        batches.append(dict(pk=pk, state=(K, V, S, P), ins=(q, kn, vn), lens=lens, next_pos=next_pos, n=n))

    def run(streams):
        outs = []
        for b, st in zip(batches, streams):
            K, V, S, P = b["state"]
            d = dict(K=to_dev(K), V=to_dev(V), S=to_dev(S), P=to_dev(P),
                     out=t.zeros(b["n"], L, Hq, D, dtype=t.bfloat16, device="cuda"),
                     ws=vz.workspace_ragged(vz.VZ_OP_DECODE, L, Hq, Hkv, D, b["pk"].total, b["n"]),
                     ins=[to_dev(x) for x in b["ins"]], base_cap=b["pk"].dev(), len=_i32(b["lens"]),
                     nxt=_i32(b["next_pos"]))
            outs.append(d)
        t.cuda.synchronize()
        for d, st in zip(outs, streams):
            with t.cuda.stream(st):
                vz.voxzip_decode_attend_score_ragged(*d["ins"], d["K"], d["V"], d["S"], d["P"], d["out"],
                                                     d["base_cap"][0], d["base_cap"][1], d["len"], d["nxt"], 0.95,
                                                     workspace=d["ws"], stream=st)
            if len(set(streams)) == 1:
                t.cuda.synchronize()
        t.cuda.synchronize()
        return [tuple(from_dev(d[k]) for k in ("out", "K", "V", "S", "P")) for d in outs]

    s0 = t.cuda.current_stream()
    seq = run([s0, s0])
    par = run([t.cuda.Stream(), t.cuda.Stream()])
    for a, b in zip(seq, par):
        for x, y in zip(a, b):
            assert np.array_equal(x, y)
