"""Continuous batching in the decode loop (paper_2608_08569_amd.loop): requests
join the running batch in free slots (Stage-1 fusion of their prefill into
the slot, Sec. 3.2.1) and leave it when they finish, between steps, while the
other sequences keep decoding (Sec. 3.1 Eq. 1-2, Sec. 3.2.2 Eq. 6-9).  Every
request's outputs, scores, positions and cache rows are bit-identical, step
after step, to the same request run alone through the single-sequence entry
points with its own eviction schedule; its fused prefill and its first step
match the oracle.  Eagerly launched steps and HIP-graph replays (captured
once, before any request joins) give the same bits."""
import numpy as np
import pytest

import oracle
import synth
from vzt import RTOL, GpuCache, check_close, check_rel, from_dev, to_dev, widen

pytestmark = pytest.mark.gpu

HQ, HKV, D = 32, 4, 128
INTERVAL = 4
GAMMA = 0.95
DT = synth.DT_BF16
# request: (prefill tokens, budget, decode steps, slot, first global step)
REQUESTS = [(1200, 256, 6, 0, 0), (700, 160, 10, 1, 0), (2500, 600, 8, 0, 6), (400, 80, 7, 2, 3),
            (900, 200, 5, 1, 10)]


def _request(i, L):
    T_in, budget, steps, slot, start = REQUESTS[i]
    key = synth.stream_key(11, "batching", i)
    off = synth.offsets_from_lengths(synth.spans_geometric(synth.stream_key(key, "spans"), T_in, 0.25, 32))
    x = synth.normal_f32(synth.stream_key(key, "kv"), 2 * L * HKV * T_in * D)
    kv = synth.as_storage(x.reshape(2, L, HKV, T_in, D), DT)
    return off, kv[0], kv[1]


def _step_inputs(i, t, L):
    key = synth.stream_key(12, "batching-step", i, t)
    mk = lambda tag, shape: synth.as_storage(
        synth.normal_f32(synth.stream_key(key, tag), int(np.prod(shape))).reshape(shape), DT)
    return mk("q", (L, HQ, D)), mk("k", (L, HKV, D)), mk("v", (L, HKV, D))


def _solo(i, L):
    """Request i alone on the single-sequence entry points: outputs per step
    and the state after each step."""
    import torch
    off, k_in, v_in = _request(i, L)
    T_in, budget, steps, _, _ = REQUESTS[i]
    n = len(off) - 1
    g = GpuCache(L, HQ, HKV, D, max(n, budget) + INTERVAL + 2, DT)
    g.fuse(to_dev(k_in), to_dev(v_in), to_dev(off))
    outs, states = [], []
    for t in range(steps):
        q, k, v = _step_inputs(i, t, L)
        g.step(to_dev(q), to_dev(k), to_dev(v), GAMMA, check_ws=False)
        if (t + 1) % INTERVAL == 0 and g.len > budget:
            g.evict(budget)
        torch.cuda.synchronize()
        outs.append(from_dev(g.out))
        K, V, S, P = g.snapshot()
        states.append((K[:, :, : g.len], V[:, :, : g.len], S[:, : g.len], P[:, : g.len], g.len, g.next_pos))
    return outs, states


def _slot_caps(L):
    caps = {}
    for i, (T_in, budget, steps, slot, _) in enumerate(REQUESTS):
        n = len(_request(i, L)[0]) - 1
        caps[slot] = max(caps.get(slot, 0), max(n, budget) + INTERVAL + 2)
    return [caps[s] for s in sorted(caps)]


def _run_batch(L, use_graph):
    """The schedule of REQUESTS through one DecodeLoop: yields, per global
    step and per active request, (request, local step, output, state)."""
    import torch
    from paper_2608_08569_amd.loop import DecodeLoop
    caps = _slot_caps(L)
    n = len(caps)
    lp = DecodeLoop(L, HQ, HKV, D, caps, [1] * n, GAMMA, interval=INTERVAL)
    for s in range(n):
        lp.retire(s)
    qb = torch.zeros(n, L, HQ, D, dtype=torch.bfloat16, device="cuda")
    kb = torch.zeros(n, L, HKV, D, dtype=torch.bfloat16, device="cuda")
    vb = torch.zeros_like(kb)
    if use_graph:
        lp.capture(qb, kb, vb)
    base = np.concatenate([[0], np.cumsum(caps)[:-1]]).astype(np.int64)
    holder = {}  # slot -> (request, start step)
    last = max(r[4] + r[2] for r in REQUESTS)
    fused = {}
    results = []
    for gstep in range(last):
        # leave, then join, between steps
        for s, (i, start) in list(holder.items()):
            if gstep - start == REQUESTS[i][2]:
                lp.retire(s)
                del holder[s]
        for i, (T_in, budget, steps, slot, start) in enumerate(REQUESTS):
            if start == gstep:
                assert slot not in holder, "the schedule reuses a slot that is still busy"
                off, k_in, v_in = _request(i, L)
                lp.admit(slot, to_dev(k_in), to_dev(v_in), to_dev(off), budget=budget)
                holder[slot] = (i, start)
                torch.cuda.synchronize()
                b, ln = int(base[slot]), len(off) - 1
                fused[i] = (from_dev(lp.k[:, :, b: b + ln]), from_dev(lp.v[:, :, b: b + ln]),
                            from_dev(lp.score[:, b: b + ln]), from_dev(lp.pos[:, b: b + ln]))
        q = np.zeros((n, L, HQ, D), np.uint16)
        k = np.zeros((n, L, HKV, D), np.uint16)
        v = np.zeros((n, L, HKV, D), np.uint16)
        for s, (i, start) in holder.items():
            q[s], k[s], v[s] = _step_inputs(i, gstep - start, L)
        qb.copy_(to_dev(q))
        kb.copy_(to_dev(k))
        vb.copy_(to_dev(v))
        if use_graph:
            lp.replay()
            _ = (qb.float() * 2).sum().item()  # eager work between replays
        else:
            lp.step(qb, kb, vb)
        torch.cuda.synchronize()
        st = from_dev(lp.status)
        out = from_dev(lp.out)
        lens, nxts = from_dev(lp.length), from_dev(lp.next_pos)
        for s in range(n):
            if s not in holder:
                assert st[s] == 1, f"idle slot {s} reported status {st[s]}"
                continue
            assert st[s] == 0, f"slot {s} status {st[s]}"
            i, start = holder[s]
            b, ln = int(base[s]), int(lens[s])
            state = (from_dev(lp.k[:, :, b: b + ln]), from_dev(lp.v[:, :, b: b + ln]),
                     from_dev(lp.score[:, b: b + ln]), from_dev(lp.pos[:, b: b + ln]), ln, int(nxts[s]))
            results.append((i, gstep - start, out[s], state))
    return results, fused


def _compare(L, use_graph):
    results, fused = _run_batch(L, use_graph)
    solo = {i: _solo(i, L) for i in range(len(REQUESTS))}
    seen = set()
    for i, t, out, state in results:
        outs, states = solo[i]
        assert np.array_equal(out, outs[t]), f"request {i} step {t}: output differs from the request alone"
        ref = states[t]
        for name, a, b in zip(("K", "V", "score", "pos"), state[:4], ref[:4]):
            assert np.array_equal(a, b), f"request {i} step {t}: {name} differs from the request alone"
        assert state[4:] == ref[4:], f"request {i} step {t}: length/next position {state[4:]} vs {ref[4:]}"
        seen.add((i, t))
    assert seen == {(i, t) for i, r in enumerate(REQUESTS) for t in range(r[2])}
    # evictions happened on each request's own schedule
    for i, (T_in, budget, steps, _, _) in enumerate(REQUESTS):
        lens = [solo[i][1][t][4] for t in range(steps)]
        assert any(x == budget for x in lens), f"request {i} never evicted"
    return results, fused


@pytest.mark.parametrize("L,use_graph", [(4, False), (4, True), (32, True)])
def test_requests_join_and_leave_bit_identical_to_running_alone(L, use_graph):
    """L = 4 takes the chunked decode path, L = 32 (128 (layer, KV head)
    items) the whole-range path with its order, merge and fold kernels."""
    _compare(L, use_graph)


def test_joined_requests_match_the_oracle():
    """Each request's fused prefill in its slot, and its first step there, against
    the oracle (state-synced from the fused state)."""
    L = 4
    results, fused = _run_batch(L, False)
    first = {i: (out, state) for i, t, out, state in results if t == 0}
    for i in range(len(REQUESTS)):
        off, k_in, v_in = _request(i, L)
        K0, V0, S0, P0 = fused[i]
        n = len(off) - 1
        for name, x, got in (("K", k_in, K0), ("V", v_in, V0)):
            ref = oracle.fuse(x, off, DT)
            check_close(widen(got, DT), ref, RTOL[DT], f"request {i} fused {name}")
        assert not S0.any() and np.array_equal(P0, np.tile(np.arange(n, dtype=np.int32), (L, 1)))
        q, k, v = _step_inputs(i, 0, L)
        cap = n + 1
        pad = lambda a, fill=0: np.concatenate([a, np.full(a.shape[:-2] + (1,) + a.shape[-1:], fill, a.dtype)], -2)
        Kc, Vc = pad(K0), pad(V0)
        ref_o, ref_s, ref_p, _ = oracle.decode_step(q, k, v, Kc, Vc, np.zeros((L, cap)), np.concatenate(
            [P0, np.zeros((L, 1), np.int32)], 1), n, n, GAMMA, DT)
        out, state = first[i]
        check_close(widen(out, DT), ref_o, RTOL[DT], f"request {i} first output")
        check_rel(state[2], ref_s, RTOL[DT], f"request {i} first scores")
        assert np.array_equal(state[3], ref_p)
