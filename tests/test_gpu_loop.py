"""The decode loop on the ragged entry points (paper_2608_08569_amd.loop):
one step captured as a HIP graph and replayed per token gives the same bits
as the same steps launched eagerly, in the all-layer and the per-layer mode,
with the eviction schedule (also over 32 layers, where the one call takes the
whole-range path: order, range, merge and fold kernels in the graph);
per-layer calls give the same bits as one call over all layers; the first
step matches the oracle."""
import numpy as np
import pytest

import oracle
import synth
from vzt import RTOL, check_close, check_rel, from_dev, to_dev, widen

pytestmark = pytest.mark.gpu

L, HQ, HKV, D = 4, 32, 4, 128
T_IN = [1200, 4000, 300]
BUDGETS = [256, 900, 96]
INTERVAL = 2
STEPS = 8


def _loop(L=L):
    import torch
    from paper_2608_08569_amd.loop import DecodeLoop
    offs = [synth.offsets_from_lengths(synth.spans_geometric(synth.stream_key(5, "loop", i), T, 0.25, 32))
            for i, T in enumerate(T_IN)]
    n_spans = np.array([len(o) - 1 for o in offs], dtype=np.int64)
    caps = np.maximum(n_spans, BUDGETS) + INTERVAL + 1
    lp = DecodeLoop(L, HQ, HKV, D, caps, BUDGETS, 0.95, interval=INTERVAL)
    in_base = np.concatenate([[0], np.cumsum(T_IN)[:-1]]).astype(np.int64)
    x = synth.normal_f32(synth.stream_key(5, "loop-kv"), 2 * L * HKV * sum(T_IN) * D)
    kv = synth.as_storage(x.reshape(2, L, HKV, sum(T_IN), D), synth.DT_BF16)
    off_base = np.concatenate([[0], np.cumsum(n_spans + 1)[:-1]]).astype(np.int64)
    dev = lambda a, dt: torch.tensor(a, dtype=dt, device="cuda")
    lp.fuse(to_dev(kv[0]), to_dev(kv[1]), dev(in_base, torch.int64), dev(T_IN, torch.int32),
            dev(np.concatenate(offs), torch.int32), dev(off_base, torch.int64), dev(n_spans, torch.int32),
            int(n_spans.max()))
    torch.cuda.synchronize()
    assert np.all(from_dev(lp.status) == 0)
    return lp


def _inputs(step, L=L):
    n = len(T_IN)
    key = synth.stream_key(6, "loop-step", step)
    mk = lambda tag, shape: synth.as_storage(
        synth.normal_f32(synth.stream_key(key, tag), int(np.prod(shape))).reshape(shape), synth.DT_BF16)
    return mk("q", (n, L, HQ, D)), mk("k", (n, L, HKV, D)), mk("v", (n, L, HKV, D))


def _state(lp):
    import torch
    torch.cuda.synchronize()
    return [from_dev(t) for t in (lp.k, lp.v, lp.score, lp.pos, lp.length, lp.next_pos)]


def _layer_major(a):
    # [n][L][H][d] -> [L][n][1][H][d]
    return np.ascontiguousarray(np.transpose(a, (1, 0, 2, 3))[:, :, None])


@pytest.mark.parametrize("per_layer,L", [(False, L), (True, L), (False, 32)])
def test_graph_replay_matches_eager_steps(per_layer, L):
    import torch
    eager, graph = _loop(L), _loop(L)
    n = len(T_IN)
    if per_layer:
        qb = torch.zeros(L, n, 1, HQ, D, dtype=torch.bfloat16, device="cuda")
        kb = torch.zeros(L, n, 1, HKV, D, dtype=torch.bfloat16, device="cuda")
        vb = torch.zeros_like(kb)
        qmix = torch.zeros_like(qb)

        def layer_query(l, q, outs):
            # layer l's query depends on layer l - 1's output, as in a forward pass
            if l == 0:
                return q[0]
            return torch.add(q[l], outs[l - 1], out=qmix[l])
    else:
        qb = torch.zeros(n, L, HQ, D, dtype=torch.bfloat16, device="cuda")
        kb = torch.zeros(n, L, HKV, D, dtype=torch.bfloat16, device="cuda")
        vb = torch.zeros_like(kb)
        layer_query = None
    graph.capture(qb, kb, vb, layer_query)
    for a, b in zip(_state(eager), _state(graph)):
        assert np.array_equal(a, b), "capture changed the state"
    for step in range(STEPS):
        q, k, v = _inputs(step, L)
        if per_layer:
            q, k, v = _layer_major(q), _layer_major(k), _layer_major(v)
        qd, kd, vd = to_dev(q), to_dev(k), to_dev(v)
        eager.step(qd, kd, vd, layer_query)
        qb.copy_(qd)
        kb.copy_(kd)
        vb.copy_(vd)
        graph.replay()
        torch.cuda.synchronize()
        _ = (qd.float() * 2).sum().item()  # eager work between replays
        for a, b in zip(_state(eager), _state(graph)):
            assert np.array_equal(a, b), f"step {step}: replay differs from the eager step"
        outs_e = eager.out_layers if per_layer else [eager.out]
        outs_g = graph.out_layers if per_layer else [graph.out]
        for a, b in zip(outs_e, outs_g):
            assert np.array_equal(from_dev(a), from_dev(b))
    lens = from_dev(graph.length)
    assert np.all(lens <= np.maximum(BUDGETS, 0) + INTERVAL)


def test_per_layer_calls_match_one_call_and_the_oracle():
    """The first step in both modes: per-layer calls give the bits of one call
    over all layers (the same chunking), and both match the oracle."""
    one, per = _loop(), _loop()
    n = len(T_IN)
    q, k, v = _inputs(0)
    K0, V0, S0, P0, len0, nxt0 = _state(one)
    one.step(to_dev(q), to_dev(k), to_dev(v))
    ql, kl, vl = (to_dev(_layer_major(x)) for x in (q, k, v))
    per.step(ql, kl, vl, lambda l, qq, outs: qq[l])
    for a, b in zip(_state(one), _state(per)):
        assert np.array_equal(a, b)
    out_one = from_dev(one.out)
    for l in range(L):
        assert np.array_equal(from_dev(per.out_layers[l])[:, 0], out_one[:, l])
    base = np.concatenate([[0], np.cumsum(from_dev(one.cap))[:-1]])
    caps = from_dev(one.cap)
    S1 = from_dev(one.score)
    for s in range(n):
        sl = slice(int(base[s]), int(base[s] + caps[s]))
        ln = int(len0[s])
        ref_o, ref_s, _, _ = oracle.decode_step(q[s], k[s], v[s], K0[:, :, sl], V0[:, :, sl],
                                                S0[:, sl].astype(np.float64), P0[:, sl], ln, int(nxt0[s]), 0.95,
                                                synth.DT_BF16)
        check_close(widen(out_one[s], synth.DT_BF16), ref_o, RTOL[synth.DT_BF16], f"seq {s} output")
        check_rel(S1[:, sl][:, : ln + 1], ref_s, RTOL[synth.DT_BF16], f"seq {s} score")
