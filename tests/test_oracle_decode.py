"""Pins of the oracle's decode step: Eq. (1) append, Eq. (2) attention and
Eq. (6) decayed score.

Attention has a plain definition, so it is pinned against a library routine
(torch's scaled_dot_product_attention in float64 on the CPU, with the KV
heads repeated for the grouped query heads), plus special cases with closed
forms.  The score is pinned by its closed-form total mass and the gamma = 0
and gamma = 1 special cases."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth


def _state(seed, L, Hq, Hkv, d, cap, length, dtype, scale=1.0):
    key = synth.stream_key(seed, "dec-test", L, Hq, Hkv, d, cap, length)
    q = synth.normal_f32(synth.stream_key(key, "q"), L * Hq * d).reshape(L, Hq, d) * np.float32(scale)
    kn = synth.normal_f32(synth.stream_key(key, "kn"), L * Hkv * d).reshape(L, Hkv, d)
    vn = synth.normal_f32(synth.stream_key(key, "vn"), L * Hkv * d).reshape(L, Hkv, d)
    kc, vc, score, pos = synth.random_state(seed, L, Hkv, d, cap, length, dtype, next_pos=length + 50)
    return (synth.as_storage(q, dtype), synth.as_storage(kn, dtype), synth.as_storage(vn, dtype),
            kc, vc, score, pos)


def _sdpa_reference(q, kn, vn, kc, vc, length, dtype):
    """torch SDPA (float64, CPU) over the cache with the new row appended."""
    qf = torch.from_numpy(synth.storage_to_f64(q, dtype))
    K = synth.storage_to_f64(kc, dtype)[:, :, :length]
    V = synth.storage_to_f64(vc, dtype)[:, :, :length]
    K = np.concatenate([K, synth.storage_to_f64(kn, dtype)[:, :, None]], axis=2)
    V = np.concatenate([V, synth.storage_to_f64(vn, dtype)[:, :, None]], axis=2)
    Hq, Hkv = q.shape[1], kc.shape[1]
    Kt = torch.from_numpy(K).repeat_interleave(Hq // Hkv, dim=1)
    Vt = torch.from_numpy(V).repeat_interleave(Hq // Hkv, dim=1)
    o = torch.nn.functional.scaled_dot_product_attention(qf[:, :, None, :], Kt, Vt)[:, :, 0, :]
    logits = torch.einsum("lhd,lhtd->lht", qf, Kt) / math.sqrt(q.shape[-1])
    p = torch.softmax(logits, dim=-1)
    return o.numpy(), p.numpy()


@pytest.mark.parametrize("dtype", [oracle.F32, oracle.BF16])
@pytest.mark.parametrize("shape", [(1, 4, 1, 64, 80, 70), (2, 32, 4, 128, 300, 257), (1, 6, 3, 16, 10, 1)])
def test_attention_matches_library_sdpa(dtype, shape):
    L, Hq, Hkv, d, cap, length = shape
    q, kn, vn, kc, vc, score, pos = _state(1, L, Hq, Hkv, d, cap, length, dtype)
    out, s, p, pr = oracle.decode_step(q, kn, vn, kc, vc, score, pos, length, length + 50,
                                       0.9, dtype, want_p=True)
    o_ref, p_ref = _sdpa_reference(q, kn, vn, kc, vc, length, dtype)
    np.testing.assert_allclose(out, o_ref, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(pr, p_ref, rtol=1e-10, atol=1e-15)
    # every query head's softmax row sums to one
    np.testing.assert_allclose(pr.sum(axis=-1), 1.0, rtol=0, atol=1e-13)


def test_grouped_heads_read_their_own_kv_head():
    # KV heads with disjoint value spaces: head h's output must come from KV head h // (Hq/Hkv)
    L, Hq, Hkv, d, cap, length = 1, 8, 4, 8, 20, 12
    q, kn, vn, kc, vc, score, pos = _state(2, L, Hq, Hkv, d, cap, length, oracle.F32)
    vc = np.zeros_like(vc)
    vn = np.zeros_like(vn)
    for g in range(Hkv):
        vc[0, g, :length, g] = 1.0
        vn[0, g, g] = 1.0
    out, *_ = oracle.decode_step(q, kn, vn, kc, vc, score, pos, length, 99, 0.5, oracle.F32)
    for h in range(Hq):
        g = h // (Hq // Hkv)
        expect = np.zeros(d)
        expect[g] = 1.0
        np.testing.assert_allclose(out[0, h], expect, atol=1e-14)


def test_single_key_returns_its_value_exactly():
    L, Hq, Hkv, d, cap = 2, 4, 2, 16, 4
    q, kn, vn, kc, vc, score, pos = _state(3, L, Hq, Hkv, d, cap, 0, oracle.BF16)
    out, s, p, _ = oracle.decode_step(q, kn, vn, kc, vc, score, pos, 0, 7, 0.95, oracle.BF16)
    vf = synth.storage_to_f64(vn, oracle.BF16)
    for h in range(Hq):
        assert np.array_equal(out[:, h], vf[:, h // 2])
    assert np.all(s[:, 0] == Hq)       # each head puts mass 1 on the only key
    assert np.all(p[:, 0] == 7)        # appended at position next_pos


def test_zero_query_gives_uniform_weights_and_mean_value():
    L, Hq, Hkv, d, cap, length = 1, 4, 1, 32, 64, 40
    q, kn, vn, kc, vc, score, pos = _state(4, L, Hq, Hkv, d, cap, length, oracle.F32)
    q = np.zeros_like(q)
    out, s, p, pr = oracle.decode_step(q, kn, vn, kc, vc, score, pos, length, 500, 0.0,
                                       oracle.F32, want_p=True)
    T = length + 1
    np.testing.assert_allclose(pr, 1.0 / T, rtol=1e-14)
    V = np.concatenate([synth.storage_to_f64(vc, 0)[0, 0, :length], synth.storage_to_f64(vn, 0)[0, :1]])
    np.testing.assert_allclose(out[0, 0], V.mean(axis=0), rtol=1e-12, atol=1e-14)
    # gamma = 0: the score is the current step's head-summed mass, Hq / T per key
    np.testing.assert_allclose(s[0], Hq / T, rtol=1e-13)


def test_explicit_scale_is_used():
    L, Hq, Hkv, d, cap, length = 1, 2, 1, 16, 30, 20
    q, kn, vn, kc, vc, score, pos = _state(5, L, Hq, Hkv, d, cap, length, oracle.F32)
    o1, *_ = oracle.decode_step(q, kn, vn, kc, vc, score, pos, length, 99, 0.9, oracle.F32,
                                sm_scale=0.5 / math.sqrt(d))
    q_half = (q * np.float32(0.5)).astype(np.float32)
    o2, *_ = oracle.decode_step(q_half, kn, vn, kc, vc, score, pos, length, 99, 0.9, oracle.F32)
    np.testing.assert_allclose(o1, o2, rtol=1e-12, atol=1e-14)


def _run_steps(gamma, steps, Hq=4, Hkv=2, d=16, L=2, n0=6):
    """Decode ``steps`` tokens from a cache of n0 tokens with zero scores."""
    cap = n0 + steps + 1
    kc, vc, _, pos = synth.random_state(6, L, Hkv, d, cap, n0, oracle.F32, next_pos=n0)
    score = np.zeros((L, cap))
    length, nxt = n0, n0
    ps = []
    for t in range(steps):
        key = synth.stream_key(6, "steps", t)
        q = synth.normal_f32(synth.stream_key(key, "q"), L * Hq * d).reshape(L, Hq, d) * np.float32(2)
        kn = synth.normal_f32(synth.stream_key(key, "k"), L * Hkv * d).reshape(L, Hkv, d)
        vn = synth.normal_f32(synth.stream_key(key, "v"), L * Hkv * d).reshape(L, Hkv, d)
        _, s, p, pr = oracle.decode_step(q, kn, vn, kc, vc, score, pos, length, nxt, gamma,
                                         oracle.F32, want_p=True)
        kc[:, :, length], vc[:, :, length] = kn, vn
        score[:, : length + 1], pos[:, : length + 1] = s, p
        ps.append(pr)
        length += 1
        nxt += 1
    return score[:, :length], ps, Hq


@pytest.mark.parametrize("gamma", [0.0, 0.5, 0.9, 0.95, 1.0])
def test_total_score_mass_closed_form(gamma):
    k = 9
    A, _, Hq = _run_steps(gamma, k)
    expect = Hq * k if gamma == 1.0 else Hq * (1 - gamma ** k) / (1 - gamma)
    np.testing.assert_allclose(A.sum(axis=1), expect, rtol=1e-12)


def test_gamma_one_is_plain_accumulation_and_new_slot_starts_undecayed():
    A1, ps, Hq = _run_steps(1.0, 5)
    A9, ps9, _ = _run_steps(0.9, 5)
    n0 = 6
    # the newest token has only its own step's head-summed mass
    np.testing.assert_allclose(A9[:, -1], ps9[-1][:, :, -1].sum(axis=1), rtol=1e-13)
    # gamma = 1: a key's score is the sum over steps of its head-summed mass
    plain = np.zeros_like(A1)
    for t, pr in enumerate(ps):
        plain[:, : n0 + t + 1] += pr.sum(axis=1)
    np.testing.assert_allclose(A1, plain, rtol=1e-12)
    # decayed scores are strictly below the undecayed ones for keys older than one step
    assert np.all(A9[:, :-1] < A1[:, :-1])


def test_bad_shapes_rejected():
    q, kn, vn, kc, vc, score, pos = _state(7, 1, 6, 4, 8, 10, 5, oracle.F32)
    with pytest.raises(ValueError):  # 6 query heads do not split over 4 KV heads
        oracle.decode_step(q, kn, vn, kc, vc, score, pos, 5, 9, 0.9, oracle.F32)
    q, kn, vn, kc, vc, score, pos = _state(7, 1, 4, 2, 8, 10, 10, oracle.F32)
    with pytest.raises(ValueError):  # no free slot to append into
        oracle.decode_step(q, kn, vn, kc, vc, score, pos, 10, 11, 0.9, oracle.F32)
