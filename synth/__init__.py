"""Seeded synthetic inputs for the VoxZip hot path.

This module is shared by the oracle side (tests, CPU baseline) and the HIP
side (tests, bench, smoke).  It holds no arithmetic of the method itself:
it only draws random numbers and lays out tensors of the shapes the paper's
workloads have (long audio, GQA caches, ASR spans of a few tokens each).

Random numbers come from SplitMix64 used as a counter-based generator
(Steele, Lea, Flood, "Fast splittable pseudorandom number generators",
OOPSLA 2014; reference constants as in Vigna's public-domain C version):
output i of the stream with key ``k`` is ``mix64(k + (i + 1) * 0x9E3779B97F4A7C15)``.
Every tensor has its own stream key, derived by hashing
(seed, config tag, tensor tag, index...) with the same mix function, so any
tensor can be regenerated alone and the values never depend on a library RNG.
Normals use the Box-Muller transform in float64, then round to float32 and,
for bfloat16 storage, round-to-nearest-even to bfloat16 bits.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

GOLDEN = 0x9E3779B97F4A7C15
_M1 = 0xBF58476D1CE4E5B9
_M2 = 0x94D049BB133111EB
_MASK = (1 << 64) - 1

DT_F32 = 0
DT_BF16 = 1


# ----------------------------------------------------------------------------
# SplitMix64, scalar (Python int) and vectorised (numpy uint64) forms
# ----------------------------------------------------------------------------
def mix64_int(z: int) -> int:
    z &= _MASK
    z = ((z ^ (z >> 30)) * _M1) & _MASK
    z = ((z ^ (z >> 27)) * _M2) & _MASK
    return z ^ (z >> 31)


def stream_key(*parts) -> int:
    """Hash a tuple of ints/strings into a 64-bit stream key."""
    k = 0x5EED5EED5EED5EED
    for p in parts:
        if isinstance(p, str):
            v = 0
            for ch in p.encode():
                v = mix64_int(v ^ ch)
            p = v
        k = mix64_int(k ^ (int(p) & _MASK))
    return k


def splitmix_u64(key: int, start: int, count: int) -> np.ndarray:
    """Outputs start .. start+count-1 of the SplitMix64 stream with state ``key``."""
    i = np.arange(start + 1, start + 1 + count, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(key & _MASK) + i * np.uint64(GOLDEN)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(_M1)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(_M2)
        z = z ^ (z >> np.uint64(31))
    return z


def uniform01(key: int, start: int, count: int) -> np.ndarray:
    """float64 uniforms in [0, 1) from the top 53 bits."""
    return (splitmix_u64(key, start, count) >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)


def _normal_block(key: int, start_pair: int, n_pairs: int) -> np.ndarray:
    u = splitmix_u64(key, 2 * start_pair, 2 * n_pairs)
    u1 = ((u[0::2] >> np.uint64(11)).astype(np.float64) + 1.0) * (2.0 ** -53)  # (0, 1]
    u2 = (u[1::2] >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)          # [0, 1)
    r = np.sqrt(-2.0 * np.log(u1))
    t = 2.0 * math.pi * u2
    out = np.empty(2 * n_pairs, dtype=np.float64)
    out[0::2] = r * np.cos(t)
    out[1::2] = r * np.sin(t)
    return out


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def normal_f32(key: int, n: int) -> np.ndarray:
    """n standard normals (Box-Muller, fp64) rounded to float32."""
    out = np.empty(n, dtype=np.float32)
    n_pairs = (n + 1) // 2
    block = 1 << 21
    starts = list(range(0, n_pairs, block))

    def work(s):
        m = min(block, n_pairs - s)
        z = _normal_block(key, s, m)
        lo = 2 * s
        hi = min(n, lo + 2 * m)
        out[lo:hi] = z[: hi - lo]

    if len(starts) == 1:
        work(0)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(work, starts))
    return out


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def as_storage(x_f32: np.ndarray, dtype: int) -> np.ndarray:
    """float32 values -> storage array (float32, or uint16 bfloat16 bits)."""
    if dtype == DT_F32:
        return np.ascontiguousarray(x_f32, dtype=np.float32)
    return f32_to_bf16_bits(x_f32)


def storage_to_f64(x: np.ndarray, dtype: int) -> np.ndarray:
    if dtype == DT_F32:
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    return bf16_bits_to_f32(x).astype(np.float64)


# ----------------------------------------------------------------------------
# Integer draws used for span lengths
# ----------------------------------------------------------------------------
def uniform_int(key: int, start: int, count: int, lo: int, hi: int) -> np.ndarray:
    """iid integers uniform on {lo..hi} (inclusive)."""
    u = uniform01(key, start, count)
    return lo + np.floor(u * (hi - lo + 1)).astype(np.int64)


def geometric(key: int, start: int, count: int, p: float) -> np.ndarray:
    """iid Geometric(p) on {0,1,2,...} (failures before the first success)."""
    u = 1.0 - uniform01(key, start, count)  # (0, 1]
    return np.floor(np.log(u) / math.log1p(-p)).astype(np.int64)


def spans_geometric(key: int, total: int, p: float = 0.25, max_len: int = 32,
                    p_one: float = 0.0, extra: int = 1) -> np.ndarray:
    """Span lengths covering exactly ``total`` tokens.

    A length is 1 with probability ``p_one``; otherwise ``extra + Geometric(p)``;
    draws above ``max_len`` are discarded and drawn again.  Spans are drawn until
    their sum reaches ``total``; the last one is truncated to fit.
    """
    lens = []
    covered = 0
    cursor = 0
    while covered < total:
        n = max(1024, int(1.5 * (total - covered) / 2) + 64)
        g = extra + geometric(key, cursor, n, p)
        if p_one > 0.0:
            one = uniform01(stream_key(key, "one"), cursor, n) < p_one
            g = np.where(one, 1, g)
        cursor += n
        g = g[g <= max_len]
        c = np.cumsum(g)
        need = total - covered
        idx = np.searchsorted(c, need)  # first index with cumsum >= need
        if idx < len(g):
            take = g[: idx + 1].copy()
            take[-1] -= c[idx] - need
            lens.append(take)
            covered = total
        else:
            lens.append(g)
            covered += int(c[-1])
    out = np.concatenate(lens).astype(np.int64)
    assert out.sum() == total and out.min() >= 1
    return out


def spans_uniform_exact(key: int, n_spans: int, lo: int, hi: int, total: int) -> np.ndarray:
    """``n_spans`` iid lengths uniform on {lo..hi}, redrawn as a whole vector
    until they sum to exactly ``total``."""
    for attempt in range(1 << 20):
        g = uniform_int(key, attempt * n_spans, n_spans, lo, hi)
        if int(g.sum()) == total:
            return g
    raise RuntimeError("no span vector with the requested sum")


def offsets_from_lengths(lens: np.ndarray) -> np.ndarray:
    off = np.zeros(len(lens) + 1, dtype=np.int32)
    off[1:] = np.cumsum(lens)
    return off


# ----------------------------------------------------------------------------
# Workload configurations (the paper's shapes: Qwen3-Omni-like GQA caches)
# ----------------------------------------------------------------------------
@dataclass
class Workload:
    name: str
    n_layers: int
    n_q_heads: int
    kv_heads: int
    d: int
    dtype: int
    n_audio: int              # audio tokens before fusion
    n_text: int               # text tokens after the audio, never fused (length-1 spans)
    span_kind: str            # "uniform", "geom4", "geom5mix"
    gamma: float
    budget: int
    steps: int
    interval: int = 1
    n_sink: int = 4
    kv_scale: bool = False    # per-channel log-uniform K/V scale in [0.5, 4]
    q_bias: bool = False      # bias queries so attention concentrates on ~5% of keys
    seed: int = 0
    extra: dict = field(default_factory=dict)

    @property
    def n_recent(self) -> int:
        return self.budget // 5

    @property
    def dtype_name(self) -> str:
        return "f32" if self.dtype == DT_F32 else "bf16"


def workload(name: str, seed: int = 0) -> Workload:
    if name == "tiny":
        return Workload("tiny", 1, 4, 1, 64, DT_F32, 512, 0, "uniform", 0.9, 128, 32, seed=seed)
    if name == "layer":
        return Workload("layer", 1, 32, 4, 128, DT_BF16, 4096, 256, "geom4", 0.95, 1024, 128, seed=seed)
    if name == "long32k":
        return Workload("long32k", 48, 32, 4, 128, DT_BF16, 32768, 0, "geom4", 0.95, 8192, 256,
                        kv_scale=True, seed=seed)
    if name == "aggr64k":
        return Workload("aggr64k", 48, 32, 4, 128, DT_BF16, 65536, 0, "geom5mix", 0.95, 3277, 512,
                        q_bias=True, seed=seed)
    raise KeyError(name)


BATCH = 16  # sequences of the batched-decode workload


def batch_lengths(seed: int = 0) -> np.ndarray:
    """Audio tokens of the 16 sequences of the batched workload, iid uniform on {2048..32768}."""
    return uniform_int(stream_key(seed, "batch16", "lengths"), 0, BATCH, 2048, 32768).astype(np.int64)


def batch_workloads(seed: int = 0) -> list:
    """One Workload per sequence of the batched workload: 48 layers, 32Q/4KV,
    d = 128, bf16, spans of mean length 4 (as "layer"), budget len / 4 of the
    sequence's audio tokens, eviction every 16 steps, 128 steps.  The sequence
    index (0..15) is the ``seq`` argument of the per-sequence generators."""
    return [Workload("batch16", 48, 32, 4, 128, DT_BF16, int(n), 0, "geom4", 0.95, int(n) // 4, 128,
                     interval=16, seed=seed) for n in batch_lengths(seed)]


def span_lengths(w: Workload, seq: int = 0) -> np.ndarray:
    key = stream_key(w.seed, w.name, "spans", seq)
    if w.span_kind == "uniform":
        audio = spans_uniform_exact(key, 64, 1, 16, w.n_audio)
    elif w.span_kind == "geom4":
        audio = spans_geometric(key, w.n_audio, p=0.25, max_len=32)
    elif w.span_kind == "geom5mix":
        # length 1 with probability 0.1, else 2 + Geometric(p) with mean 5.444 (cap 64): overall mean 5
        audio = spans_geometric(key, w.n_audio, p=1.0 / 4.444, max_len=64, p_one=0.1, extra=2)
    else:
        raise KeyError(w.span_kind)
    text = np.ones(w.n_text, dtype=np.int64)
    return np.concatenate([audio, text])


def channel_scales(w: Workload, which: str) -> np.ndarray:
    """[L][Hkv][d] per-channel scales, log-uniform on [0.5, 4] (ones when disabled)."""
    if not w.kv_scale:
        return np.ones((w.n_layers, w.kv_heads, w.d), dtype=np.float64)
    u = uniform01(stream_key(w.seed, w.name, "scale", which), 0, w.n_layers * w.kv_heads * w.d)
    lo, hi = math.log(0.5), math.log(4.0)
    return np.exp(lo + (hi - lo) * u).reshape(w.n_layers, w.kv_heads, w.d)


def prefill_kv(w: Workload, which: str, n_tokens: int | None = None, seq: int = 0,
               layers: range | None = None) -> np.ndarray:
    """Prefill K or V, storage dtype, shape [L][Hkv][T_in][d] (only ``layers`` if given)."""
    T = w.n_audio + w.n_text if n_tokens is None else n_tokens
    layers = range(w.n_layers) if layers is None else layers
    out = np.empty((len(layers), w.kv_heads, T, w.d),
                   dtype=np.float32 if w.dtype == DT_F32 else np.uint16)
    scales = channel_scales(w, which)
    for li, l in enumerate(layers):
        key = stream_key(w.seed, w.name, "prefill", which, seq, l)
        z = normal_f32(key, w.kv_heads * T * w.d).reshape(w.kv_heads, T, w.d)
        if w.kv_scale:
            z = (z.astype(np.float64) * scales[l][:, None, :]).astype(np.float32)
        out[li] = as_storage(z, w.dtype)
    return out


def q_bias(w: Workload) -> np.ndarray:
    """[L][Hq][d] query bias for concentrated attention (zeros when disabled).

    b = beta * u with u uniform on the unit sphere; beta is set so that the
    standard deviation of b . k / sqrt(d) over span-mean keys is 3.  A mean of
    ``n`` iid N(0, 1) rows has per-channel variance 1/n, so that deviation is
    beta * sqrt(mean(1/n)) / sqrt(d) over the span lengths n.
    """
    if not w.q_bias:
        return np.zeros((w.n_layers, w.n_q_heads, w.d), dtype=np.float64)
    g = normal_f32(stream_key(w.seed, w.name, "qbias"), w.n_layers * w.n_q_heads * w.d)
    g = g.astype(np.float64).reshape(w.n_layers, w.n_q_heads, w.d)
    u = g / np.linalg.norm(g, axis=-1, keepdims=True)
    lens = span_lengths(w)
    beta = 3.0 * math.sqrt(w.d) / math.sqrt(float(np.mean(1.0 / lens)))
    return beta * u


def decode_inputs(w: Workload, step: int, seq: int = 0, bias: np.ndarray | None = None):
    """(q [L][Hq][d], k_new [L][Hkv][d], v_new [L][Hkv][d]) in storage dtype for one step."""
    L, Hq, Hkv, d = w.n_layers, w.n_q_heads, w.kv_heads, w.d
    q = normal_f32(stream_key(w.seed, w.name, "q", seq, step), L * Hq * d).reshape(L, Hq, d)
    if w.q_bias:
        b = q_bias(w) if bias is None else bias
        q = (q.astype(np.float64) + b).astype(np.float32)
    k = normal_f32(stream_key(w.seed, w.name, "knew", seq, step), L * Hkv * d).reshape(L, Hkv, d)
    v = normal_f32(stream_key(w.seed, w.name, "vnew", seq, step), L * Hkv * d).reshape(L, Hkv, d)
    if w.kv_scale:
        k = (k.astype(np.float64) * channel_scales(w, "k")).astype(np.float32)
        v = (v.astype(np.float64) * channel_scales(w, "v")).astype(np.float32)
    return as_storage(q, w.dtype), as_storage(k, w.dtype), as_storage(v, w.dtype)


def random_state(seed: int, n_layers: int, kv_heads: int, d: int, cap: int, length: int,
                 dtype: int, next_pos: int | None = None, tie_levels: int = 0):
    """A random resident cache: K/V [L][Hkv][cap][d] (slots >= length zero),
    scores [L][cap] float32 >= 0, positions [L][cap] int32 (a random subset of
    [0, next_pos) holding 0..3 and the most recent positions, in shuffled slot order).

    ``tie_levels`` > 0 quantises the scores to that many distinct values so that
    ties are common.
    """
    next_pos = length if next_pos is None else next_pos
    key = stream_key(seed, "state", n_layers, kv_heads, d, cap, length, dtype, next_pos)
    k = normal_f32(stream_key(key, "k"), n_layers * kv_heads * cap * d).reshape(n_layers, kv_heads, cap, d)
    v = normal_f32(stream_key(key, "v"), n_layers * kv_heads * cap * d).reshape(n_layers, kv_heads, cap, d)
    k[:, :, length:, :] = 0
    v[:, :, length:, :] = 0
    u = uniform01(stream_key(key, "score"), 0, n_layers * cap).reshape(n_layers, cap)
    if tie_levels > 0:
        u = np.floor(u * tie_levels) / tie_levels
    score = (u * 0.5).astype(np.float32)
    score[:, length:] = 0
    pos = np.zeros((n_layers, cap), dtype=np.int32)
    for l in range(n_layers):
        # keep 0..min(4, length)-1 and the most recent, fill the rest from the middle
        n_keep_hi = min(length, max(0, length // 3))
        must = list(range(min(4, length))) + list(range(next_pos - n_keep_hi, next_pos))
        must = sorted(set(p for p in must if 0 <= p < next_pos))[:length]
        pool = np.setdiff1d(np.arange(next_pos), np.array(must, dtype=np.int64))
        r = uniform01(stream_key(key, "pick", l), 0, len(pool))
        extra = pool[np.argsort(r, kind="stable")[: length - len(must)]]
        chosen = np.concatenate([np.array(must, dtype=np.int64), np.sort(extra)])
        perm = np.argsort(uniform01(stream_key(key, "perm", l), 0, length), kind="stable")
        pos[l, :length] = chosen[perm]
    return as_storage(k, dtype), as_storage(v, dtype), score, pos
