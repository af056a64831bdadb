"""Python entry points of the fp64 VoxZip oracle (``voxzip_oracle.c``).

TEST INFRASTRUCTURE: only the tests, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  It shares no code
with the HIP library and never imports it.

Array conventions follow the C routines: storage arrays are float32, or
uint16 holding bfloat16 bits (``dtype`` 0 / 1); results are float64.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "voxzip_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
F32, BF16 = 0, 1

_lib = None


def build(out: str = _LIB, src: str = _SRC, extra: tuple = ()) -> str:
    """Compile the oracle with gcc (-O2, IEEE arithmetic, OpenMP over layers)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-fno-fast-math",
           *extra, "-o", out + ".tmp", src, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def load(path: str | None = None):
    """Load the oracle library (building it first if it is not there)."""
    global _lib
    if path is None and _lib is not None:
        return _lib
    p = path or os.environ.get("VOXZIP_ORACLE_LIB") or _LIB
    if not os.path.exists(p):
        build(p)
    lib = ctypes.CDLL(p)
    P = ctypes.c_void_p
    i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.orc_threads.restype = ctypes.c_int
    lib.orc_set_threads.argtypes = [ctypes.c_int]
    lib.orc_set_threads.restype = None
    lib.orc_fuse.argtypes = [P, i32, P, i32, P, i32, i32, i32, i32, P]
    lib.orc_decode_step.argtypes = [P, P, P, P, P, P, P, i32, i32, f64, f64,
                                    i32, i32, i32, i32, i32, i32, P, P, P, P]
    lib.orc_evict_select.argtypes = [P, P, i32, i32, i32, i32, i32, i32, i32, P, P]
    lib.orc_build_offsets.argtypes = [P, P, P, P, i32, i64, i32, ctypes.c_float, P, P]
    for f in (lib.orc_fuse, lib.orc_decode_step, lib.orc_evict_select, lib.orc_build_offsets):
        f.restype = ctypes.c_int
    if path is None:
        _lib = lib
    return lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _store(a, dtype):
    want = np.float32 if dtype == F32 else np.uint16
    a = np.ascontiguousarray(a)
    if a.dtype != want:
        raise TypeError(f"storage array must be {np.dtype(want)}, got {a.dtype}")
    return a


def threads(lib=None) -> int:
    return (lib or load()).orc_threads()


def set_threads(n: int, lib=None) -> None:
    """Threads of the oracle's parallel loops from now on (timing only)."""
    (lib or load()).orc_set_threads(int(n))


def fuse(x, off, dtype, anchor=None, lib=None):
    """Eq. (4) group means of x [L][H][T_in][d] over spans ``off`` -> float64 [L][H][n][d]."""
    lib = lib or load()
    x = _store(x, dtype)
    off = np.ascontiguousarray(off, dtype=np.int32)
    L, H, T, d = x.shape
    n = len(off) - 1
    if anchor is not None:
        anchor = _store(anchor, dtype)
        assert anchor.shape == (L, H, n, d)
    out = np.empty((L, H, n, d), dtype=np.float64)
    rc = lib.orc_fuse(_p(x), T, _p(off), n, _p(anchor), L, H, d, dtype, _p(out))
    if rc != 0:
        raise ValueError("orc_fuse rejected its arguments")
    return out


def decode_step(q, k_new, v_new, k_cache, v_cache, score, pos, length, next_pos,
                gamma, dtype, sm_scale=0.0, want_p=False, lib=None):
    """One decode step from a given pre-step state (Eq. 1, 2, 6).

    Returns (out [L][Hq][d], score [L][len+1], pos [L][len+1], p or None).
    ``score`` is the pre-step score array [L][cap] (any float dtype, widened to fp64).
    """
    lib = lib or load()
    q, k_new, v_new = _store(q, dtype), _store(k_new, dtype), _store(v_new, dtype)
    k_cache, v_cache = _store(k_cache, dtype), _store(v_cache, dtype)
    L, Hkv, cap, d = k_cache.shape
    Hq = q.shape[1]
    score = np.ascontiguousarray(score, dtype=np.float64)
    pos = np.ascontiguousarray(pos, dtype=np.int32)
    assert score.shape == (L, cap) and pos.shape == (L, cap)
    T = length + 1
    out = np.empty((L, Hq, d), dtype=np.float64)
    s_out = np.empty((L, T), dtype=np.float64)
    p_out = np.empty((L, T), dtype=np.int32)
    pr = np.empty((L, Hq, T), dtype=np.float64) if want_p else None
    rc = lib.orc_decode_step(_p(q), _p(k_new), _p(v_new), _p(k_cache), _p(v_cache),
                             _p(score), _p(pos), length, next_pos, float(gamma), float(sm_scale),
                             L, Hq, Hkv, d, cap, dtype, _p(out), _p(s_out), _p(p_out), _p(pr))
    if rc != 0:
        raise ValueError("orc_decode_step rejected its arguments")
    return out, s_out, p_out, pr


def evict_select(score, pos, length, budget, n_sink=4, n_recent=-1, next_pos=None, lib=None):
    """Kept slots per layer in ascending position order -> (keep [L][new_len], new_len)."""
    lib = lib or load()
    score = np.ascontiguousarray(score, dtype=np.float64)
    pos = np.ascontiguousarray(pos, dtype=np.int32)
    L, cap = score.shape
    if next_pos is None:
        next_pos = int(pos[:, :length].max()) + 1 if length > 0 else 0
    keep = np.empty((L, budget), dtype=np.int32)
    nl = np.zeros(1, dtype=np.int32)
    rc = lib.orc_evict_select(_p(score), _p(pos), length, budget, n_sink, n_recent, next_pos,
                              L, cap, _p(keep), _p(nl))
    if rc != 0:
        raise ValueError("orc_evict_select rejected its arguments")
    return keep[:, : int(nl[0])], int(nl[0])


def gather_rows(x, keep):
    """Eq. (7)-(8) concatenation: rows ``keep[l]`` of x[l] (K/V [L][H][cap][d] or [L][cap])."""
    L = x.shape[0]
    if x.ndim == 4:
        return np.stack([x[l][:, keep[l], :] for l in range(L)])
    return np.stack([x[l][keep[l]] for l in range(L)])


def build_offsets(t_start_ms, t_end_ms, conf, text_len, t_total_ms, L_a,
                  conf_threshold=0.3, lib=None):
    """Stage-1 span offsets (confidence filter, Eq. 3, uniform groups, background)."""
    lib = lib or load()
    ts = np.ascontiguousarray(t_start_ms, dtype=np.int64)
    te = np.ascontiguousarray(t_end_ms, dtype=np.int64)
    cf = np.ascontiguousarray(conf, dtype=np.float32)
    tl = np.ascontiguousarray(text_len, dtype=np.int32)
    off = np.zeros(L_a + 1, dtype=np.int32)
    n = np.zeros(1, dtype=np.int32)
    rc = lib.orc_build_offsets(_p(ts), _p(te), _p(cf), _p(tl), len(ts), int(t_total_ms), int(L_a),
                               float(conf_threshold), _p(off), _p(n))
    if rc != 0:
        raise ValueError("orc_build_offsets rejected its arguments")
    return off[: int(n[0]) + 1].copy()


class Run:
    """The whole method run by the oracle: fuse, then decode steps with eviction.

    State: K/V in storage dtype [L][Hkv][cap][d], scores float64 [L][cap],
    positions int32 [L][cap], kept in ascending position order after every
    eviction (Eq. 7-8).
    """

    def __init__(self, k_in, v_in, off, dtype, n_q_heads, cap, gamma, budget,
                 n_sink=4, n_recent=-1, interval=1, lib=None):
        self.lib = lib or load()
        self.dtype = dtype
        self.Hq = n_q_heads
        self.gamma = gamma
        self.budget = budget
        self.n_sink = n_sink
        self.n_recent = budget // 5 if n_recent < 0 else n_recent
        self.interval = interval
        L, H, _, d = k_in.shape
        n = len(off) - 1
        self.L, self.Hkv, self.d, self.cap = L, H, d, cap
        kf = fuse(k_in, off, dtype, lib=self.lib)
        vf = fuse(v_in, off, dtype, lib=self.lib)
        store = np.float32 if dtype == F32 else np.uint16
        self.k = np.zeros((L, H, cap, d), dtype=store)
        self.v = np.zeros((L, H, cap, d), dtype=store)
        self.k[:, :, :n] = _round_store(kf, dtype)
        self.v[:, :, :n] = _round_store(vf, dtype)
        self.score = np.zeros((L, cap), dtype=np.float64)
        self.pos = np.zeros((L, cap), dtype=np.int32)
        self.pos[:, :n] = np.arange(n, dtype=np.int32)
        self.len = n
        self.next_pos = n
        self.t = 0

    def step(self, q, k_new, v_new):
        out, s, p, _ = decode_step(q, k_new, v_new, self.k, self.v, self.score, self.pos,
                                   self.len, self.next_pos, self.gamma, self.dtype, lib=self.lib)
        T = self.len + 1
        self.k[:, :, self.len] = k_new
        self.v[:, :, self.len] = v_new
        self.score[:, :T] = s
        self.pos[:, :T] = p
        self.len = T
        self.next_pos += 1
        self.t += 1
        if self.t % self.interval == 0 and self.len > self.budget:
            self.evict()
        return out

    def evict(self):
        keep, nl = evict_select(self.score, self.pos, self.len, self.budget, self.n_sink,
                                self.n_recent, self.next_pos, lib=self.lib)
        self.k[:, :, :nl] = gather_rows(self.k, keep)
        self.v[:, :, :nl] = gather_rows(self.v, keep)
        self.score[:, :nl] = gather_rows(self.score, keep)
        self.pos[:, :nl] = gather_rows(self.pos, keep)
        self.len = nl


def _round_store(x64, dtype):
    """float64 -> storage dtype, rounding through float32 (nearest-even at each step)."""
    f = x64.astype(np.float32)
    if dtype == F32:
        return f
    b = f.view(np.uint32)
    return ((b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)
