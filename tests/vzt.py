"""Shared helpers of the GPU parity tests: moving storage arrays between numpy
and the device, the tolerance rule, and a GPU-side cache state."""
from __future__ import annotations

import numpy as np

import synth

RTOL = {synth.DT_F32: 1e-5, synth.DT_BF16: 2e-2}


def torch():
    import torch as t
    return t


def to_dev(a: np.ndarray, dtype: int | None = None):
    """numpy storage (float32 / uint16 bf16 bits / int32) -> contiguous cuda tensor."""
    t = torch()
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return t.from_numpy(a.view(np.int16)).view(t.bfloat16).cuda()
    return t.from_numpy(a).cuda()


def from_dev(x) -> np.ndarray:
    t = torch()
    x = x.detach().cpu().contiguous()
    if x.dtype == t.bfloat16:
        return x.view(t.int16).numpy().view(np.uint16)
    return x.numpy()


def widen(a: np.ndarray, dtype: int) -> np.ndarray:
    return synth.storage_to_f64(a, dtype)


def check_close(got: np.ndarray, ref: np.ndarray, rtol: float, what: str = "") -> float:
    """|got - ref| <= rtol*|ref| + rtol*rms(ref over the last axis), element by element.
    Returns the largest error in units of the allowed error."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    rms = np.sqrt(np.mean(ref * ref, axis=-1, keepdims=True))
    allow = rtol * np.abs(ref) + rtol * rms + 1e-30
    err = np.abs(got - ref)
    worst = float(np.max(err / allow))
    if worst > 1.0:
        idx = np.unravel_index(np.argmax(err / allow), err.shape)
        raise AssertionError(f"{what}: element {idx} got {got[idx]!r} ref {ref[idx]!r} "
                             f"(err {err[idx]:.3g}, allowed {allow[idx]:.3g})")
    return worst


def check_rel(got: np.ndarray, ref: np.ndarray, rtol: float, what: str = "") -> float:
    """|got - ref| <= rtol*|ref|, element by element: the bound for the decayed
    scores, which are non-negative, so that the smallest ones (the slots
    Eq. (9) evicts) are held to their own size.  Returns the largest error in
    units of the allowed error."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    allow = rtol * np.abs(ref) + 1e-38
    err = np.abs(got - ref)
    worst = float(np.max(err / allow))
    if worst > 1.0:
        idx = np.unravel_index(np.argmax(err / allow), err.shape)
        raise AssertionError(f"{what}: element {idx} got {got[idx]!r} ref {ref[idx]!r} "
                             f"(err {err[idx]:.3g}, allowed {allow[idx]:.3g})")
    return worst


def decode_header_bytes(L: int) -> int:
    """Bytes of a decode workspace's header: 256 reserved bytes, then one
    8-byte arrival counter per layer, padded to 256 bytes."""
    return 256 + (8 * L + 255) // 256 * 256


def bf16_ulp(x: np.ndarray) -> np.ndarray:
    ax = np.maximum(np.abs(x), 2.0 ** -126)
    return 2.0 ** (np.floor(np.log2(ax)) - 7)


class GpuCache:
    """Device-side cache state driven through the C ABI binding."""

    def __init__(self, L, Hq, Hkv, d, cap, dtype):
        t = torch()
        import paper_2608_08569_amd as vz
        self.vz = vz
        self.L, self.Hq, self.Hkv, self.d, self.cap, self.dtype = L, Hq, Hkv, d, cap, dtype
        tdt = t.float32 if dtype == synth.DT_F32 else t.bfloat16
        self.k = t.zeros(L, Hkv, cap, d, dtype=tdt, device="cuda")
        self.v = t.zeros(L, Hkv, cap, d, dtype=tdt, device="cuda")
        self.score = t.zeros(L, cap, dtype=t.float32, device="cuda")
        self.pos = t.zeros(L, cap, dtype=t.int32, device="cuda")
        self.out = t.zeros(L, Hq, d, dtype=tdt, device="cuda")
        self.ws_dec = vz.workspace(vz.VZ_OP_DECODE, L, Hq, Hkv, d, cap)
        self.ws_ev = vz.workspace(vz.VZ_OP_EVICT, L, Hq, Hkv, d, cap)
        self.len = 0
        self.next_pos = 0

    def fuse(self, k_in_dev, v_in_dev, off_dev, anchor_k=None, anchor_v=None):
        n = off_dev.numel() - 1
        self.vz.voxzip_fuse_spans(k_in_dev, v_in_dev, off_dev, self.k, self.v, self.score, self.pos,
                                  anchor_k, anchor_v)
        self.len = n
        self.next_pos = n

    def load(self, k, v, score, pos, length, next_pos):
        """Set the state from host arrays (storage dtype)."""
        t = torch()
        self.k.copy_(to_dev(k))
        self.v.copy_(to_dev(v))
        self.score.copy_(t.from_numpy(np.ascontiguousarray(score, dtype=np.float32)))
        self.pos.copy_(t.from_numpy(np.ascontiguousarray(pos, dtype=np.int32)))
        self.len, self.next_pos = length, next_pos

    def snapshot(self, layers=None):
        """Host copies of K, V, score and pos: every layer, or the listed ones
        (gathered on the device first, so a long cache pulls only those)."""
        torch().cuda.synchronize()
        if layers is None:
            return (from_dev(self.k), from_dev(self.v), from_dev(self.score), from_dev(self.pos))
        idx = torch().tensor(list(layers), dtype=torch().long, device="cuda")
        return tuple(from_dev(x.index_select(0, idx)) for x in (self.k, self.v, self.score, self.pos))

    def step(self, q_dev, k_dev, v_dev, gamma, sm_scale=0.0, check_ws=True):
        self.vz.voxzip_decode_attend_score(q_dev, k_dev, v_dev, self.k, self.v, self.score, self.pos, self.out,
                                           self.len, self.next_pos, gamma, sm_scale, workspace=self.ws_dec)
        self.len += 1
        self.next_pos += 1
        if check_ws:
            self.check_decode_workspace()

    def fused_decode_path(self) -> bool:
        """Whether the library takes its MFMA decode path for this shape."""
        G = self.Hq // self.Hkv
        return self.dtype == synth.DT_BF16 and self.d == 128 and self.Hkv in (1, 2, 4, 8) and G <= 8

    def check_decode_workspace(self):
        """After every call the decode workspace's header is still zero: its
        256 reserved bytes (no kernel writes outside its partial-result rows)
        and the per-layer arrival counters after them (the last workgroup of
        each layer resets its counter)."""
        torch().cuda.synchronize()
        hdr = from_dev(self.ws_dec[:decode_header_bytes(self.L)]).view(np.uint32)
        assert not hdr.any(), f"decode workspace header not zero at word {np.flatnonzero(hdr)[:4]}"

    def evict(self, budget, n_sink=4, n_recent=-1, kept=None):
        self.len = self.vz.voxzip_evict_compact(self.k, self.v, self.score, self.pos, self.len, budget,
                                                self.next_pos, n_sink, n_recent, kept_pos_out=kept,
                                                workspace=self.ws_ev)
        return self.len
