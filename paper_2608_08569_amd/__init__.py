"""VoxZip hot path on MI355X: Python binding of libvoxzip.so.

The functions below carry the names of the C entry points in
``include/voxzip.h`` and only marshal arguments: torch tensors are passed as
device pointers together with their sizes and the current HIP stream.  All
work runs in the library's HIP kernels.  There is no fallback: if the library
is not built, importing the binding's functions raises.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("VOXZIP_LIB", os.path.join(HERE, "libvoxzip.so"))

VZ_OK, VZ_ERR_INVALID, VZ_ERR_SHAPE, VZ_ERR_CAPACITY = 0, -1, -2, -3
VZ_ERR_UNSUPPORTED, VZ_ERR_HIP, VZ_ERR_WORKSPACE = -4, -5, -6
VZ_IDLE = 1  # per-sequence status of a ragged call: an idle batch slot (cap 0)
VZ_F32, VZ_BF16 = 0, 1
VZ_OP_DECODE, VZ_OP_EVICT, VZ_OP_DECODE_EVICT = 1, 2, 3
VZ_NOALLOC_SCRATCH_BYTES = 64 << 20

_lib = None


class VoxzipError(RuntimeError):
    def __init__(self, status: int, text: str):
        super().__init__(f"{text} (status {status})")
        self.status = status


def lib() -> ctypes.CDLL:
    """The loaded C library with argument types declared."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built: run __graft_entry__.build() "
                          "or python paper_2608_08569_amd/build.py")
    L = ctypes.CDLL(LIB_PATH)
    P, i32, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
    L.voxzip_fuse_spans.argtypes = [P, P, i32, P, i32, P, P, P, P, P, P, i32, i32, i32, i32, i32, P]
    L.voxzip_decode_attend_score.argtypes = [P, P, P, P, P, P, P, P, i32, i32, f32, f32,
                                             i32, i32, i32, i32, i32, i32, P, sz, P]
    L.voxzip_evict_compact.argtypes = [P, P, P, P, i32, i32, i32, i32, i32, P, P,
                                       i32, i32, i32, i32, i32, P, sz, P]
    L.voxzip_decode_evict.argtypes = [P, P, P, P, P, P, P, P, i32, i32, f32, f32, i32, i32, i32, P, P,
                                      i32, i32, i32, i32, i32, i32, P, sz, P]
    L.voxzip_decode_evict_noalloc.argtypes = [P, P, P, P, P, P, P, P, i32, i32, f32, f32, i32, i32, i32, P, P,
                                              i32, i32, i32, i32, i32, i32, P]
    L.voxzip_build_span_offsets.argtypes = [P, P, P, P, i32, ctypes.c_int64, i32, f32, P, P]
    L.voxzip_build_span_offsets.restype = ctypes.c_int
    L.voxzip_workspace_bytes.argtypes = [i32, i32, i32, i32, i32, i32]
    L.voxzip_workspace_bytes.restype = sz
    i64 = ctypes.c_int64
    L.voxzip_workspace_bytes_ragged.argtypes = [i32, i32, i32, i32, i32, i64, i32]
    L.voxzip_workspace_bytes_ragged.restype = sz
    L.voxzip_fuse_spans_ragged.argtypes = [P, P, P, P, i64, P, P, P, i64, i32, P, P, P, P, P, P, P, P, i64, i32,
                                           P, i32, i32, i32, i32, P]
    L.voxzip_decode_attend_score_ragged.argtypes = [P, P, P, P, P, P, P, P, P, P, P, P, i64, i32, f32, f32,
                                                    i32, i32, i32, i32, i32, P, P, sz, P]
    L.voxzip_evict_compact_ragged.argtypes = [P, P, P, P, P, P, P, P, P, i64, i32, i32, i32, P, P, P,
                                              i32, i32, i32, i32, P, sz, P]
    for f in (L.voxzip_fuse_spans, L.voxzip_decode_attend_score, L.voxzip_evict_compact, L.voxzip_decode_evict,
              L.voxzip_fuse_spans_ragged, L.voxzip_decode_attend_score_ragged, L.voxzip_evict_compact_ragged):
        f.restype = ctypes.c_int
    L.voxzip_status_string.argtypes = [ctypes.c_int]
    L.voxzip_status_string.restype = ctypes.c_char_p
    L.voxzip_last_error.restype = ctypes.c_char_p
    L.voxzip_version.restype = ctypes.c_int
    _lib = L
    return L


def _check(status: int) -> None:
    if status != VZ_OK:
        L = lib()
        raise VoxzipError(status, f"{L.voxzip_status_string(status).decode()}: "
                                  f"{L.voxzip_last_error().decode()}")


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return VZ_F32
    if t.dtype == torch.bfloat16:
        return VZ_BF16
    raise TypeError(f"unsupported tensor dtype {t.dtype}")


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensors must be on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _expect(t, shape, what: str, dtype=None):
    """The C entry points cannot see tensor sizes, so the binding checks them:
    a wrong shape or element type raises here instead of reaching a kernel."""
    if t is None:
        return
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{what} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{what} has dtype {t.dtype}, expected {dtype}")


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def voxzip_build_span_offsets(t_start_ms, t_end_ms, conf, text_len, t_total_ms: int, L_a: int,
                              conf_threshold: float = 0.3):
    """Stage-1 span offsets on the host (numpy arrays in, int32 offsets out:
    n_spans + 1 entries, ready for voxzip_fuse_spans once copied to the GPU)."""
    import numpy as np
    ts = np.ascontiguousarray(t_start_ms, dtype=np.int64)
    te = np.ascontiguousarray(t_end_ms, dtype=np.int64)
    cf = np.ascontiguousarray(conf, dtype=np.float32)
    tl = np.ascontiguousarray(text_len, dtype=np.int32)
    n_seg = len(ts)
    if not (len(te) == len(cf) == len(tl) == n_seg):
        raise ValueError("segment arrays differ in length")
    off = np.zeros(max(int(L_a), 0) + 1, dtype=np.int32)
    n = np.zeros(1, dtype=np.int32)
    hp = lambda a: ctypes.c_void_p(a.ctypes.data)
    _check(lib().voxzip_build_span_offsets(hp(ts), hp(te), hp(cf), hp(tl), n_seg, int(t_total_ms), int(L_a),
                                           float(conf_threshold), hp(off), hp(n)))
    return off[: int(n[0]) + 1].copy()


def voxzip_workspace_bytes(op: int, n_layers: int, n_q_heads: int, kv_heads: int, d: int, cap: int) -> int:
    return int(lib().voxzip_workspace_bytes(op, n_layers, n_q_heads, kv_heads, d, cap))


def voxzip_fuse_spans(k_in, v_in, span_off, k_out, v_out, score_out, pos_out,
                      anchor_k=None, anchor_v=None, stream=None) -> None:
    """Stage-1 fusion; k_in/v_in [L][H][T_in][d], k_out/v_out [L][H][cap][d],
    span_off int32 [n+1] on the device.  v_in and v_out may both be None (k
    alone: the embedding-space form, k_in = [1][1][L_a][d_model])."""
    import torch
    L, H, T_in, d = k_in.shape
    cap = k_out.shape[2]
    n = span_off.numel() - 1
    _expect(v_in, k_in.shape, "v_in", k_in.dtype)
    _expect(k_out, (L, H, cap, d), "k_out", k_in.dtype)
    _expect(v_out, (L, H, cap, d), "v_out", k_in.dtype)
    _expect(score_out, (L, cap), "score_out", torch.float32)
    _expect(pos_out, (L, cap), "pos_out", torch.int32)
    _expect(span_off, (n + 1,), "span_off", torch.int32)
    _expect(anchor_k, (L, H, n, d), "anchor_k", k_in.dtype)
    _expect(anchor_v, (L, H, n, d), "anchor_v", k_in.dtype)
    _check(lib().voxzip_fuse_spans(_ptr(k_in), _ptr(v_in), T_in, _ptr(span_off), n,
                                   _ptr(anchor_k), _ptr(anchor_v), _ptr(k_out), _ptr(v_out),
                                   _ptr(score_out), _ptr(pos_out), L, H, d, cap,
                                   _dtype_code(k_in), _stream(stream)))


def voxzip_decode_attend_score(q, k_new, v_new, k_cache, v_cache, score, pos, out, length, next_pos,
                               gamma, sm_scale=0.0, workspace=None, stream=None) -> None:
    """One decode step over all layers; q/out [L][Hq][d], caches [L][Hkv][cap][d]."""
    import torch
    L, Hkv, cap, d = k_cache.shape
    Hq = q.shape[1]
    dt = k_cache.dtype
    _expect(q, (L, Hq, d), "q", dt)
    _expect(out, (L, Hq, d), "out", dt)
    _expect(k_new, (L, Hkv, d), "k_new", dt)
    _expect(v_new, (L, Hkv, d), "v_new", dt)
    _expect(v_cache, k_cache.shape, "v_cache", dt)
    _expect(score, (L, cap), "score", torch.float32)
    _expect(pos, (L, cap), "pos", torch.int32)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().voxzip_decode_attend_score(_ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache),
                                            _ptr(v_cache), _ptr(score), _ptr(pos), _ptr(out),
                                            int(length), int(next_pos), float(gamma), float(sm_scale),
                                            L, Hq, Hkv, d, cap, _dtype_code(k_cache), _ptr(workspace),
                                            ws_bytes, _stream(stream)))


def voxzip_evict_compact(k_cache, v_cache, score, pos, length, budget, next_pos, n_sink=4, n_recent=-1,
                         kept_pos_out=None, workspace=None, stream=None) -> int:
    """Stage-2 eviction in place; returns the new resident length."""
    import torch
    L, Hkv, cap, d = k_cache.shape
    _expect(v_cache, k_cache.shape, "v_cache", k_cache.dtype)
    _expect(score, (L, cap), "score", torch.float32)
    _expect(pos, (L, cap), "pos", torch.int32)
    _expect(kept_pos_out, (L, int(budget)), "kept_pos_out", torch.int32)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    new_len = ctypes.c_int32(0)
    _check(lib().voxzip_evict_compact(_ptr(k_cache), _ptr(v_cache), _ptr(score), _ptr(pos), int(length),
                                      int(budget), int(n_sink), int(n_recent), int(next_pos),
                                      _ptr(kept_pos_out), ctypes.byref(new_len), L, Hkv, d, cap,
                                      _dtype_code(k_cache), _ptr(workspace), ws_bytes, _stream(stream)))
    return int(new_len.value)


def voxzip_decode_evict(q, k_new, v_new, k_cache, v_cache, score, pos, out, length, next_pos, gamma, budget,
                        n_sink=4, n_recent=-1, kept_pos_out=None, sm_scale=0.0, workspace=None,
                        stream=None) -> int:
    """One generation step: the decode step at (length, next_pos), then the
    eviction of the length + 1 slots it leaves; returns the new resident length
    (the caller's next length; its next next_pos is next_pos + 1)."""
    import torch
    L, Hkv, cap, d = k_cache.shape
    Hq = q.shape[1]
    dt = k_cache.dtype
    _expect(q, (L, Hq, d), "q", dt)
    _expect(out, (L, Hq, d), "out", dt)
    _expect(k_new, (L, Hkv, d), "k_new", dt)
    _expect(v_new, (L, Hkv, d), "v_new", dt)
    _expect(v_cache, k_cache.shape, "v_cache", dt)
    _expect(score, (L, cap), "score", torch.float32)
    _expect(pos, (L, cap), "pos", torch.int32)
    _expect(kept_pos_out, (L, int(budget)), "kept_pos_out", torch.int32)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    new_len = ctypes.c_int32(0)
    _check(lib().voxzip_decode_evict(_ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), _ptr(score),
                                     _ptr(pos), _ptr(out), int(length), int(next_pos), float(gamma),
                                     float(sm_scale), int(budget), int(n_sink), int(n_recent), _ptr(kept_pos_out),
                                     ctypes.byref(new_len), L, Hq, Hkv, d, cap, _dtype_code(k_cache),
                                     _ptr(workspace), ws_bytes, _stream(stream)))
    return int(new_len.value)


def voxzip_decode_evict_noalloc(q, k_new, v_new, k_cache, v_cache, score, pos, out, length, next_pos, gamma,
                                budget, n_sink=4, n_recent=-1, kept_pos_out=None, sm_scale=0.0,
                                stream=None) -> int:
    """voxzip_decode_evict without a workspace (the library's own per-GPU
    scratch array); returns the new resident length."""
    import torch
    L, Hkv, cap, d = k_cache.shape
    Hq = q.shape[1]
    dt = k_cache.dtype
    _expect(q, (L, Hq, d), "q", dt)
    _expect(out, (L, Hq, d), "out", dt)
    _expect(k_new, (L, Hkv, d), "k_new", dt)
    _expect(v_new, (L, Hkv, d), "v_new", dt)
    _expect(v_cache, k_cache.shape, "v_cache", dt)
    _expect(score, (L, cap), "score", torch.float32)
    _expect(pos, (L, cap), "pos", torch.int32)
    _expect(kept_pos_out, (L, int(budget)), "kept_pos_out", torch.int32)
    new_len = ctypes.c_int32(0)
    _check(lib().voxzip_decode_evict_noalloc(_ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache),
                                             _ptr(score), _ptr(pos), _ptr(out), int(length), int(next_pos),
                                             float(gamma), float(sm_scale), int(budget), int(n_sink), int(n_recent),
                                             _ptr(kept_pos_out), ctypes.byref(new_len), L, Hq, Hkv, d, cap,
                                             _dtype_code(k_cache), _stream(stream)))
    return int(new_len.value)


def workspace(op: int, n_layers: int, n_q_heads: int, kv_heads: int, d: int, cap: int, device="cuda"):
    """A zero-filled workspace tensor of the size the library asks for."""
    import torch
    n = voxzip_workspace_bytes(op, n_layers, n_q_heads, kv_heads, d, cap)
    return torch.zeros(max(n, 1), dtype=torch.uint8, device=device)


# ---- ragged batches: packed caches [L][H][total][d], per-sequence device arrays ----

def _seq_array(t, n: int, dtype_name: str, what: str):
    """Device pointer of a per-sequence array (int32 or int64, n entries)."""
    import torch
    want = torch.int64 if dtype_name == "int64" else torch.int32
    if t.dtype != want:
        raise TypeError(f"{what} must be {dtype_name}")
    if t.numel() != n:
        raise ValueError(f"{what} must have one entry per sequence ({n})")
    return _ptr(t)


def voxzip_workspace_bytes_ragged(op: int, n_layers: int, n_q_heads: int, kv_heads: int, d: int, total: int,
                                  n_seqs: int) -> int:
    return int(lib().voxzip_workspace_bytes_ragged(op, n_layers, n_q_heads, kv_heads, d, int(total), n_seqs))


def workspace_ragged(op: int, n_layers: int, n_q_heads: int, kv_heads: int, d: int, total: int, n_seqs: int,
                     device="cuda"):
    """A zero-filled workspace tensor for a ragged call."""
    import torch
    n = voxzip_workspace_bytes_ragged(op, n_layers, n_q_heads, kv_heads, d, total, n_seqs)
    return torch.zeros(max(n, 1), dtype=torch.uint8, device=device)


def voxzip_fuse_spans_ragged(k_in, v_in, in_base, T_in, span_off, off_base, n_spans, max_spans: int,
                             k_out, v_out, score_out, pos_out, seq_base, cap, status=None,
                             anchor_k=None, anchor_v=None, stream=None) -> None:
    """Stage-1 fusion of every sequence of a ragged batch; k_in/v_in
    [L][H][total_in][d], span_off int32 [total_off], outputs [L][H][total][d]."""
    import torch
    L, H, total_in, d = k_in.shape
    total = k_out.shape[2]
    n = seq_base.numel()
    _expect(v_in, k_in.shape, "v_in", k_in.dtype)
    _expect(k_out, (L, H, total, d), "k_out", k_in.dtype)
    _expect(v_out, (L, H, total, d), "v_out", k_in.dtype)
    _expect(score_out, (L, total), "score_out", torch.float32)
    _expect(pos_out, (L, total), "pos_out", torch.int32)
    if span_off.dtype != torch.int32 or span_off.dim() != 1:
        raise TypeError("span_off must be a 1-D int32 tensor")
    _expect(anchor_k, (L, H, total, d), "anchor_k", k_in.dtype)
    _expect(anchor_v, (L, H, total, d), "anchor_v", k_in.dtype)
    _check(lib().voxzip_fuse_spans_ragged(
        _ptr(k_in), _ptr(v_in), _seq_array(in_base, n, "int64", "in_base"), _seq_array(T_in, n, "int32", "T_in"),
        total_in, _ptr(span_off), _seq_array(off_base, n, "int64", "off_base"),
        _seq_array(n_spans, n, "int32", "n_spans"), span_off.numel(), int(max_spans), _ptr(anchor_k),
        _ptr(anchor_v), _ptr(k_out), _ptr(v_out), _ptr(score_out), _ptr(pos_out),
        _seq_array(seq_base, n, "int64", "seq_base"), _seq_array(cap, n, "int32", "cap"), total, n,
        None if status is None else _seq_array(status, n, "int32", "status"), L, H, d, _dtype_code(k_in),
        _stream(stream)))


def voxzip_decode_attend_score_ragged(q, k_new, v_new, k_cache, v_cache, score, pos, out, seq_base, cap, length,
                                      next_pos, gamma, sm_scale=0.0, status=None, workspace=None,
                                      stream=None) -> None:
    """One decode step of every sequence of a ragged batch; q/out [S][L][Hq][d],
    k_new/v_new [S][L][Hkv][d], caches [L][Hkv][total][d]; length and next_pos
    int32 [S] on the device (not advanced here)."""
    import torch
    L, Hkv, total, d = k_cache.shape
    n, Hq = q.shape[0], q.shape[2]
    dt = k_cache.dtype
    _expect(q, (n, L, Hq, d), "q", dt)
    _expect(out, (n, L, Hq, d), "out", dt)
    _expect(k_new, (n, L, Hkv, d), "k_new", dt)
    _expect(v_new, (n, L, Hkv, d), "v_new", dt)
    _expect(v_cache, k_cache.shape, "v_cache", dt)
    _expect(score, (L, total), "score", torch.float32)
    _expect(pos, (L, total), "pos", torch.int32)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().voxzip_decode_attend_score_ragged(
        _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), _ptr(score), _ptr(pos), _ptr(out),
        _seq_array(seq_base, n, "int64", "seq_base"), _seq_array(cap, n, "int32", "cap"),
        _seq_array(length, n, "int32", "length"), _seq_array(next_pos, n, "int32", "next_pos"), total, n,
        float(gamma), float(sm_scale), L, Hq, Hkv, d, _dtype_code(k_cache),
        None if status is None else _seq_array(status, n, "int32", "status"), _ptr(workspace), ws_bytes,
        _stream(stream)))


def voxzip_evict_compact_ragged(k_cache, v_cache, score, pos, seq_base, cap, length, budget, next_pos,
                                n_sink=4, n_recent=-1, kept_pos_out=None, new_len_out=None, status=None,
                                workspace=None, stream=None) -> None:
    """Stage-2 eviction of every sequence of a ragged batch, in place;
    new_len_out (int32 [S], device) receives min(length, budget)."""
    import torch
    L, Hkv, total, d = k_cache.shape
    n = seq_base.numel()
    _expect(v_cache, k_cache.shape, "v_cache", k_cache.dtype)
    _expect(score, (L, total), "score", torch.float32)
    _expect(pos, (L, total), "pos", torch.int32)
    _expect(kept_pos_out, (L, total), "kept_pos_out", torch.int32)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().voxzip_evict_compact_ragged(
        _ptr(k_cache), _ptr(v_cache), _ptr(score), _ptr(pos), _seq_array(seq_base, n, "int64", "seq_base"),
        _seq_array(cap, n, "int32", "cap"), _seq_array(length, n, "int32", "length"),
        _seq_array(budget, n, "int32", "budget"), _seq_array(next_pos, n, "int32", "next_pos"), total, n,
        int(n_sink), int(n_recent), _ptr(kept_pos_out),
        None if new_len_out is None else _seq_array(new_len_out, n, "int32", "new_len_out"),
        None if status is None else _seq_array(status, n, "int32", "status"), L, Hkv, d, _dtype_code(k_cache),
        _ptr(workspace), ws_bytes, _stream(stream)))
