"""The C ABI without a GPU: the library loads, exports every entry point the
header declares, and rejects bad arguments on the host with the documented
status codes (no HIP call is made on these paths)."""
import ctypes
import os
import re

import pytest

import paper_2608_08569_amd as vz

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = ctypes.c_void_p(0x10000)  # never dereferenced: every case fails validation first
MISALIGNED = ctypes.c_void_p(0x10008)  # a workspace address off the 16-byte grid


def _declared():
    names = []
    for fn in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if fn.endswith(".h"):
            txt = open(os.path.join(ROOT, "include", fn)).read()
            names += re.findall(r"VZ_API\s+[\w\s\*]+?\b(voxzip_\w+)\s*\(", txt)
    return names


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert {"voxzip_fuse_spans", "voxzip_decode_attend_score", "voxzip_evict_compact"} <= set(names)
    L = vz.lib()
    for n in names:
        assert hasattr(L, n), n


def test_status_strings_and_version():
    L = vz.lib()
    assert L.voxzip_version() >= 100
    for code in (0, -1, -2, -3, -4, -5, -6, vz.VZ_IDLE):
        assert L.voxzip_status_string(code).decode() not in ("", "unknown status")


def _decode(**kw):
    a = dict(q=FAKE, kn=FAKE, vn=FAKE, kc=FAKE, vc=FAKE, s=FAKE, p=FAKE, o=FAKE, len=10, next_pos=10,
             gamma=0.95, scale=0.0, L=2, Hq=32, Hkv=4, d=128, cap=64, dtype=vz.VZ_BF16, ws=FAKE,
             ws_bytes=1 << 30)
    a.update(kw)
    return vz.lib().voxzip_decode_attend_score(a["q"], a["kn"], a["vn"], a["kc"], a["vc"], a["s"], a["p"],
                                               a["o"], a["len"], a["next_pos"], a["gamma"], a["scale"],
                                               a["L"], a["Hq"], a["Hkv"], a["d"], a["cap"], a["dtype"],
                                               a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), vz.VZ_ERR_INVALID),
    (dict(gamma=1.5), vz.VZ_ERR_INVALID),
    (dict(gamma=-0.1), vz.VZ_ERR_INVALID),
    (dict(gamma=float("nan")), vz.VZ_ERR_INVALID),
    (dict(scale=float("inf")), vz.VZ_ERR_INVALID),
    (dict(len=-1), vz.VZ_ERR_INVALID),
    (dict(len=64), vz.VZ_ERR_CAPACITY),
    (dict(Hq=30), vz.VZ_ERR_SHAPE),
    (dict(Hq=0), vz.VZ_ERR_SHAPE),
    (dict(L=0), vz.VZ_ERR_SHAPE),
    (dict(Hq=68, Hkv=4), vz.VZ_ERR_UNSUPPORTED),
    (dict(d=96), vz.VZ_ERR_UNSUPPORTED),
    (dict(d=256), vz.VZ_ERR_UNSUPPORTED),    # wide rows are for fusion only
    (dict(dtype=7), vz.VZ_ERR_UNSUPPORTED),
    (dict(ws=None), vz.VZ_ERR_WORKSPACE),
    (dict(ws_bytes=16), vz.VZ_ERR_WORKSPACE),
    (dict(ws=MISALIGNED), vz.VZ_ERR_WORKSPACE),   # 8 bytes past a 16-byte boundary
])
def test_decode_rejects(kw, code):
    assert _decode(**kw) == code
    assert vz.lib().voxzip_last_error().decode().startswith("voxzip_decode_attend_score")


def _evict(**kw):
    a = dict(kc=FAKE, vc=FAKE, s=FAKE, p=FAKE, len=100, budget=50, n_sink=4, n_recent=-1, next_pos=100,
             kept=None, L=2, Hkv=4, d=128, cap=128, dtype=vz.VZ_BF16, ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    nl = ctypes.c_int32(-7)
    rc = vz.lib().voxzip_evict_compact(a["kc"], a["vc"], a["s"], a["p"], a["len"], a["budget"], a["n_sink"],
                                       a["n_recent"], a["next_pos"], a["kept"], ctypes.byref(nl), a["L"],
                                       a["Hkv"], a["d"], a["cap"], a["dtype"], a["ws"], a["ws_bytes"], None)
    return rc, nl.value


@pytest.mark.parametrize("kw,code", [
    (dict(s=None), vz.VZ_ERR_INVALID),
    (dict(budget=0), vz.VZ_ERR_INVALID),
    (dict(n_sink=-1), vz.VZ_ERR_INVALID),
    (dict(n_sink=40, n_recent=20), vz.VZ_ERR_INVALID),
    (dict(next_pos=99), vz.VZ_ERR_INVALID),
    (dict(len=129), vz.VZ_ERR_CAPACITY),
    (dict(d=32), vz.VZ_ERR_UNSUPPORTED),
    (dict(kept=FAKE, next_pos=(1 << 18) + 1), vz.VZ_ERR_UNSUPPORTED),
    (dict(ws=None), vz.VZ_ERR_WORKSPACE),
    (dict(ws_bytes=8), vz.VZ_ERR_WORKSPACE),
    (dict(ws=MISALIGNED), vz.VZ_ERR_WORKSPACE),
])
def test_evict_rejects(kw, code):
    rc, _ = _evict(**kw)
    assert rc == code


def test_evict_without_work_returns_length_and_queues_nothing():
    rc, nl = _evict(len=40, budget=50, ws=None, ws_bytes=0)
    assert rc == vz.VZ_OK and nl == 40


def _fuse(**kw):
    a = dict(ki=ctypes.c_void_p(0x100000), vi=ctypes.c_void_p(0x200000), T=100, off=FAKE, n=30, ak=None,
             av=None, ko=ctypes.c_void_p(0x400000), vo=ctypes.c_void_p(0x800000), so=FAKE, po=FAKE,
             L=1, H=1, d=64, cap=32, dtype=vz.VZ_F32)
    a.update(kw)
    return vz.lib().voxzip_fuse_spans(a["ki"], a["vi"], a["T"], a["off"], a["n"], a["ak"], a["av"], a["ko"],
                                      a["vo"], a["so"], a["po"], a["L"], a["H"], a["d"], a["cap"], a["dtype"],
                                      None)


@pytest.mark.parametrize("kw,code", [
    (dict(off=None), vz.VZ_ERR_INVALID),
    (dict(ak=FAKE), vz.VZ_ERR_INVALID),
    (dict(ko=ctypes.c_void_p(0x100000 + 64)), vz.VZ_ERR_INVALID),   # k_out inside k_in
    (dict(vo=ctypes.c_void_p(0x400000 + 256)), vz.VZ_ERR_INVALID),  # v_out overlaps k_out
    (dict(n=33), vz.VZ_ERR_CAPACITY),
    (dict(n=101, cap=200), vz.VZ_ERR_SHAPE),
    (dict(d=102), vz.VZ_ERR_UNSUPPORTED),                          # float32 rows: a multiple of 4 elements
    (dict(d=100, dtype=vz.VZ_BF16), vz.VZ_ERR_UNSUPPORTED),        # bf16 rows: a multiple of 8 elements
    (dict(d=16392, dtype=vz.VZ_BF16), vz.VZ_ERR_UNSUPPORTED),      # wider than 16384
    (dict(vi=None), vz.VZ_ERR_INVALID),                            # v_out without v_in
    (dict(vo=None), vz.VZ_ERR_INVALID),                            # v_in without v_out
    (dict(vi=None, vo=None, ak=FAKE, av=FAKE), vz.VZ_ERR_INVALID),  # anchor_v without v_in
])
def test_fuse_rejects(kw, code):
    assert _fuse(**kw) == code


def test_workspace_sizes():
    L = vz.lib()
    assert L.voxzip_workspace_bytes(vz.VZ_OP_DECODE, 48, 32, 4, 128, 8210) > 0
    assert L.voxzip_workspace_bytes(vz.VZ_OP_EVICT, 48, 32, 4, 128, 8210) > 0
    assert L.voxzip_workspace_bytes(99, 48, 32, 4, 128, 8210) == 0
    assert L.voxzip_workspace_bytes(vz.VZ_OP_DECODE, 0, 32, 4, 128, 8210) == 0


def test_binding_has_no_cpu_path():
    # the product path must refuse host tensors instead of computing anything
    torch = pytest.importorskip("torch")
    x = torch.zeros(1, 1, 4, 64)
    with pytest.raises(ValueError):
        vz.voxzip_fuse_spans(x, x, torch.zeros(2, dtype=torch.int32), x, x, torch.zeros(1, 4),
                             torch.zeros(1, 4, dtype=torch.int32))


# ---- ragged twins: host-side rejections (no HIP call on these paths) ----

def _decode_ragged(**kw):
    a = dict(q=FAKE, kn=FAKE, vn=FAKE, kc=FAKE, vc=FAKE, s=FAKE, p=FAKE, o=FAKE, base=FAKE, cap=FAKE, len=FAKE,
             nxt=FAKE, total=4096, n=4, gamma=0.95, scale=0.0, L=2, Hq=32, Hkv=4, d=128, dtype=vz.VZ_BF16,
             status=None, ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    return vz.lib().voxzip_decode_attend_score_ragged(
        a["q"], a["kn"], a["vn"], a["kc"], a["vc"], a["s"], a["p"], a["o"], a["base"], a["cap"], a["len"],
        a["nxt"], a["total"], a["n"], a["gamma"], a["scale"], a["L"], a["Hq"], a["Hkv"], a["d"], a["dtype"],
        a["status"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(len=None), vz.VZ_ERR_INVALID),
    (dict(base=None), vz.VZ_ERR_INVALID),
    (dict(gamma=2.0), vz.VZ_ERR_INVALID),
    (dict(n=0), vz.VZ_ERR_SHAPE),
    (dict(n=40000), vz.VZ_ERR_SHAPE),
    (dict(total=0), vz.VZ_ERR_SHAPE),
    (dict(total=(1 << 26) + 1), vz.VZ_ERR_SHAPE),
    (dict(Hq=30), vz.VZ_ERR_SHAPE),
    (dict(d=96), vz.VZ_ERR_UNSUPPORTED),
    (dict(L=70000), vz.VZ_ERR_UNSUPPORTED),
    (dict(ws_bytes=64), vz.VZ_ERR_WORKSPACE),
    (dict(ws=MISALIGNED), vz.VZ_ERR_WORKSPACE),
])
def test_decode_ragged_rejects(kw, code):
    assert _decode_ragged(**kw) == code
    assert vz.lib().voxzip_last_error().decode().startswith("voxzip_decode_attend_score_ragged")


def _evict_ragged(**kw):
    a = dict(kc=FAKE, vc=FAKE, s=FAKE, p=FAKE, base=FAKE, cap=FAKE, len=ctypes.c_void_p(0x20000), budget=FAKE,
             nxt=FAKE, total=4096, n=4, n_sink=4, n_recent=-1, kept=None, new_len=None, status=None, L=2, Hkv=4,
             d=128, dtype=vz.VZ_BF16, ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    return vz.lib().voxzip_evict_compact_ragged(
        a["kc"], a["vc"], a["s"], a["p"], a["base"], a["cap"], a["len"], a["budget"], a["nxt"], a["total"], a["n"],
        a["n_sink"], a["n_recent"], a["kept"], a["new_len"], a["status"], a["L"], a["Hkv"], a["d"], a["dtype"],
        a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(budget=None), vz.VZ_ERR_INVALID),
    (dict(n_sink=-1), vz.VZ_ERR_INVALID),
    (dict(new_len=ctypes.c_void_p(0x20000 + 8)), vz.VZ_ERR_INVALID),   # overlaps len
    (dict(n=0), vz.VZ_ERR_SHAPE),
    (dict(dtype=5), vz.VZ_ERR_UNSUPPORTED),
    (dict(ws=None), vz.VZ_ERR_WORKSPACE),
])
def test_evict_ragged_rejects(kw, code):
    assert _evict_ragged(**kw) == code


def _fuse_ragged(**kw):
    a = dict(ki=ctypes.c_void_p(0x100000), vi=ctypes.c_void_p(0x200000), ib=FAKE, T=FAKE, total_in=100, off=FAKE,
             ob=FAKE, ns=FAKE, total_off=50, max_spans=30, ak=None, av=None, ko=ctypes.c_void_p(0x400000),
             vo=ctypes.c_void_p(0x800000), so=FAKE, po=FAKE, base=FAKE, cap=FAKE, total=64, n=2, status=None,
             L=1, H=1, d=64, dtype=vz.VZ_F32)
    a.update(kw)
    return vz.lib().voxzip_fuse_spans_ragged(
        a["ki"], a["vi"], a["ib"], a["T"], a["total_in"], a["off"], a["ob"], a["ns"], a["total_off"],
        a["max_spans"], a["ak"], a["av"], a["ko"], a["vo"], a["so"], a["po"], a["base"], a["cap"], a["total"],
        a["n"], a["status"], a["L"], a["H"], a["d"], a["dtype"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(ob=None), vz.VZ_ERR_INVALID),
    (dict(ak=FAKE), vz.VZ_ERR_INVALID),
    (dict(ko=ctypes.c_void_p(0x100000 + 64)), vz.VZ_ERR_INVALID),   # k_out inside k_in
    (dict(max_spans=-1), vz.VZ_ERR_SHAPE),
    (dict(max_spans=65), vz.VZ_ERR_SHAPE),                          # more spans than output slots
    (dict(total_off=0), vz.VZ_ERR_SHAPE),
    (dict(n=0), vz.VZ_ERR_SHAPE),
    (dict(d=102), vz.VZ_ERR_UNSUPPORTED),
    (dict(vi=None), vz.VZ_ERR_INVALID),
    (dict(vi=None, vo=None, ak=FAKE, av=FAKE), vz.VZ_ERR_INVALID),
])
def test_fuse_ragged_rejects(kw, code):
    assert _fuse_ragged(**kw) == code


def test_ragged_workspace_sizes():
    L = vz.lib()
    one = L.voxzip_workspace_bytes(vz.VZ_OP_DECODE, 48, 32, 4, 128, 8210)
    rag = L.voxzip_workspace_bytes_ragged(vz.VZ_OP_DECODE, 48, 32, 4, 128, 8210, 1)
    assert rag >= one > 0
    assert L.voxzip_workspace_bytes_ragged(vz.VZ_OP_EVICT, 48, 32, 4, 128, 80000, 16) > 0
    assert L.voxzip_workspace_bytes_ragged(vz.VZ_OP_DECODE, 48, 32, 4, 128, 80000, 0) == 0
    assert L.voxzip_workspace_bytes_ragged(vz.VZ_OP_DECODE, 48, 32, 4, 128, 1 << 27, 4) == 0
    assert L.voxzip_workspace_bytes_ragged(7, 48, 32, 4, 128, 80000, 16) == 0


def test_binding_checks_shapes_before_any_launch():
    # wrong shapes never reach the library (no GPU needed: the check comes first)
    torch = pytest.importorskip("torch")

    class Meta:  # a tensor stand-in with a shape and a dtype only
        def __init__(self, shape, dtype):
            self.shape, self.dtype = shape, dtype

    bf, f32, i32 = torch.bfloat16, torch.float32, torch.int32
    with pytest.raises(ValueError, match="q has shape"):
        vz._expect(Meta((3, 32, 128), bf), (2, 32, 128), "q", bf)
    with pytest.raises(TypeError, match="score has dtype"):
        vz._expect(Meta((2, 64), i32), (2, 64), "score", f32)
    vz._expect(Meta((2, 64), f32), (2, 64), "score", f32)
    vz._expect(None, (2, 64), "kept_pos_out", i32)


def _step(**kw):
    a = dict(q=FAKE, kn=FAKE, vn=FAKE, kc=FAKE, vc=FAKE, s=FAKE, p=FAKE, o=FAKE, len=10, next_pos=10,
             gamma=0.95, scale=0.0, budget=8, n_sink=4, n_recent=-1, kept=None, nl=ctypes.byref(ctypes.c_int32()),
             L=2, Hq=32, Hkv=4, d=128, cap=64, dtype=vz.VZ_BF16, ws=FAKE, ws_bytes=0)
    a.update(kw)
    return vz.lib().voxzip_decode_evict(a["q"], a["kn"], a["vn"], a["kc"], a["vc"], a["s"], a["p"], a["o"],
                                        a["len"], a["next_pos"], a["gamma"], a["scale"], a["budget"],
                                        a["n_sink"], a["n_recent"], a["kept"], a["nl"], a["L"], a["Hq"],
                                        a["Hkv"], a["d"], a["cap"], a["dtype"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), vz.VZ_ERR_INVALID),
    (dict(nl=None), vz.VZ_ERR_INVALID),
    (dict(gamma=2.0), vz.VZ_ERR_INVALID),
    (dict(len=64, next_pos=70), vz.VZ_ERR_CAPACITY),          # no slot for the new token
    (dict(budget=0), vz.VZ_ERR_INVALID),
    (dict(n_sink=4, n_recent=5), vz.VZ_ERR_INVALID),          # windows exceed the budget
    (dict(next_pos=9), vz.VZ_ERR_INVALID),                    # next_pos below len
    (dict(next_pos=2 ** 31 - 1), vz.VZ_ERR_INVALID),          # next_pos + 1 overflows
    (dict(kept=FAKE, next_pos=1 << 18), vz.VZ_ERR_UNSUPPORTED),
    (dict(d=96), vz.VZ_ERR_UNSUPPORTED),
    (dict(ws=None, ws_bytes=1 << 20), vz.VZ_ERR_WORKSPACE),
    (dict(ws_bytes=16), vz.VZ_ERR_WORKSPACE),                 # every case stops before any launch
    (dict(ws=MISALIGNED, ws_bytes=1 << 30), vz.VZ_ERR_WORKSPACE),
])
def test_step_rejects(kw, code):
    assert _step(**kw) == code
    assert vz.lib().voxzip_last_error().decode().startswith("voxzip_decode_evict")


def test_step_workspace_holds_both_parts():
    for L, Hq, Hkv, d, cap in ((48, 32, 4, 128, 8194), (2, 8, 8, 64, 100)):
        dec = vz.voxzip_workspace_bytes(vz.VZ_OP_DECODE, L, Hq, Hkv, d, cap)
        ev = vz.voxzip_workspace_bytes(vz.VZ_OP_EVICT, L, Hq, Hkv, d, cap)
        both = vz.voxzip_workspace_bytes(vz.VZ_OP_DECODE_EVICT, L, Hq, Hkv, d, cap)
        assert dec + ev <= both <= dec + ev + 256

