"""GPU: voxzip_decode_evict_noalloc (the generation step on the library's own
per-GPU scratch array, for callers that cannot allocate) gives the bits of
voxzip_decode_evict with a workspace -- every output row, the cache, scores,
positions, kept positions and the new length -- on calls in a row whose
sizes shrink (the array keeps the previous call's contents), and rejects a
call whose workspace would not fit the array before queueing anything."""
import ctypes

import numpy as np
import pytest

import synth
from test_gpu_range import layered_state, step_inputs
from vzt import from_dev, to_dev

pytestmark = pytest.mark.gpu


def _pair(L, Hq, Hkv, d, length, cap, seed):
    import torch
    k, v, s, p = layered_state(seed, L, Hkv, d, cap, length, synth.DT_BF16, length + 9)
    mk = lambda: dict(k=to_dev(k), v=to_dev(v), score=to_dev(s), pos=to_dev(p),
                      out=torch.zeros(L, Hq, d, dtype=torch.bfloat16, device="cuda"))
    return mk(), mk()


@pytest.mark.parametrize("cases", [[
    # (L, Hq, Hkv, length, budget, kept): the 48-layer step at its budget (one
    # launch, fold and eviction in the decode kernel), then smaller calls
    (48, 32, 4, 8192, 8192, False),
    (32, 32, 4, 3000, 2990, True),      # 11 evictions (radix select in the decode kernel), kept positions
    (16, 16, 2, 2000, 1500, False),     # 501 moves: decode, then the eviction launches (lists in the scratch)
]])
def test_noalloc_equals_workspace_call(cases):
    import torch
    import paper_2608_08569_amd as vz
    d = 128
    for i, (L, Hq, Hkv, length, budget, kept) in enumerate(cases):
        cap = length + 2
        a, b = _pair(L, Hq, Hkv, d, length, cap, seed=50 + i)
        q, kn, vn = (to_dev(x) for x in step_inputs(synth.stream_key(51, "noalloc", i), 0, L, Hq, Hkv, d,
                                                    synth.DT_BF16))
        ka = torch.full((L, budget), -1, dtype=torch.int32, device="cuda") if kept else None
        kb = torch.full((L, budget), -1, dtype=torch.int32, device="cuda") if kept else None
        ws = vz.workspace(vz.VZ_OP_DECODE_EVICT, L, Hq, Hkv, d, cap)
        n_a = vz.voxzip_decode_evict(q, kn, vn, a["k"], a["v"], a["score"], a["pos"], a["out"], length, length + 9,
                                     0.95, budget, kept_pos_out=ka, workspace=ws)
        n_b = vz.voxzip_decode_evict_noalloc(q, kn, vn, b["k"], b["v"], b["score"], b["pos"], b["out"], length,
                                             length + 9, 0.95, budget, kept_pos_out=kb)
        torch.cuda.synchronize()
        assert n_a == n_b == min(length + 1, budget), (i, n_a, n_b)
        for name in ("out", "k", "v", "score", "pos"):
            assert np.array_equal(from_dev(a[name]), from_dev(b[name])), (i, name)
        if kept:
            assert np.array_equal(from_dev(ka), from_dev(kb)), i


def test_noalloc_rejects_a_call_beyond_its_scratch():
    """A cache whose workspace exceeds the scratch array: VZ_ERR_WORKSPACE,
    with the sizes in the error text, before any launch (the pointers are
    never dereferenced)."""
    import paper_2608_08569_amd as vz
    L, Hq, Hkv, d, cap = 48, 32, 4, 128, 40000
    assert vz.voxzip_workspace_bytes(vz.VZ_OP_DECODE_EVICT, L, Hq, Hkv, d, cap) > vz.VZ_NOALLOC_SCRATCH_BYTES
    fake = ctypes.c_void_p(0x10000)
    new_len = ctypes.c_int32(-1)
    lib = vz.lib()
    rc = lib.voxzip_decode_evict_noalloc(fake, fake, fake, fake, fake, fake, fake, fake, 30000, 30000, 0.95, 0.0,
                                         8192, 4, -1, None, ctypes.byref(new_len), L, Hq, Hkv, d, cap, vz.VZ_BF16,
                                         None)
    assert rc == vz.VZ_ERR_WORKSPACE
    assert b"bytes of scratch memory" in lib.voxzip_last_error()
    assert new_len.value == -1
