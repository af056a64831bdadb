"""A decode loop over a batch of sequences, on the ragged entry points.

The cache of every sequence lives in one packed ``[L][Hkv][total][d]`` cache
(sequence s at slots ``seq_base[s] ..``), and the per-sequence lengths,
positions and budgets live in device arrays.  No step of the loop reads a
length back to the host, so a whole decode step can be captured once in a HIP
graph and replayed for every token:

* all-layer mode: one decode call over every layer (the layers' queries are
  all known before the step);
* per-layer mode: one decode call per layer, each after a caller-supplied
  function that builds the layer's query from the previous layer's output
  (the dependency a model's forward pass has between layers).

Eviction (Sec. 3.2.2) runs every ``interval`` steps, so two graphs are kept: a
plain step and a step followed by the eviction.  The arithmetic of the method
runs in the library's kernels; this module only sequences the calls and
advances the device-side lengths.
"""
from __future__ import annotations

import numpy as np

from . import (VZ_OP_DECODE, VZ_OP_EVICT, voxzip_decode_attend_score_ragged, voxzip_evict_compact_ragged,
               voxzip_fuse_spans_ragged, workspace_ragged)


class DecodeLoop:
    """Packed state of ``n`` sequences and the calls of one decode step.

    caps, budgets: per-sequence slot capacities and eviction budgets (host
    sequences of ints).  The caller fills the cache with :meth:`fuse` (or
    writes ``k``, ``v``, ``score``, ``pos`` and :meth:`set_lengths` itself).
    """

    def __init__(self, n_layers, n_q_heads, kv_heads, d, caps, budgets, gamma, interval=1, n_sink=4,
                 n_recent=-1, dtype=None, device="cuda"):
        import torch
        self.torch = torch
        dtype = torch.bfloat16 if dtype is None else dtype
        self.L, self.Hq, self.Hkv, self.d = n_layers, n_q_heads, kv_heads, d
        self.gamma, self.interval, self.n_sink, self.n_recent = gamma, interval, n_sink, n_recent
        caps = np.asarray(caps, dtype=np.int64)
        self.n = len(caps)
        base = np.concatenate([[0], np.cumsum(caps)[:-1]]).astype(np.int64)
        self.total = int(caps.sum())
        dev = lambda a, dt: torch.tensor(np.asarray(a), dtype=dt, device=device)
        self.seq_base = dev(base, torch.int64)
        self.cap = dev(caps, torch.int32)
        self.budget = dev(budgets, torch.int32)
        self.length = torch.zeros(self.n, dtype=torch.int32, device=device)
        self.next_pos = torch.zeros_like(self.length)
        self.new_len = torch.zeros_like(self.length)
        self.status = torch.zeros_like(self.length)
        L, H = n_layers, kv_heads
        self.k = torch.zeros(L, H, self.total, d, dtype=dtype, device=device)
        self.v = torch.zeros_like(self.k)
        self.score = torch.zeros(L, self.total, dtype=torch.float32, device=device)
        self.pos = torch.zeros(L, self.total, dtype=torch.int32, device=device)
        self.out = torch.zeros(self.n, L, n_q_heads, d, dtype=dtype, device=device)
        self.out_layers = [torch.zeros(self.n, 1, n_q_heads, d, dtype=dtype, device=device) for _ in range(L)]
        # per-layer calls use one-layer views of the same planes
        self.ws_all = workspace_ragged(VZ_OP_DECODE, L, n_q_heads, kv_heads, d, self.total, self.n, device)
        self.ws_layer = workspace_ragged(VZ_OP_DECODE, 1, n_q_heads, kv_heads, d, self.total, self.n, device)
        self.ws_evict = workspace_ragged(VZ_OP_EVICT, L, n_q_heads, kv_heads, d, self.total, self.n, device)
        self.steps = 0
        self._graphs = {}

    # ---- state ----
    def set_lengths(self, lengths, next_pos=None):
        lengths = np.asarray(lengths, dtype=np.int32)
        self.length.copy_(self.torch.from_numpy(lengths))
        self.next_pos.copy_(self.torch.from_numpy(lengths if next_pos is None else np.asarray(next_pos, np.int32)))

    def fuse(self, k_in, v_in, in_base, T_in, span_off, off_base, n_spans, max_spans):
        """Stage-1 fusion of every sequence's prefill into the packed cache;
        lengths and positions start at the span counts."""
        voxzip_fuse_spans_ragged(k_in, v_in, in_base, T_in, span_off, off_base, n_spans, max_spans, self.k,
                                 self.v, self.score, self.pos, self.seq_base, self.cap, status=self.status)
        self.length.copy_(n_spans)
        self.next_pos.copy_(n_spans)
        self.steps = 0

    # ---- one step ----
    def _decode_all(self, q, k_new, v_new):
        voxzip_decode_attend_score_ragged(q, k_new, v_new, self.k, self.v, self.score, self.pos, self.out,
                                          self.seq_base, self.cap, self.length, self.next_pos, self.gamma,
                                          status=self.status, workspace=self.ws_all)

    def _decode_layers(self, q, k_new, v_new, layer_query):
        for l in range(self.L):
            ql = layer_query(l, q, self.out_layers)  # [n][1][Hq][d]; may read out_layers[l - 1]
            voxzip_decode_attend_score_ragged(
                ql, k_new[l], v_new[l], self.k[l: l + 1], self.v[l: l + 1], self.score[l: l + 1],
                self.pos[l: l + 1], self.out_layers[l], self.seq_base, self.cap, self.length, self.next_pos,
                self.gamma, status=self.status, workspace=self.ws_layer)

    def _evict(self):
        voxzip_evict_compact_ragged(self.k, self.v, self.score, self.pos, self.seq_base, self.cap, self.length,
                                    self.budget, self.next_pos, n_sink=self.n_sink, n_recent=self.n_recent,
                                    new_len_out=self.new_len, status=self.status, workspace=self.ws_evict)
        self.length.copy_(self.new_len)

    def _step(self, q, k_new, v_new, layer_query, evict):
        if layer_query is None:
            self._decode_all(q, k_new, v_new)
        else:
            self._decode_layers(q, k_new, v_new, layer_query)
        self.length.add_(1)
        self.next_pos.add_(1)
        if evict:
            self._evict()

    def _evict_due(self) -> bool:
        return (self.steps + 1) % self.interval == 0

    def step(self, q, k_new, v_new, layer_query=None):
        """One decode step of every sequence, launched eagerly.

        All-layer mode: q [n][L][Hq][d], k_new / v_new [n][L][Hkv][d]; the
        outputs land in ``out`` [n][L][Hq][d].  Per-layer mode (with
        ``layer_query(l, q, out_layers)`` returning layer l's query
        [n][1][Hq][d]): k_new / v_new are layer-major [L][n][1][Hkv][d] and the
        outputs land in ``out_layers[l]`` [n][1][Hq][d]."""
        self._step(q, k_new, v_new, layer_query, self._evict_due())
        self.steps += 1

    # ---- HIP graphs ----
    def capture(self, q, k_new, v_new, layer_query=None):
        """Capture the plain step and the step with eviction as HIP graphs
        reading the given input buffers (refill them before each replay).
        One eager warm-up step runs first; the state is restored afterwards,
        so capture() leaves the cache as it found it."""
        torch = self.torch
        state = (self.k, self.v, self.score, self.pos, self.length, self.next_pos)
        saved = [t.clone() for t in state]
        stream = torch.cuda.Stream()
        stream.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(stream):
            self._step(q, k_new, v_new, layer_query, True)  # warm-up outside capture
        torch.cuda.current_stream().wait_stream(stream)
        for evict in (False, True):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                self._step(q, k_new, v_new, layer_query, evict)
            self._graphs[evict] = g
        torch.cuda.synchronize()
        # capture only records work; undo the warm-up step
        for t, s in zip(state, saved):
            t.copy_(s)
        torch.cuda.synchronize()

    def replay(self):
        """One decode step by graph replay (the inputs given to capture() hold
        this step's values)."""
        self._graphs[self._evict_due()].replay()
        self.steps += 1
