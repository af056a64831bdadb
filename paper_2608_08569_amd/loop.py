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

Eviction (Sec. 3.2.2) runs every ``interval`` steps of each sequence, so two
graphs are kept: a plain step and a step followed by the eviction.

Continuous batching: each sequence owns a fixed region of the packed planes
(a batch slot).  A finished request leaves with :meth:`retire`, which marks
its slot idle (capacity 0 on the device: every call skips it), and a new
request joins with :meth:`admit`, which fuses its prefill (Stage 1) into a
free slot and restores the slot's capacity, between two steps.  Neither
changes a launch shape, so captured step graphs keep replaying.  Each
sequence counts its own steps on the device, and its evictions fall on its
own ``interval`` boundaries (a sequence not due this step is given an
unreachable budget), so a request behaves exactly as it would alone whenever
it joins.

The arithmetic of the method runs in the library's kernels; this module only
sequences the calls and advances the device-side lengths and step counts.
"""
from __future__ import annotations

import numpy as np

from . import (VZ_OP_DECODE, VZ_OP_EVICT, voxzip_decode_attend_score_ragged, voxzip_evict_compact_ragged,
               voxzip_fuse_spans_ragged, workspace_ragged)


class DecodeLoop:
    """Packed state of ``n`` batch slots and the calls of one decode step.

    caps, budgets: per-slot capacities (slot regions of the planes) and
    eviction budgets (host sequences of ints).  Every slot starts active; the
    caller fills the cache with :meth:`fuse` (or writes ``k``, ``v``,
    ``score``, ``pos`` and :meth:`set_lengths` itself), or retires slots and
    admits requests into them one by one (:meth:`retire`, :meth:`admit`).
    """

    NEVER = 1 << 30  # budget of a sequence whose eviction is not due this step

    def __init__(self, n_layers, n_q_heads, kv_heads, d, caps, budgets, gamma, interval=1, n_sink=4,
                 n_recent=-1, dtype=None, device="cuda"):
        import torch
        self.torch = torch
        dtype = torch.bfloat16 if dtype is None else dtype
        self.L, self.Hq, self.Hkv, self.d = n_layers, n_q_heads, kv_heads, d
        self.gamma, self.interval, self.n_sink, self.n_recent = gamma, interval, n_sink, n_recent
        caps = np.asarray(caps, dtype=np.int64)
        self.n = len(caps)
        self.slot_cap = caps.copy()
        self.active = np.ones(self.n, dtype=bool)
        self.age_h = np.zeros(self.n, dtype=np.int64)  # steps since each slot's request started (host mirror)
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
        self.age = torch.zeros_like(self.length)  # steps since each slot's request started
        self._rem = torch.zeros_like(self.length)
        self._due = torch.zeros(self.n, dtype=torch.bool, device=device)
        self._never = torch.full((self.n,), self.NEVER, dtype=torch.int32, device=device)
        self._eff_budget = torch.zeros_like(self.length)
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
        self.age.zero_()
        self.age_h[:] = 0
        self.steps = 0

    # ---- continuous batching ----
    def retire(self, s: int):
        """Request in slot s leaves the batch: the slot turns idle (capacity
        0 on the device), so every later call skips it.  Its cache rows and
        last outputs stay in place until the slot is reused."""
        self.cap[s] = 0
        self.active[s] = False

    def admit(self, s: int, k_in, v_in, span_off, budget: int | None = None):
        """A new request joins the batch in idle slot s: its prefill K/V
        (``[L][Hkv][T_in][d]``) is fused over its spans (``span_off``, int32
        ``[n_spans + 1]`` on the device) into the slot's region (Sec. 3.2.1),
        its length and next position start at n_spans, its step count at 0,
        and the slot's capacity comes back.  ``budget`` replaces the slot's
        eviction budget when given.  Returns n_spans."""
        torch = self.torch
        if self.active[s]:
            raise ValueError(f"slot {s} is in use: retire it first")
        L, H, T_in, d = k_in.shape
        if (L, H, d) != (self.L, self.Hkv, self.d):
            raise ValueError(f"prefill has shape {tuple(k_in.shape)}, expected [{self.L}][{self.Hkv}][T][{self.d}]")
        n_spans = int(span_off.numel()) - 1
        if n_spans < 1 or n_spans + 1 > self.slot_cap[s]:
            raise ValueError(f"{n_spans} spans do not fit slot {s} of {self.slot_cap[s]} slots with a free one")
        dev = lambda a, dt: torch.tensor(a, dtype=dt, device=self.k.device)
        one = np.zeros(self.n, dtype=np.int64)
        at = lambda x: np.where(np.arange(self.n) == s, x, 0)
        cap_adm = at(self.slot_cap[s])  # every other slot idle for this call
        voxzip_fuse_spans_ragged(k_in, v_in, dev(one, torch.int64), dev(at(T_in), torch.int32), span_off,
                                 dev(one, torch.int64), dev(at(n_spans), torch.int32), n_spans, self.k, self.v,
                                 self.score, self.pos, self.seq_base, dev(cap_adm, torch.int32),
                                 status=self.status)
        self.length[s] = n_spans
        self.next_pos[s] = n_spans
        self.age[s] = 0
        if budget is not None:
            self.budget[s] = int(budget)
        self.cap[s] = int(self.slot_cap[s])
        self.active[s] = True
        self.age_h[s] = 0
        return n_spans

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
        budget = self.budget
        if self.interval > 1:
            # only sequences at their own interval boundary evict this step
            torch = self.torch
            torch.remainder(self.age, self.interval, out=self._rem)
            torch.eq(self._rem, 0, out=self._due)
            torch.where(self._due, self.budget, self._never, out=self._eff_budget)
            budget = self._eff_budget
        voxzip_evict_compact_ragged(self.k, self.v, self.score, self.pos, self.seq_base, self.cap, self.length,
                                    budget, self.next_pos, n_sink=self.n_sink, n_recent=self.n_recent,
                                    new_len_out=self.new_len, status=self.status, workspace=self.ws_evict)
        self.length.copy_(self.new_len)

    def _step(self, q, k_new, v_new, layer_query, evict):
        if layer_query is None:
            self._decode_all(q, k_new, v_new)
        else:
            self._decode_layers(q, k_new, v_new, layer_query)
        self.length.add_(1)
        self.next_pos.add_(1)
        self.age.add_(1)
        if evict:
            self._evict()

    def _evict_due(self) -> bool:
        """Whether some active sequence reaches its eviction step now."""
        return bool(np.any(self.active & ((self.age_h + 1) % self.interval == 0)))

    def step(self, q, k_new, v_new, layer_query=None):
        """One decode step of every sequence, launched eagerly.

        All-layer mode: q [n][L][Hq][d], k_new / v_new [n][L][Hkv][d]; the
        outputs land in ``out`` [n][L][Hq][d].  Per-layer mode (with
        ``layer_query(l, q, out_layers)`` returning layer l's query
        [n][1][Hq][d]): k_new / v_new are layer-major [L][n][1][Hkv][d] and the
        outputs land in ``out_layers[l]`` [n][1][Hq][d]."""
        self._step(q, k_new, v_new, layer_query, self._evict_due())
        self.steps += 1
        self.age_h += 1

    # ---- HIP graphs ----
    def capture(self, q, k_new, v_new, layer_query=None):
        """Capture the plain step and the step with eviction as HIP graphs
        reading the given input buffers (refill them before each replay).
        One eager warm-up step runs first; the state is restored afterwards,
        so capture() leaves the cache as it found it."""
        torch = self.torch
        state = (self.k, self.v, self.score, self.pos, self.length, self.next_pos, self.age)
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
        self.age_h += 1
