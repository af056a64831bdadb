#!/usr/bin/env python3
"""Benchmark of the VoxZip hot path on one MI355X.

Workload: the 32k-context long-audio cache -- 48 layers, 32 query / 4 KV
heads, head size 128, bfloat16, 32,768 audio tokens fused by Stage 1 into
~8.2k span tokens, budget B = 8192 (4x), gamma = 0.95, 256 decode steps with
an eviction check after every step.

One bench step = one request over that workload: Stage-1 fusion of the
prefill cache, then 256 decode steps (append, attention, decayed score,
eviction).  Inputs are generated once and stay resident in HBM.  The value is
decode tokens per second over whole requests (fusion included).

Also reported:
  roofline      the generation step's kernel (the dominant one, one launch
                per step: attend + score + evict): algorithmic bytes per
                launch over its mean duration, timed with HIP events on the
                stream it runs on, against 8 TB/s;
  cpu_baseline  the fp64 oracle on the host cores over a bounded sample.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

HBM_PEAK_GBS = 8000.0
PROFILE_PMC = os.path.join(ROOT, "profiles", "decode_long32k_pmc.md")
PROFILE_KEPT = os.path.join(ROOT, "profiles", "kept_sets_long32k.md")
KERNEL_SRC = [os.path.join(ROOT, "paper_2608_08569_amd", "csrc", f)
              for f in ("decode_range.hip", "decode_mfma.h", "select.h", "vz_internal.h")]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def decode_bytes_per_layer(T, Hq, Hkv, d, s):
    """Algorithmic HBM bytes of one decode launch, per layer: every resident
    key and value row once, the score read-modify-write, the appended row, q and o."""
    return T * (2 * Hkv * d * s + 8) + 2 * Hkv * d * s + 2 * Hq * d * s


def evict_bytes_per_layer(T, E, Hkv, d, s):
    """Score and position read of every slot plus the moved rows (read + write)."""
    return 8 * T + 2 * E * (2 * Hkv * d * s + 8)


def kernel_sha() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SRC:
        if os.path.exists(p):
            h.update(open(p, "rb").read())
    return h.hexdigest()[:16]


def read_traffic():
    """HBM bytes per generation-step launch from the committed rocprofv3
    counter summary, only if it was taken on the current kernel source."""
    if not os.path.exists(PROFILE_PMC):
        return None
    txt = open(PROFILE_PMC).read()
    m_sha = re.search(r"kernel_source_sha:\s*([0-9a-f]+)", txt)
    m_b = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", txt)
    if not (m_sha and m_b) or m_sha.group(1) != kernel_sha():
        return None
    return float(m_b.group(1))


def read_kept_agreement():
    """The free-running kept-set agreement with the oracle recorded by
    ``bench.py --kept-sets`` (informational), only if it was taken on the
    current kernel source."""
    if not os.path.exists(PROFILE_KEPT):
        return None
    txt = open(PROFILE_KEPT).read()
    f = {k: re.search(rf"{k}:\s*(\S+)", txt) for k in ("kernel_source_sha", "kept_jaccard_min", "kept_jaccard_mean",
                                                       "kept_layers")}
    if not all(f.values()) or f["kernel_source_sha"].group(1) != kernel_sha():
        return None
    return {"jaccard_min": float(f["kept_jaccard_min"].group(1)),
            "jaccard_mean": float(f["kept_jaccard_mean"].group(1)),
            "layers": [int(x) for x in f["kept_layers"].group(1).split(",")], "steps": 256,
            "source": "profiles/kept_sets_long32k.md (bench.py --kept-sets: GPU and oracle free running)"}


def cpu_model() -> str:
    """The host CPU's model string (Linux), or "unknown"."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def copy_gbps(torch, stream, n_bytes: int = 1 << 30, reps: int = 10) -> float:
    """Bytes moved (read + written) per second by a plain device-to-device
    copy of n_bytes, timed with HIP events: the practical ceiling beside the
    8 TB/s peak."""
    a = torch.empty(n_bytes, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    for _ in range(2):
        b.copy_(a)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        b.copy_(a)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del a, b
    return 2 * n_bytes / (ms * 1e-3) / 1e9


def cpu_report(max_seconds: float = 8.0) -> dict:
    """The oracle as it stands, timed on the host per workload: single-threaded
    and with its OpenMP loop over layers on several cores (the batch: a pool
    of threads over sequences, one oracle thread each).  The layer workload
    runs whole; long32k and aggr64k on a sample of layers and batch16 on
    layer 0 of every sequence, their step times scaled to whole-model
    tokens.  Each run steps until max_seconds; the first step of aggr64k
    holds its large eviction.  Reports median step times and tokens/s."""
    import concurrent.futures as cf
    import oracle
    lib = oracle.load()
    n_all = oracle.threads(lib)
    rep = {"cpu_model": cpu_model(), "nproc": os.cpu_count(), "omp_max_threads": n_all, "workloads": []}

    def timed(step, steps_max):
        times, t_all = [], time.time()
        for t in range(steps_max):
            ts = time.perf_counter()
            step(t)
            times.append(time.perf_counter() - ts)
            if time.time() - t_all > max_seconds:
                break
        return float(np.median(times)), len(times)

    for name in ("layer", "long32k", "aggr64k"):
        w = synth.workload(name)
        off = synth.offsets_from_lengths(synth.span_lengths(w))
        n = len(off) - 1
        for threads in ((1,) if w.n_layers == 1 else (1, min(n_all, 8))):
            sample = 1 if w.n_layers == 1 else (2 if threads == 1 else threads)
            ls = range(min(sample, w.n_layers))
            oracle.set_threads(threads, lib)
            run = oracle.Run(synth.prefill_kv(w, "k", layers=ls), synth.prefill_kv(w, "v", layers=ls), off, w.dtype,
                             w.n_q_heads, max(n, w.budget) + 4, w.gamma, w.budget, lib=lib)
            ins = [synth.decode_inputs(w, t) for t in range(8)]

            def step(t, run=run, ins=ins, k=len(ls)):
                q, kn, vn = ins[t % len(ins)]
                run.step(q[:k], kn[:k], vn[:k])
            med, steps = timed(step, w.steps)
            per_token = med * w.n_layers / len(ls)
            rep["workloads"].append({"workload": name, "threads": min(threads, len(ls)), "layers_sampled": len(ls),
                                     "steps_timed": steps, "ms_per_token": per_token * 1e3,
                                     "tokens_per_s": 1.0 / per_token})
            log(f"[cpu] {name}, {threads} thread(s): {per_token * 1e3:.1f} ms per token")
    ws_list = synth.batch_workloads()
    runs = []
    oracle.set_threads(1, lib)
    for i, w in enumerate(ws_list):
        off = synth.offsets_from_lengths(synth.span_lengths(w, seq=i))
        n = len(off) - 1
        runs.append(oracle.Run(synth.prefill_kv(w, "k", seq=i, layers=range(1)),
                               synth.prefill_kv(w, "v", seq=i, layers=range(1)), off, w.dtype, w.n_q_heads,
                               max(n, w.budget) + w.interval + 1, w.gamma, w.budget, interval=w.interval, lib=lib))
    w0 = ws_list[0]
    b_ins = [[tuple(x[:1] for x in synth.decode_inputs(w, t, seq=i)) for t in range(4)] for i, w in enumerate(ws_list)]
    for threads in (1, min(n_all, len(runs))):
        pool = cf.ThreadPoolExecutor(threads)

        def one(i, t):
            runs[i].step(*b_ins[i][t % 4])

        def step(t):
            list(pool.map(lambda i: one(i, t), range(len(runs))))
        med, steps = timed(step, w0.steps)
        pool.shutdown()
        per_step = med * w0.n_layers  # all 16 sequences, 48 layers: 16 tokens
        rep["workloads"].append({"workload": "batch16", "threads": threads, "layers_sampled": 1, "steps_timed": steps,
                                 "ms_per_token": per_step / len(runs) * 1e3, "tokens_per_s": len(runs) / per_step})
        log(f"[cpu] batch16, {threads} thread(s): {per_step / len(runs) * 1e3:.1f} ms per token")
    oracle.set_threads(n_all, lib)
    return rep


def cpu_baseline(w, n_layers_sample: int, max_seconds: float):
    """The oracle (as it stands) on a sample: the first n layers, fused on the
    host, then decode steps with eviction until max_seconds of step time."""
    import oracle
    t0 = time.time()
    lib = oracle.load()
    ls = range(n_layers_sample)
    off = synth.offsets_from_lengths(synth.span_lengths(w))
    n = len(off) - 1
    k_in = synth.prefill_kv(w, "k", layers=ls)
    v_in = synth.prefill_kv(w, "v", layers=ls)
    cap = max(n, w.budget) + 4
    run = oracle.Run(k_in, v_in, off, w.dtype, w.n_q_heads, cap, w.gamma, w.budget, lib=lib)
    log(f"[cpu] oracle setup {time.time() - t0:.1f}s")
    step_times = []
    t_all = time.time()
    for t in range(256):
        q, kn, vn = synth.decode_inputs(w, t)
        ts = time.perf_counter()
        run.step(q[:n_layers_sample], kn[:n_layers_sample], vn[:n_layers_sample])
        step_times.append(time.perf_counter() - ts)
        if time.time() - t_all > max_seconds:
            break
    per_step_all_layers = float(np.mean(step_times)) * (w.n_layers / n_layers_sample)
    return {
        "value": 1.0 / per_step_all_layers,
        "unit": "tokens/s",
        "cores": int(min(oracle.threads(lib), n_layers_sample)),
        "kind": "oracle",
        "sample": (f"{len(step_times)} decode steps (append, attend, score, evict) of the 32k workload on "
                   f"{n_layers_sample} of {w.n_layers} layers, after host-side fusion; time per step "
                   f"scaled by {w.n_layers}/{n_layers_sample} to a whole-model token; host CPU {cpu_model()}"),
    }


def kept_sets_report(args, torch, vz) -> dict:
    """Free-running agreement of the kept sets (Sec. 3.2.2 Eq. 9): the 32k
    request (fusion, then 256 generation steps with eviction) on the GPU over
    all layers, and the oracle's own run (fp64 scores) over a sample of the
    layers from the same inputs, neither side ever resynchronised.  After
    every step, per sampled layer, the Jaccard index of the two resident
    position sets.  GPU and oracle scores differ by rounding (bfloat16
    probabilities on the GPU), so a near-tie at the eviction threshold can
    keep a different slot; the two runs then go on from different caches."""
    import oracle
    w = synth.workload("long32k")
    L, Hq, Hkv, d = w.n_layers, w.n_q_heads, w.kv_heads, w.d
    layers = [int(x) for x in args.kept_layers.split(",")]
    off = synth.offsets_from_lengths(synth.span_lengths(w))
    n = len(off) - 1
    t0 = time.time()
    k_in = synth.prefill_kv(w, "k")
    v_in = synth.prefill_kv(w, "v")
    to_dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    cap = max(n, w.budget) + 2
    K = torch.zeros(L, Hkv, cap, d, dtype=torch.bfloat16, device="cuda")
    V = torch.zeros_like(K)
    S = torch.zeros(L, cap, dtype=torch.float32, device="cuda")
    P = torch.zeros(L, cap, dtype=torch.int32, device="cuda")
    out = torch.zeros(L, Hq, d, dtype=torch.bfloat16, device="cuda")
    ws = vz.workspace(vz.VZ_OP_DECODE_EVICT, L, Hq, Hkv, d, cap)
    vz.voxzip_fuse_spans(to_dev(k_in), to_dev(v_in), torch.from_numpy(off).cuda(), K, V, S, P)
    idx = torch.tensor(layers, dtype=torch.long, device="cuda")
    run = oracle.Run(k_in[layers], v_in[layers], off, w.dtype, Hq, cap, w.gamma, w.budget)
    del k_in, v_in
    log(f"[kept] inputs and fusion {time.time() - t0:.1f}s; oracle on layers {layers}")
    length, nxt = n, n
    jac = np.zeros((args.decode_steps, len(layers)))
    for t in range(args.decode_steps):
        q, kn, vn = synth.decode_inputs(w, t)
        length = vz.voxzip_decode_evict(to_dev(q), to_dev(kn), to_dev(vn), K, V, S, P, out, length, nxt, w.gamma,
                                        w.budget, workspace=ws)
        nxt += 1
        run.step(q[layers], kn[layers], vn[layers])
        assert run.len == length
        gpu_pos = P.index_select(0, idx)[:, :length].cpu().numpy()
        for j in range(len(layers)):
            a, b = set(gpu_pos[j].tolist()), set(run.pos[j, :length].tolist())
            jac[t, j] = len(a & b) / len(a | b)
        if t % 32 == 31:
            log(f"[kept] step {t + 1}: mean Jaccard {jac[t].mean():.5f}")
    diverged = [int(np.argmax(jac[:, j] < 1.0)) if np.any(jac[:, j] < 1.0) else None for j in range(len(layers))]
    return {"kept_set_agreement": {
        "workload": "long32k", "layers": layers, "steps": args.decode_steps, "budget": w.budget,
        "jaccard_final": [float(x) for x in jac[-1]],
        "jaccard_min": float(jac.min()),
        "jaccard_mean": float(jac.mean()),
        "first_step_with_a_difference": diverged,
        "steps_identical_frac": float(np.mean(jac == 1.0)),
        "curve_every_16_steps": [float(x) for x in jac.mean(axis=1)[15::16]],
    }}


class Sequence:
    """One sequence of a workload on its own stream: span structure from the
    seeded generator, K/V and per-step q/k/v drawn on the GPU from a seeded
    torch generator (N(0,1), plus the workload's query bias), cache and
    workspaces sized as in the parity tests."""

    def __init__(self, torch, vz, w, seq, steps, stream):
        self.vz, self.w, self.stream = vz, w, stream
        L, Hq, Hkv, d = w.n_layers, w.n_q_heads, w.kv_heads, w.d
        gen = torch.Generator(device="cuda")
        gen.manual_seed(synth.stream_key(w.seed, w.name, "bench", seq) & 0x7FFFFFFFFFFFFFFF)
        off = synth.offsets_from_lengths(synth.span_lengths(w, seq=seq))
        self.n = len(off) - 1
        T_in = w.n_audio + w.n_text
        bf = torch.bfloat16
        rn = lambda *shape: torch.randn(*shape, generator=gen, device="cuda", dtype=torch.float32).to(bf)
        self.k_in, self.v_in = rn(L, Hkv, T_in, d), rn(L, Hkv, T_in, d)
        self.off = torch.from_numpy(off).cuda()
        bias = torch.from_numpy(synth.q_bias(w)).to("cuda", torch.float32) if w.q_bias else None
        self.steps_in = []
        for _ in range(steps):
            q = torch.randn(L, Hq, d, generator=gen, device="cuda")
            q = (q + bias if bias is not None else q).to(bf)
            self.steps_in.append((q, rn(L, Hkv, d), rn(L, Hkv, d)))
        self.cap = max(self.n, w.budget) + w.interval + 1
        self.K = torch.zeros(L, Hkv, self.cap, d, dtype=bf, device="cuda")
        self.V = torch.zeros_like(self.K)
        self.S = torch.zeros(L, self.cap, dtype=torch.float32, device="cuda")
        self.P = torch.zeros(L, self.cap, dtype=torch.int32, device="cuda")
        self.out = torch.zeros(L, Hq, d, dtype=bf, device="cuda")
        self.ws_d = vz.workspace(vz.VZ_OP_DECODE, L, Hq, Hkv, d, self.cap)
        self.ws_s = vz.workspace(vz.VZ_OP_DECODE_EVICT, L, Hq, Hkv, d, self.cap)

    def start(self):
        self.vz.voxzip_fuse_spans(self.k_in, self.v_in, self.off, self.K, self.V, self.S, self.P,
                                  stream=self.stream)
        self.len = self.nxt = self.n
        return 0

    def step(self, t):
        """Decode step t (and the eviction when it is due); returns algorithmic bytes."""
        w, vz = self.w, self.vz
        L, Hq, Hkv, d = w.n_layers, w.n_q_heads, w.kv_heads, w.d
        q, kn, vn = self.steps_in[t]
        T = self.len + 1
        b = L * decode_bytes_per_layer(T, Hq, Hkv, d, 2)
        if (t + 1) % w.interval == 0 and T > w.budget:  # a step with its eviction: one call
            new_len = vz.voxzip_decode_evict(q, kn, vn, self.K, self.V, self.S, self.P, self.out, self.len,
                                             self.nxt, w.gamma, w.budget, workspace=self.ws_s, stream=self.stream)
            b += L * evict_bytes_per_layer(T, T - w.budget, Hkv, d, 2)
        else:
            vz.voxzip_decode_attend_score(q, kn, vn, self.K, self.V, self.S, self.P, self.out, self.len, self.nxt,
                                          w.gamma, workspace=self.ws_d, stream=self.stream)
            new_len = T
        self.len, self.nxt = new_len, self.nxt + 1
        return b


class RaggedBatch:
    """All sequences of the batched workload in one packed cache, driven
    through the ragged entry points: one fusion call per request, one decode
    call per step for every sequence, one eviction call every `interval`
    steps.  Inputs are drawn exactly as for Sequence (same seeds), then packed;
    lengths live on the device (the host mirrors them only to count bytes)."""

    def __init__(self, torch, vz, ws_, steps):
        self.torch, self.vz, self.ws_ = torch, vz, ws_
        w = ws_[0]
        L, Hq, Hkv, d = w.n_layers, w.n_q_heads, w.kv_heads, w.d
        bf = torch.bfloat16
        n = len(ws_)
        offs = [synth.offsets_from_lengths(synth.span_lengths(x, seq=i)) for i, x in enumerate(ws_)]
        self.n_spans = np.array([len(o) - 1 for o in offs], dtype=np.int64)
        self.budget = np.array([x.budget for x in ws_], dtype=np.int64)
        T_in = np.array([x.n_audio + x.n_text for x in ws_], dtype=np.int64)
        caps = np.maximum(self.n_spans, self.budget) + w.interval + 1
        in_base = np.concatenate([[0], np.cumsum(T_in)[:-1]]).astype(np.int64)
        base = np.concatenate([[0], np.cumsum(caps)[:-1]]).astype(np.int64)
        off_base = np.concatenate([[0], np.cumsum(self.n_spans + 1)[:-1]]).astype(np.int64)
        self.total = int(caps.sum())
        self.k_in = torch.empty(L, Hkv, int(T_in.sum()), d, dtype=bf, device="cuda")
        self.v_in = torch.empty_like(self.k_in)
        self.q = [torch.empty(n, L, Hq, d, dtype=bf, device="cuda") for _ in range(steps)]
        self.kn = [torch.empty(n, L, Hkv, d, dtype=bf, device="cuda") for _ in range(steps)]
        self.vn = [torch.empty(n, L, Hkv, d, dtype=bf, device="cuda") for _ in range(steps)]
        for i, x in enumerate(ws_):
            gen = torch.Generator(device="cuda")
            gen.manual_seed(synth.stream_key(x.seed, x.name, "bench", i) & 0x7FFFFFFFFFFFFFFF)
            rn = lambda *shape: torch.randn(*shape, generator=gen, device="cuda", dtype=torch.float32).to(bf)
            sl = slice(int(in_base[i]), int(in_base[i] + T_in[i]))
            self.k_in[:, :, sl] = rn(L, Hkv, int(T_in[i]), d)
            self.v_in[:, :, sl] = rn(L, Hkv, int(T_in[i]), d)
            for t in range(steps):
                self.q[t][i] = torch.randn(L, Hq, d, generator=gen, device="cuda").to(bf)
                self.kn[t][i] = rn(L, Hkv, d)
                self.vn[t][i] = rn(L, Hkv, d)
        dev = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a).astype(dt)).cuda()
        self.off = dev(np.concatenate(offs), np.int32)
        self.in_base, self.T_in, self.off_base = dev(in_base, np.int64), dev(T_in, np.int32), dev(off_base, np.int64)
        self.n_spans_d, self.base, self.cap = dev(self.n_spans, np.int32), dev(base, np.int64), dev(caps, np.int32)
        self.budget_d = dev(self.budget, np.int32)
        self.K = torch.zeros(L, Hkv, self.total, d, dtype=bf, device="cuda")
        self.V = torch.zeros_like(self.K)
        self.S = torch.zeros(L, self.total, dtype=torch.float32, device="cuda")
        self.P = torch.zeros(L, self.total, dtype=torch.int32, device="cuda")
        self.out = torch.zeros(n, L, Hq, d, dtype=bf, device="cuda")
        self.len_d = torch.zeros(n, dtype=torch.int32, device="cuda")
        self.nxt_d = torch.zeros_like(self.len_d)
        self.new_len = torch.zeros_like(self.len_d)
        self.ws_d = vz.workspace_ragged(vz.VZ_OP_DECODE, L, Hq, Hkv, d, self.total, n)
        self.ws_e = vz.workspace_ragged(vz.VZ_OP_EVICT, L, Hq, Hkv, d, self.total, n)

    def start(self):
        vz = self.vz
        vz.voxzip_fuse_spans_ragged(self.k_in, self.v_in, self.in_base, self.T_in, self.off, self.off_base,
                                    self.n_spans_d, int(self.n_spans.max()), self.K, self.V, self.S, self.P,
                                    self.base, self.cap)
        self.len_d.copy_(self.n_spans_d)
        self.nxt_d.copy_(self.n_spans_d)
        self.len = self.n_spans.copy()

    def step(self, t):
        """Decode step t of every sequence (and the eviction when it is due);
        returns the algorithmic bytes."""
        w, vz = self.ws_[0], self.vz
        L, Hq, Hkv, d = w.n_layers, w.n_q_heads, w.kv_heads, w.d
        vz.voxzip_decode_attend_score_ragged(self.q[t], self.kn[t], self.vn[t], self.K, self.V, self.S, self.P,
                                             self.out, self.base, self.cap, self.len_d, self.nxt_d, w.gamma,
                                             workspace=self.ws_d)
        T = self.len + 1
        b = sum(L * decode_bytes_per_layer(int(x), Hq, Hkv, d, 2) for x in T)
        self.len = T
        self.len_d += 1
        self.nxt_d += 1
        if (t + 1) % w.interval == 0:
            vz.voxzip_evict_compact_ragged(self.K, self.V, self.S, self.P, self.base, self.cap, self.len_d,
                                           self.budget_d, self.nxt_d, new_len_out=self.new_len,
                                           workspace=self.ws_e)
            self.len_d.copy_(self.new_len)
            E = np.maximum(self.len - self.budget, 0)
            b += sum(L * evict_bytes_per_layer(int(x), int(e), Hkv, d, 2) for x, e in zip(T, E) if e > 0)
            self.len = np.minimum(self.len, self.budget)
        return b


def other_workload(args, torch, vz):
    """aggr64k (one sequence, 512 steps) or batch16 (16 sequences of 2k-32k
    tokens, 128 steps each, eviction every 16 steps; through the ragged entry
    points, or with --batch-streams one call sequence per sequence on 16
    streams): whole requests (fusion + all steps), tokens/s over the wall
    clock and the algorithmic bytes of the path per second."""
    if args.workload == "aggr64k":
        ws_ = [synth.workload("aggr64k")]
    else:
        ws_ = synth.batch_workloads()
    steps = ws_[0].steps
    t0 = time.time()
    ragged = args.workload == "batch16" and not args.batch_streams
    if ragged:
        batch = RaggedBatch(torch, vz, ws_, steps)
        n_seqs, n_spans = len(ws_), int(batch.n_spans.sum())
    else:
        seqs = [Sequence(torch, vz, w, i, steps, torch.cuda.Stream()) for i, w in enumerate(ws_)]
        n_seqs, n_spans = len(seqs), sum(s.n for s in seqs)
    torch.cuda.synchronize()
    log(f"[gpu] {args.workload}: {n_seqs} sequence(s), {n_spans} spans, inputs ready in {time.time() - t0:.1f}s")

    def request():
        if ragged:
            batch.start()
            b = sum(batch.step(t) for t in range(steps))
            return n_seqs * steps, b
        b = 0
        for s in seqs:
            s.start()
        for t in range(steps):
            for s in seqs:
                b += s.step(t)
        return n_seqs * steps, b

    for _ in range(args.warmup):
        request()
    torch.cuda.synchronize()
    tokens = path_bytes = 0
    t_start = time.perf_counter()
    for _ in range(args.steps):
        tk, b = request()
        tokens += tk
        path_bytes += b
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    w = ws_[0]
    if args.workload == "aggr64k":
        desc = (f"48 layers, 32Q/4KV, d=128, bf16; 65536 audio tokens (spans of mean length 5, 10 percent of "
                f"length 1) fused to {seqs[0].n} spans, B=3277, queries biased to about 5 percent of the keys, "
                f"512 decode steps with eviction")
    else:
        lens = "/".join(str(x.n_audio) for x in ws_)
        how = ("one packed cache, one ragged decode call per step for all sequences" if ragged
               else "one HIP stream and one call sequence per sequence")
        desc = (f"16 sequences of {lens} audio tokens (spans of mean length 4), budget len/4 each, eviction "
                f"every 16 steps, 128 decode steps each; {how}")
    print(json.dumps({
        "metric": "decode attend+score+evict tokens/s and HBM GB/s (% of peak)",
        "value": tokens / elapsed, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": elapsed * 1e3 / args.steps, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": args.workload, "description": desc, "layers": w.n_layers,
                   "sequences": n_seqs, "decode_steps_per_request": steps},
        "path_gbps": path_bytes / elapsed / 1e9,
        "path_frac_of_hbm_peak": path_bytes / elapsed / 1e9 / HBM_PEAK_GBS,
    }), flush=True)


def serve_workload(args, torch, vz):
    """Continuous batching (paper_2608_08569_amd.loop): a stream of requests
    served through 16 batch slots of one packed cache.  Each request has the
    batched workload's shape (48 layers, 32Q/4KV, d = 128, bf16, audio of
    2k-32k tokens with spans of mean length 4, budget len / 4, eviction every
    16 of its own steps) and generates 64-256 tokens; when it has generated
    them it leaves, and the next waiting request is admitted into the freed
    slot (its prefill fused there, Sec. 3.2.1).  Every step is one graph
    replay (decode of all active slots + eviction when some slot is due).
    All prefill caches and per-step inputs are drawn on the GPU and resident
    before the timed region; the value is generated tokens per second over
    the whole stream, admissions included."""
    from paper_2608_08569_amd.loop import DecodeLoop
    L, Hq, Hkv, d, interval, gamma = 48, 32, 4, 128, 16, 0.95
    n_slots, n_req = 16, args.serve_requests
    key = synth.stream_key(0, "serve16")
    T_audio = synth.uniform_int(synth.stream_key(key, "lengths"), 0, n_req, 2048, 32768).astype(np.int64)
    gen_len = synth.uniform_int(synth.stream_key(key, "generate"), 0, n_req, 64, 256).astype(np.int64)
    offs = [synth.offsets_from_lengths(synth.spans_geometric(synth.stream_key(key, "spans", i), int(T), 0.25, 32))
            for i, T in enumerate(T_audio)]
    n_spans = np.array([len(o) - 1 for o in offs], dtype=np.int64)
    budgets = T_audio // 4
    cap = int(np.max(np.maximum(n_spans, budgets))) + interval + 1
    t0 = time.time()
    bf = torch.bfloat16
    gen = torch.Generator(device="cuda")
    gen.manual_seed(key & 0x7FFFFFFFFFFFFFFF)
    rn = lambda *shape: torch.randn(*shape, generator=gen, device="cuda", dtype=torch.float32).to(bf)
    pre = [(rn(L, Hkv, int(T), d), rn(L, Hkv, int(T), d)) for T in T_audio]
    offs_d = [torch.from_numpy(o).cuda() for o in offs]
    G = int(gen_len.max())
    Q = rn(n_req * G, L, Hq, d)
    KN = rn(n_req * G, L, Hkv, d)
    VN = rn(n_req * G, L, Hkv, d)
    lp = DecodeLoop(L, Hq, Hkv, d, [cap] * n_slots, [1] * n_slots, gamma, interval=interval)
    qb = torch.zeros(n_slots, L, Hq, d, dtype=bf, device="cuda")
    kb = torch.zeros(n_slots, L, Hkv, d, dtype=bf, device="cuda")
    vb = torch.zeros_like(kb)
    # input row of each slot's step: its request's first row plus the slot's
    # device-side step count (no host-to-device copy per step)
    idx = torch.zeros(n_slots, dtype=torch.int64, device="cuda")
    slot_row0 = torch.zeros(n_slots, dtype=torch.int64, device="cuda")
    for s in range(n_slots):
        lp.retire(s)
    lp.capture(qb, kb, vb)
    torch.cuda.synchronize()
    log(f"[gpu] serve16: {n_req} requests ({int(T_audio.sum())} audio tokens, {int(gen_len.sum())} to generate), "
        f"slot capacity {cap}, inputs ready in {time.time() - t0:.1f}s")

    def run():
        """The whole stream; returns (generated tokens, algorithmic bytes, steps)."""
        waiting = list(range(n_req))
        holder = {}  # slot -> [request, tokens generated, resident length (host mirror)]
        tokens = path_bytes = steps = 0
        while waiting or holder:
            for s in list(holder):
                i, g, _ = holder[s]
                if g == gen_len[i]:
                    lp.retire(s)
                    del holder[s]
            for s in range(n_slots):
                if s not in holder and waiting:
                    i = waiting.pop(0)
                    lp.admit(s, pre[i][0], pre[i][1], offs_d[i], budget=int(budgets[i]))
                    slot_row0[s] = i * G
                    holder[s] = [i, 0, int(n_spans[i])]
            if not holder:
                break
            torch.add(slot_row0, lp.age, out=idx)
            idx.clamp_(0, n_req * G - 1)  # idle slots count on; their rows are never used
            torch.index_select(Q, 0, idx, out=qb)
            torch.index_select(KN, 0, idx, out=kb)
            torch.index_select(VN, 0, idx, out=vb)
            lp.replay()
            steps += 1
            for s, h in holder.items():
                i, g, ln = h
                T = ln + 1
                path_bytes += L * decode_bytes_per_layer(T, Hq, Hkv, d, 2)
                if (g + 1) % interval == 0 and T > budgets[i]:
                    path_bytes += L * evict_bytes_per_layer(T, T - int(budgets[i]), Hkv, d, 2)
                    T = int(budgets[i])
                h[1], h[2] = g + 1, T
                tokens += 1
        return tokens, path_bytes, steps

    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    tokens = path_bytes = steps = 0
    for _ in range(args.steps):
        tk, b, st = run()
        tokens += tk
        path_bytes += b
        steps += st
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    print(json.dumps({
        "metric": "decode attend+score+evict tokens/s and HBM GB/s (% of peak)",
        "value": tokens / elapsed, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": elapsed * 1e3 / args.steps, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "serve16",
                   "description": (f"continuous batching: {n_req} requests of 2k-32k audio tokens (spans of mean "
                                   f"length 4, budget len/4, eviction every 16 of their own steps) generating "
                                   f"64-256 tokens each, through 16 batch slots of one packed cache; a request "
                                   f"leaves when done and the next is admitted (prefill fused into the freed "
                                   f"slot); one graph replay per step; one step = the whole stream"),
                   "layers": L, "slots": n_slots, "requests": n_req, "generated_tokens": tokens // args.steps,
                   "decode_steps": steps // args.steps},
        "path_gbps": path_bytes / elapsed / 1e9,
        "path_frac_of_hbm_peak": path_bytes / elapsed / 1e9 / HBM_PEAK_GBS,
    }), flush=True)


def loop_workload(args, torch, vz):
    """long32k through the decode loop (paper_2608_08569_amd.loop): one
    decode call per layer, layer l's query being its own input query plus
    layer l - 1's output (the dependency of a forward pass), eviction after
    every step; launched eagerly (long32k-layers) or replayed per token from a
    HIP graph (long32k-graph).  Same fused cache and inputs as the headline."""
    from paper_2608_08569_amd.loop import DecodeLoop
    w = synth.workload("long32k")
    L, Hq, Hkv, d = w.n_layers, w.n_q_heads, w.kv_heads, w.d
    t0 = time.time()
    off = synth.offsets_from_lengths(synth.span_lengths(w))
    n_spans = len(off) - 1
    T_in = w.n_audio + w.n_text
    bf = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    k_in, v_in = bf(synth.prefill_kv(w, "k")), bf(synth.prefill_kv(w, "v"))
    steps = args.decode_steps
    inputs = []
    for t in range(steps):
        q, kn, vn = synth.decode_inputs(w, t)
        inputs.append((bf(q).view(L, 1, 1, Hq, d), bf(kn).view(L, 1, 1, Hkv, d), bf(vn).view(L, 1, 1, Hkv, d)))
    log(f"[gpu] {args.workload}: inputs ready in {time.time() - t0:.1f}s: {n_spans} spans")
    cap = max(n_spans, w.budget) + 2
    lp = DecodeLoop(L, Hq, Hkv, d, [cap], [w.budget], w.gamma, interval=1)
    i64 = lambda v: torch.tensor(v, dtype=torch.int64, device="cuda")
    i32 = lambda v: torch.tensor(v, dtype=torch.int32, device="cuda")
    off_d = torch.from_numpy(off).cuda()
    qmix = torch.zeros(L, 1, 1, Hq, d, dtype=torch.bfloat16, device="cuda")

    def layer_query(l, q, outs):
        return q[0] if l == 0 else torch.add(q[l], outs[l - 1], out=qmix[l])

    graph = args.workload == "long32k-graph"
    qb, kb, vb = (torch.zeros_like(x) for x in inputs[0])

    def start():
        lp.fuse(k_in, v_in, i64([0]), i32([T_in]), off_d, i64([0]), i32([n_spans]), n_spans)

    start()
    if graph:
        lp.capture(qb, kb, vb, layer_query)

    def request():
        start()
        b = 0
        length = n_spans
        for t in range(steps):
            q, kn, vn = inputs[t]
            if graph:
                qb.copy_(q)
                kb.copy_(kn)
                vb.copy_(vn)
                lp.replay()
            else:
                lp.step(q, kn, vn, layer_query)
            T = length + 1
            b += L * decode_bytes_per_layer(T, Hq, Hkv, d, 2)
            if T > w.budget:
                b += L * evict_bytes_per_layer(T, T - w.budget, Hkv, d, 2)
            length = min(T, w.budget)
        return steps, b

    for _ in range(args.warmup):
        request()
    torch.cuda.synchronize()
    tokens = path_bytes = 0
    t_start = time.perf_counter()
    for _ in range(args.steps):
        tk, b = request()
        tokens += tk
        path_bytes += b
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    how = "replayed per token from a HIP graph" if graph else "launched eagerly"
    print(json.dumps({
        "metric": "decode attend+score+evict tokens/s and HBM GB/s (% of peak)",
        "value": tokens / elapsed, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": elapsed * 1e3 / args.steps, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": args.workload,
                   "description": (f"the 32k workload ({n_spans} spans, B=8192, 48 layers, 32Q/4KV, d=128) with "
                                   f"one decode call per layer, each layer's query depending on the previous "
                                   f"layer's output, eviction every step, {how}; one step = fusion + "
                                   f"{steps} decode steps"),
                   "layers": L, "sequences": 1, "decode_steps_per_request": steps},
        "us_per_token": elapsed * 1e6 / tokens,
        "path_gbps": path_bytes / elapsed / 1e9,
        "path_frac_of_hbm_peak": path_bytes / elapsed / 1e9 / HBM_PEAK_GBS,
    }), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5, help="timed requests")
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--decode-steps", type=int, default=256)
    ap.add_argument("--roofline-calls", type=int, default=64,
                    help="decode calls at the steady length timed for the roofline")
    ap.add_argument("--cpu-layers", type=int, default=16)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--cpu-report", action="store_true",
                    help="only time the CPU oracle per workload (single- and multi-threaded); no GPU work")
    ap.add_argument("--kept-sets", action="store_true",
                    help="only compare the GPU's free-running kept sets with the oracle's (long32k, sampled layers)")
    ap.add_argument("--kept-layers", default="0,16,32,47", help="layers the oracle runs for --kept-sets")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a 1 GiB device copy (counter calibration for rocprofv3 --pmc)")
    ap.add_argument("--workload", default="long32k",
                    choices=["long32k", "aggr64k", "batch16", "long32k-layers", "long32k-graph", "serve16"],
                    help="long32k is the headline; the others are reported beside it")
    ap.add_argument("--serve-requests", type=int, default=48, help="requests in the serve16 stream")
    ap.add_argument("--batch-streams", action="store_true",
                    help="batch16 with one stream and one call sequence per sequence instead of the ragged calls")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path "
              "(the sharding design is described in the design notes)", file=sys.stderr)
        sys.exit(2)

    if args.cpu_report:
        print(json.dumps(cpu_report()), flush=True)
        return

    import torch
    import paper_2608_08569_amd as vz

    vz.lib()  # fail loudly if the HIP library is not built
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()

    if args.kept_sets:
        print(json.dumps(kept_sets_report(args, torch, vz)), flush=True)
        return

    if args.copy_probe:
        n = 1 << 30
        a = torch.empty(n, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n}))
        return

    if args.workload in ("long32k-layers", "long32k-graph"):
        loop_workload(args, torch, vz)
        return
    if args.workload == "serve16":
        serve_workload(args, torch, vz)
        return
    if args.workload != "long32k":
        other_workload(args, torch, vz)
        return

    w = synth.workload("long32k")
    L, Hq, Hkv, d = w.n_layers, w.n_q_heads, w.kv_heads, w.d
    s = 2
    t0 = time.time()
    off = synth.offsets_from_lengths(synth.span_lengths(w))
    n_spans = len(off) - 1
    to_dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    k_in = to_dev(synth.prefill_kv(w, "k"))
    v_in = to_dev(synth.prefill_kv(w, "v"))
    off_d = torch.from_numpy(off).cuda()
    steps_in = []
    for t in range(args.decode_steps):
        q, kn, vn = synth.decode_inputs(w, t)
        steps_in.append((to_dev(q), to_dev(kn), to_dev(vn)))
    log(f"[gpu] inputs ready in {time.time() - t0:.1f}s: {n_spans} spans")

    cap = max(n_spans, w.budget) + 2
    K = torch.zeros(L, Hkv, cap, d, dtype=torch.bfloat16, device="cuda")
    V = torch.zeros_like(K)
    S = torch.zeros(L, cap, dtype=torch.float32, device="cuda")
    P = torch.zeros(L, cap, dtype=torch.int32, device="cuda")
    out = torch.zeros(L, Hq, d, dtype=torch.bfloat16, device="cuda")
    ws_step = vz.workspace(vz.VZ_OP_DECODE_EVICT, L, Hq, Hkv, d, cap)
    ws_d = vz.workspace(vz.VZ_OP_DECODE, L, Hq, Hkv, d, cap)

    def request(timing=None):
        """Fuse, then one generation step per token (decode + eviction in one
        call); returns (decode tokens, bytes)."""
        ev = timing
        if ev is not None:
            ev["fuse"][0].record(stream)
        vz.voxzip_fuse_spans(k_in, v_in, off_d, K, V, S, P)
        if ev is not None:
            ev["fuse"][1].record(stream)
        length, nxt = n_spans, n_spans
        total_bytes = 0
        for t in range(args.decode_steps):
            q, kn, vn = steps_in[t]
            new_len = vz.voxzip_decode_evict(q, kn, vn, K, V, S, P, out, length, nxt, w.gamma, w.budget,
                                             workspace=ws_step)
            T = length + 1
            total_bytes += L * decode_bytes_per_layer(T, Hq, Hkv, d, s)
            if T > w.budget:
                total_bytes += L * evict_bytes_per_layer(T, T - w.budget, Hkv, d, s)
            length, nxt = new_len, nxt + 1
        return args.decode_steps, total_bytes, length, nxt

    for _ in range(args.warmup):
        request()
    torch.cuda.synchronize()

    mk = lambda: torch.cuda.Event(enable_timing=True)
    timings = []
    tokens = 0
    path_bytes = 0
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        ev = {"fuse": (mk(), mk())}  # no per-step events in the timed requests: each costs a pipeline drain
        tk, b, length, nxt = request(ev)
        tokens += tk
        path_bytes += b
        timings.append(ev)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start

    fuse_ms = np.array([ev["fuse"][0].elapsed_time(ev["fuse"][1]) for ev in timings])
    # Dominant kernel: the generation step at the steady length T = B + 1
    # (one launch of the whole-range kernel whose last workgroup per layer
    # folds the scores and evicts one row), continuing the request's sequence.
    # One HIP event pair on the library's stream brackets n back-to-back
    # launches (an event between two launches drains the pipeline and adds
    # ~3 us to each); the mean launch time is their interval / n.
    T_ss = w.budget + 1
    assert length == w.budget
    dec_bytes_ss = L * decode_bytes_per_layer(T_ss, Hq, Hkv, d, s)
    step_bytes_ss = dec_bytes_ss + L * evict_bytes_per_layer(T_ss, 1, Hkv, d, s)
    n_rf = args.roofline_calls

    def bracket(launch):
        for i in range(4):  # untimed
            launch(i)
        a, b = mk(), mk()
        a.record(stream)
        for i in range(n_rf):
            launch(i)
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e-3 / n_rf

    st = {"length": length, "nxt": nxt}

    def gen_step(i):
        q, kn, vn = steps_in[i % len(steps_in)]
        st["length"] = vz.voxzip_decode_evict(q, kn, vn, K, V, S, P, out, st["length"], st["nxt"], w.gamma,
                                             w.budget, workspace=ws_step)
        st["nxt"] += 1

    step_mean_s = bracket(gen_step)
    assert st["length"] == w.budget
    # the decode entry point alone (no eviction) at the same length, for
    # comparison: repeated on the final state (each call rewrites slot B),
    # the new position advancing as in the steps (the kernel's read order
    # alternates with its parity)
    q, kn, vn = steps_in[-1]
    dec_mean_s = bracket(lambda i: vz.voxzip_decode_attend_score(q, kn, vn, K, V, S, P, out, st["length"],
                                                                  st["nxt"] + i, w.gamma, workspace=ws_d))
    achieved = step_bytes_ss / step_mean_s / 1e9
    dec_achieved = dec_bytes_ss / dec_mean_s / 1e9
    traffic = read_traffic()
    fuse_bytes = L * Hkv * 2 * (32768 + n_spans) * d * s
    copy_rate = copy_gbps(torch, stream)

    result = {
        "metric": "decode attend+score+evict tokens/s and HBM GB/s (% of peak) at 32k ctx",
        "value": tokens / elapsed,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "long32k",
            "description": (f"48 layers, 32Q/4KV heads, d=128, bf16 KV cache; 32768 audio tokens fused to "
                            f"{n_spans} span tokens (Stage 1), B=8192 (M=1638, N=6550, T=4), gamma=0.95; "
                            f"one step = fusion + {args.decode_steps} generation steps (decode + eviction, "
                            f"one voxzip_decode_evict call each)"),
            "layers": L, "q_heads": Hq, "kv_heads": Hkv, "head_dim": d, "audio_tokens": 32768,
            "fused_tokens": n_spans, "budget": w.budget, "decode_steps_per_request": args.decode_steps,
        },
        "path_gbps": path_bytes / elapsed / 1e9,
        "path_frac_of_hbm_peak": path_bytes / elapsed / 1e9 / HBM_PEAK_GBS,
        "step_us_steady": step_mean_s * 1e6,
        "step_gbps_steady": achieved,
        "decode_us_mean": dec_mean_s * 1e6,
        "fuse_ms_mean": float(np.mean(fuse_ms)),
        "fuse_gbps": fuse_bytes / (float(np.mean(fuse_ms)) * 1e-3) / 1e9,
        "roofline": {
            "kernel": ("voxzip_decode_evict = decode_range_kernel<4, false, false>, one launch per generation "
                       "step: attend + score + evict (whole-range decode, one workgroup per layer and KV head; "
                       "the last workgroup of each layer folds Eq. 6 and evicts; 48 layers, T=8193, E=1)"),
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic,
            "algorithmic_bytes_per_launch": step_bytes_ss,
            "mean_launch_us": step_mean_s * 1e6,
            "launches_timed": n_rf,
            "timing": "one HIP event pair around the launches_timed back-to-back launches",
            "read_order": ("each wave reads its chunks in alternating directions on consecutive steps (parity "
                           "of the new position), so a step starts on the keys the previous one read last, "
                           "part of them still in the 256 MB memory-side Infinity Cache; achieved counts every "
                           "algorithmic byte, and traffic (L2-to-fabric requests) includes those the Infinity "
                           "Cache serves"),
            "copy_gbps": copy_rate,
            "frac_of_copy": achieved / copy_rate,
            "decode_only": {
                "entry_point": "voxzip_decode_attend_score (attend + score, no eviction; same kernel)",
                "algorithmic_bytes_per_launch": dec_bytes_ss,
                "mean_launch_us": dec_mean_s * 1e6,
                "achieved": dec_achieved,
                "frac": dec_achieved / HBM_PEAK_GBS,
            },
        },
    }
    kept = read_kept_agreement()
    if kept is not None:
        result["kept_set_agreement"] = kept
    if not args.no_cpu:
        result["cpu_baseline"] = cpu_baseline(w, args.cpu_layers, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
