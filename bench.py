#!/usr/bin/env python3
"""Throughput of the InfLLM block-memory attention step on one MI355X.

A benchmark step is one pass of the whole per-layer path over one synthetic
sequence: for every chunk, unit construction for newly evicted blocks, append,
unit scoring, top-k lookup, and chunk attention with its log-sum-exp merge
(one infllm_step call per chunk).  Inputs are seeded synthetic Q/K/V resident
in HBM before timing starts.

Prints ONE JSON line.  The headline value is chunk-encode context tokens/s on
the 128K-token Llama-3-8B-shaped layer (32 query / 8 kv heads, head_dim 128,
bf16, 128 initial tokens, 4K local window, 128-token units, r_k 4, k_m 32,
512-token chunks); the metric's other parts are in the same line: the 1M-token
streaming encode and the 16 x 128K batched decode under "extra", the MFMA
fraction of the attention kernel under "roofline".  A further extra leg runs
the 128K stream with the positional remap of Section 3.2.
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0

# HBM traffic per launch, from two rocprofv3 --pmc passes (FETCH_SIZE, then WRITE_SIZE; KiB per
# dispatch) over the default benchmark command, each divided by what the same counter reads per KiB
# moved by the plain copy of `bench.py --copy-calibration 1024`.  An entry holds for the kernel
# sources it was taken on (sha256 of each file); it is reported as null once any of them changes.
CSRC = os.path.join(ROOT, "paper_2402_04617_amd", "csrc")
COPY_FETCH = 524300.0 / 1048576.0  # FETCH_SIZE KiB per KiB read by the copy
COPY_WRITE = 1048576.0 / 1048576.0  # WRITE_SIZE KiB per KiB written by the copy
KERNEL_TRAFFIC = {
    # key: {"src": {file: sha256}, "fetch_kib": ..., "write_kib": ...}, per launch (per call for
    # infllm_score_units: its two kernels), from `rocprofv3 --pmc FETCH_SIZE` and `--pmc WRITE_SIZE`
    # runs of `bench.py --legs 1m,decode --no-cpu-baseline --steps 1 --warmup 0`, averaged over the
    # replayed launches the bench line times
    "attend_mfma_llama3-8b-128k": {"src": {"attend_mfma.hip": "8e6f615f1b8b0f3845348431fc7e85216df7b7ee1dd5f879cd23492c919980f7", "launch.h": "773b89a4b862e0906d83400bc662d292d0f41bae789623c3fb8b00f10acda697"},
                                   "fetch_kib": 20095.6, "write_kib": 16896.0},
    "score_llama3-8b-128k": {"src": {"score.hip": "b863ba9bf6e01b4901383469e615c02c7ae9b482693bef88e3f29735e4666a13", "launch.h": "773b89a4b862e0906d83400bc662d292d0f41bae789623c3fb8b00f10acda697"},
                             "fetch_kib": 2086.6 + 2281.5, "write_kib": 64.0 + 34.3},
    "append_llama3-8b-128k": {"src": {"append.hip": "d09c349a86c28dba43f0fcae0b6c8675a8486c7e054e0404c7a79a8b140f5002", "launch.h": "773b89a4b862e0906d83400bc662d292d0f41bae789623c3fb8b00f10acda697"},
                              "fetch_kib": 5717.6, "write_kib": 6659.0},
    "score_llama3-8b-1m": {"src": {"score.hip": "b863ba9bf6e01b4901383469e615c02c7ae9b482693bef88e3f29735e4666a13", "launch.h": "773b89a4b862e0906d83400bc662d292d0f41bae789623c3fb8b00f10acda697"},
                           "fetch_kib": 2086.5 + 16617.6, "write_kib": 64.0 + 282.8},
    "append_llama3-8b-1m": {"src": {"append.hip": "d09c349a86c28dba43f0fcae0b6c8675a8486c7e054e0404c7a79a8b140f5002", "launch.h": "773b89a4b862e0906d83400bc662d292d0f41bae789623c3fb8b00f10acda697"},
                            "fetch_kib": 5717.6, "write_kib": 6659.0},
    "attend_decode": {"src": {"attend_decode.hip": "e9c010e0b521a9e279ded2a3f90fe08bc8e43dc66eb5d0d9b4d86bcbdbd07953", "launch.h": "773b89a4b862e0906d83400bc662d292d0f41bae789623c3fb8b00f10acda697"},
                      "fetch_kib": 270891.2, "write_kib": 544.1},
    "score_decode": {"src": {"score.hip": "b863ba9bf6e01b4901383469e615c02c7ae9b482693bef88e3f29735e4666a13", "launch.h": "773b89a4b862e0906d83400bc662d292d0f41bae789623c3fb8b00f10acda697"},
                     "fetch_kib": 102.5 + 32281.5, "write_kib": 64.0 + 496.0},
}


def _sha(name):
    with open(os.path.join(CSRC, name), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def kernel_traffic_bytes(key):
    t = KERNEL_TRAFFIC.get(key)
    if t is None or any(_sha(f) != h for f, h in t["src"].items()):
        return None
    return 1024.0 * (t["fetch_kib"] / COPY_FETCH + t["write_kib"] / COPY_WRITE)


MASS_DECAY = 0.1  # the frequency score's decay coefficient in the paper's experiments


def measured_peaks():
    """Peaks measured on this GPU by the library's probe program (a child process): bf16 MFMA loop,
    streaming HBM read and copy.  None when the probe has not been built or fails."""
    import subprocess
    exe = os.path.join(ROOT, "paper_2402_04617_amd", "infllm_peaks")
    if not os.path.exists(exe):
        return None
    try:
        r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    except subprocess.TimeoutExpired:
        return None
    if r.returncode != 0:
        log(f"peak probe failed: {r.stderr.strip()}")
        return None
    return json.loads(r.stdout.strip().splitlines()[-1])


def copy_calibration(mib, torch, reps=3):
    """A plain device copy of `mib` MiB (read mib, write mib) repeated `reps` times: the reference
    dispatch whose FETCH_SIZE / WRITE_SIZE per KiB moved calibrates the attention kernel's counters."""
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_mib": mib, "reps": reps, "kernel": "elementwise neg (read N, write N)"}), flush=True)


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def upload_inputs(synth, torch, threads=16):
    """Q [B][Hq][S][D], K, V [B][Hkv][S][D] bf16 on the GPU, drawn span by span."""
    wl = synth.wl
    S, D = wl.seq_len, wl.head_dim
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    out = {}
    for name, H in (("q", wl.n_q_heads), ("k", wl.n_kv_heads), ("v", wl.n_kv_heads)):
        t = torch.empty((wl.batch, H, S, D), dtype=dt, device="cuda")
        fn = getattr(synth, name)
        jobs = [(b, h) for b in range(wl.batch) for h in range(H)]
        with ThreadPoolExecutor(threads) as ex:
            for (b, h), x in zip(jobs, ex.map(lambda bh: fn(bh[0], bh[1], 0, S), jobs)):
                t[b, h].copy_(torch.from_numpy(x).to(dt))
        out[name] = t
    torch.cuda.synchronize()
    return out


def attention_flops(wl, steps):
    """Algorithmic attention flops of a pass: 4*D*Hq per (query, visible key) pair."""
    from paper_2402_04617_amd import infllm as F
    p = params_of(wl)
    total = 0
    for past, n in steps:
        n_init, n_units, local_begin = F.infllm_partition(p, past)
        ctx = n_init + min(wl.topk, n_units) * wl.block_size + (past - local_begin)
        total += 4 * wl.head_dim * wl.n_q_heads * wl.batch * (n * ctx + n * (n + 1) // 2)
    return total


def attention_bytes(wl, steps, parts):
    """HBM bytes of the attention launches of a pass.  Algorithmic (the method's own data): each query
    row read once, each visible context key and value read once per kv head (GQA shares them), the
    output written once.  Split-key partials (written by the attention, read back by the merge when a
    launch splits the keys) are implementation traffic, returned apart."""
    from paper_2402_04617_amd import infllm as F
    p = params_of(wl)
    e = 2 if wl.dtype == "bf16" else 4
    # a split-key partial row: fp16 values + lse + exponent (bf16), float32 values + lse (f32)
    part_row = 2 * wl.head_dim + 8 if wl.dtype == "bf16" else 4 * (wl.head_dim + 1)
    total = partials = 0
    for (past, n), np_ in zip(steps, parts):
        n_init, n_units, local_begin = F.infllm_partition(p, past)
        keys = n_init + min(wl.topk, n_units) * wl.block_size + (past - local_begin) + n
        rows = wl.batch * wl.n_q_heads * n
        total += 2 * rows * wl.head_dim * e + 2 * wl.batch * wl.n_kv_heads * keys * wl.head_dim * e
        partials += np_ * rows * part_row if np_ > 1 else 0
    return total, partials


def params_of(wl, remap=False, mean_repr=False):
    """Method parameters of a workload; remap=True adds the positional remap with Llama-3 rotary
    frequencies (the synthetic q and k are then read as unrotated); mean_repr=True scores units by
    their mean key."""
    from paper_2402_04617_amd import infllm as F
    return F.params(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.n_init, wl.n_local, wl.block_size,
                    wl.n_repr, wl.topk, wl.dtype,
                    rope_inv_freq=F.rope_frequencies(wl.head_dim) if remap else None,
                    repr_mode="mean" if mean_repr else "tokens")


class Stream:
    """Device state of one layer over a sequence, stepped through infllm_step."""

    def __init__(self, wl, inputs, torch, remap=False, mean_repr=False, mass=False):
        from paper_2402_04617_amd import infllm as F
        self.F, self.torch, self.wl = F, torch, wl
        self.p = params_of(wl, remap, mean_repr)
        self.inp = inputs
        S, D = wl.seq_len, wl.head_dim
        # a multiple of 8 keeps every row of the key-sum table 128-byte aligned, so that scoring's
        # 1 KB loads of 64 units fetch no partial cache lines
        self.max_units = (max(1, F.infllm_partition(self.p, S)[1]) + 7) // 8 * 8
        self.mem = F.alloc_memory(self.p, wl.batch, S, self.max_units, F.recommended_ring(self.p, wl.chunk))
        ws = max(F.infllm_workspace_bytes(self.p, wl.batch, wl.chunk), F.infllm_workspace_bytes(self.p, wl.batch, 1))
        self.ws = torch.zeros(ws, dtype=torch.uint8, device="cuda")
        dt = inputs["q"].dtype
        self.out = torch.zeros((wl.batch, wl.n_q_heads, wl.chunk, D), dtype=dt, device="cuda")
        self.lse = torch.zeros((wl.batch, wl.n_q_heads, wl.chunk), dtype=torch.float32, device="cuda")
        self.scores = torch.zeros(wl.batch * wl.n_kv_heads * self.max_units, dtype=torch.float32, device="cuda")
        self.idx = torch.zeros((wl.batch, wl.n_kv_heads, max(1, wl.topk)), dtype=torch.int32, device="cuda")
        self.esize = 2 if dt == torch.bfloat16 else 4
        # after each step: the looked-up units' attention mass and the decayed frequency score
        self.mass = None
        if mass:
            self.mass = torch.zeros((wl.batch, wl.n_kv_heads, max(1, wl.topk)), dtype=torch.float32, device="cuda")
            self.freq = torch.zeros((wl.batch, wl.n_kv_heads, self.max_units), dtype=torch.float32, device="cuda")

    def ptr(self, name, past):
        return self.inp[name].data_ptr() + past * self.wl.head_dim * self.esize

    def step(self, past, n, units_built):
        wl, S, D = self.wl, self.wl.seq_len, self.wl.head_dim
        if self.mass is not None:
            # the step with the looked-up units' attention mass and the frequency score update
            self.F.infllm_step_mass(self.p, self.mem.struct, self.ptr("q", past), S * D, self.ptr("k", past),
                                    self.ptr("v", past), S * D, n, past, units_built, self.scores, self.idx,
                                    self.out, wl.chunk * D, self.lse, MASS_DECAY, self.mass, self.freq, self.ws)
        else:
            self.F.infllm_step(self.p, self.mem.struct, self.ptr("q", past), S * D, self.ptr("k", past),
                               self.ptr("v", past), S * D, n, past, units_built, self.scores, self.idx, self.out,
                               wl.chunk * D, self.lse, self.ws)
        return self.F.infllm_partition(self.p, past)[1]

    def run(self, steps, built=0, on_step=None):
        for i, (past, n) in enumerate(steps):
            built = self.step(past, n, built)
            if on_step is not None:
                on_step(i)
        return built

    def prefill_view(self, b, upto):
        """Untimed set-up of one sequence alone: encode sequence b over [0, upto) through a
        one-sequence view of the memory; returns its units built."""
        F, wl, S, D = self.F, self.wl, self.wl.seq_len, self.wl.head_dim
        m, s = self.mem, self.mem.struct
        ptr = lambda t: None if t is None else t[b].data_ptr()  # noqa: E731
        view = F.Memory(1, s.capacity, m.k[b].data_ptr(), m.v[b].data_ptr(), s.max_units, ptr(m.repr_idx),
                        ptr(m.unit_ksum), ptr(m.qprefix), ptr(m.rpart), s.ring, ptr(m.k_rot))
        off = lambda name, past: self.inp[name][b].data_ptr() + past * D * self.esize  # noqa: E731
        built = 0
        for past in range(0, upto, wl.chunk):
            n = min(wl.chunk, upto - past)
            nu = F.infllm_partition(self.p, past)[1]
            if nu > built:
                F.infllm_build_units(self.p, view, built, nu - built, past)
                built = nu
            F.infllm_append(self.p, view, off("q", past), S * D, off("k", past), off("v", past), S * D, n, past)
        nu = F.infllm_partition(self.p, upto)[1]
        if nu > built:
            F.infllm_build_units(self.p, view, built, nu - built, upto)
            built = nu
        return built

    def prefill_memory(self, upto):
        """Untimed set-up for decode: append positions [0, upto) chunk by chunk and build every unit."""
        F, wl, S, D = self.F, self.wl, self.wl.seq_len, self.wl.head_dim
        built = 0
        for past in range(0, upto, wl.chunk):
            n = min(wl.chunk, upto - past)
            nu = F.infllm_partition(self.p, past)[1]
            if nu > built:
                F.infllm_build_units(self.p, self.mem.struct, built, nu - built, past)
                built = nu
            F.infllm_append(self.p, self.mem.struct, self.ptr("q", past), S * D, self.ptr("k", past),
                            self.ptr("v", past), S * D, n, past)
        nu = F.infllm_partition(self.p, upto)[1]
        if nu > built:
            F.infllm_build_units(self.p, self.mem.struct, built, nu - built, upto)
            built = nu
        return built

    def attention_replay(self, steps, idx_hist):
        """The attention kernels alone, in the step's launch configuration on the lookups recorded from a
        real pass (the plain kernel: in the step the same launches also select the units in their
        prologue), issued back to back on the launching stream between two HIP events: returns the
        average launch duration (ms) and the number of key parts of each launch."""
        F, torch, wl, S, D = self.F, self.torch, self.wl, self.wl.seq_len, self.wl.head_dim
        parts_seen = []
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for i, (past, n) in enumerate(steps):
            parts_seen.append(F.infllm_attend_partial(self.p, self.mem.struct, self.ptr("q", past), S * D, n, past,
                                                      idx_hist[i], wl.topk, self.out, wl.chunk * D, self.lse,
                                                      self.ws))
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / len(steps), parts_seen


def time_steps(torch, fn, steps, warmup):
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(steps):
        fn()
    t1.record()
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / steps


def graph_replay_us(torch, fn, n=20, reps=5):
    """Average duration of one call of `fn` (a library call enqueueing kernels on torch's current
    stream): n calls captured into one HIP graph, replayed `reps` times between two HIP events.  The
    graph removes the host's per-call cost, which exceeds the small kernels' own duration; what is
    left is each launch plus its gap to the next.  Every call replayed here rewrites the same outputs
    from the same inputs, so replays change no state."""
    fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(n):
            fn()
    g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    del g
    return a.elapsed_time(b) * 1e3 / (n * reps)


def hbm_entry(kernel, workload, us, algorithmic_bytes, traffic=None, **more):
    """Roofline entry of an HBM-bound launch: algorithmic bytes / event-timed duration vs 8 TB/s."""
    gbs = algorithmic_bytes / (us * 1e-6) / 1e9
    e = {"kernel": kernel, "workload": workload, "bound": "hbm", "avg_us": us, "algorithmic_bytes": algorithmic_bytes,
         "achieved": gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": gbs / PEAK_HBM_GBS,
         "traffic": kernel_traffic_bytes(traffic) if traffic else None}
    e.update(more)
    return e


def score_bytes(wl, n_units, n):
    """infllm_score_units: the chunk's queries read once, each unit's key sum (float32) and score."""
    return (wl.batch * wl.n_q_heads * n * wl.head_dim * 2
            + wl.batch * wl.n_kv_heads * n_units * (wl.head_dim * 4 + 4))


def append_bytes(wl, n):
    """infllm_append of n positions: queries and the chunk's K/V read, K/V stored, the float64 running
    sum written for each new position and read for each token leaving the window, that token's key
    read, its partial representative scores (D/8 float64 per token) written."""
    B, Hq, Hkv, D = wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim
    return (B * Hq * n * D * 2 + 2 * 2 * B * Hkv * n * D * 2 + 2 * B * Hkv * n * D * 8 + B * Hkv * n * D * 2
            + B * Hkv * n * (D // 8) * 8)


def encode_leg(name, seed, steps, warmup, torch, want_roofline=True, remap=False, inputs=None, mean_repr=False,
               mass=False, **method):
    """One encode stream of workload `name`; `method` overrides method parameters (block_size,
    n_repr, topk, chunk) on the same inputs."""
    from workload import WORKLOADS, Synth
    wl = WORKLOADS[name]
    if method:
        wl = dataclasses.replace(wl, **method)
    t = time.time()
    synth = Synth(WORKLOADS[name], seed)
    if inputs is None:
        inputs = upload_inputs(synth, torch)
        log(f"{name}: inputs resident in HBM ({time.time() - t:.1f}s)")
    st = Stream(wl, inputs, torch, remap, mean_repr, mass)
    plan = wl.step_starts()
    ms = time_steps(torch, lambda: st.run(plan), steps, warmup)
    res = {"workload": name + ("+remap" if remap else "") + ("+mean-repr" if mean_repr else "") +
           ("+unit-mass" if mass else ""),
           "seq_len": wl.seq_len, "ms_per_step": ms,
           "ctx_tok_per_s": wl.seq_len * wl.batch / (ms / 1e3)}
    if method:
        res["method"] = {"block_size": wl.block_size, "n_repr": wl.n_repr, "topk": wl.topk, "chunk": wl.chunk}
    if want_roofline:
        # one more (untimed) pass recording the lookup of every chunk, then the attention replay
        idx_hist = torch.zeros((len(plan),) + tuple(st.idx.shape), dtype=torch.int32, device="cuda")
        st.run(plan, on_step=lambda i: idx_hist[i].copy_(st.idx))
        avg_ms, parts = st.attention_replay(plan, idx_hist)
        flops = attention_flops(wl, plan)
        tot_ms = avg_ms * len(plan)
        ab, pb = attention_bytes(wl, plan, parts)
        res["attention"] = {"launches": len(plan), "avg_ms": avg_ms, "total_ms": tot_ms,
                            "algorithmic_flops": flops, "tflops": flops / (tot_ms / 1e3) / 1e12,
                            "algorithmic_bytes_per_launch": ab / len(plan),
                            "split_partial_bytes_per_launch": pb / len(plan),
                            "parts_per_launch": sorted(set(parts))}
        # the memory-bound launches of the last chunk (the most units), replayed alone
        past, n = plan[-1]
        F = st.F
        nu = F.infllm_partition(st.p, past)[1]
        S, D = wl.seq_len, wl.head_dim
        us = graph_replay_us(torch, lambda: F.infllm_score_units(st.p, st.mem.struct, st.ptr("q", past), S * D, n,
                                                                 nu, st.scores, st.ws))
        res["kernels"] = [hbm_entry("infllm_score_units (query sums + score_kernel)", f"{res['workload']} last chunk",
                                    us, score_bytes(wl, nu, n), traffic=f"score_{name}", n_units=nu)]
        if not mean_repr:
            us = graph_replay_us(torch, lambda: F.infllm_append(st.p, st.mem.struct, st.ptr("q", past), S * D,
                                                                st.ptr("k", past), st.ptr("v", past), S * D, n, past))
            res["kernels"].append(hbm_entry("append_kernel (infllm_append: scan + copy)",
                                            f"{res['workload']} last chunk", us, append_bytes(wl, n),
                                            traffic=f"append_{name}"))
    return res, synth, st


def decode_leg(seed, steps, warmup, torch):
    from workload import WORKLOADS, Synth
    wl = WORKLOADS["llama3-8b-decode-16x128k"]
    t = time.time()
    synth = Synth(wl, seed)
    inputs = upload_inputs(synth, torch)
    log(f"decode: inputs resident ({time.time() - t:.1f}s)")
    st = Stream(wl, inputs, torch)
    t = time.time()
    built = st.prefill_memory(wl.prefill_len)
    torch.cuda.synchronize()
    log(f"decode: memory of {wl.prefill_len} tokens x {wl.batch} built ({time.time() - t:.1f}s)")
    plan = wl.step_starts()[-wl.decode_steps:]
    ms = time_steps(torch, lambda: st.run(plan, built=built), steps, warmup)
    us_tok = ms * 1e3 / len(plan)
    res = {"workload": wl.name, "decode_steps": len(plan), "batch": wl.batch, "us_per_step": us_tok,
           "tok_per_s": wl.batch * len(plan) / (ms / 1e3)}
    # the decode attention of the last step alone (its lookup as the step wrote it), replayed
    past, n = plan[-1]
    F, S, D = st.F, wl.seq_len, wl.head_dim
    idx = st.idx.clone()
    parts = []
    us = graph_replay_us(torch, lambda: parts.append(F.infllm_attend_partial(
        st.p, st.mem.struct, st.ptr("q", past), S * D, n, past, idx, wl.topk, st.out, wl.chunk * D, st.lse, st.ws)))
    ab, pb = attention_bytes(wl, [(past, n)], [parts[-1]])
    res["kernels"] = [hbm_entry("attend_decode_kernel (infllm_attend_partial)", f"{wl.name} step {len(plan) - 1}",
                                us, ab, traffic="attend_decode", split_partial_bytes=pb, parts=parts[-1])]
    s_us = graph_replay_us(torch, lambda: F.infllm_score_units(st.p, st.mem.struct, st.ptr("q", past), S * D, n,
                                                               F.infllm_partition(st.p, past)[1], st.scores, st.ws))
    res["kernels"].append(hbm_entry("infllm_score_units (query sums + score_kernel)",
                                    f"{wl.name} step {len(plan) - 1}", s_us,
                                    score_bytes(wl, F.infllm_partition(st.p, past)[1], n), traffic="score_decode"))
    return res, st


def multilayer_leg(st1, layers, steps, warmup, torch):
    """Streaming encode of a whole model's attention memory: `layers` layers of the 1M workload,
    each with its own context memory resident in HBM (no offload), chunk-major (every layer's
    step for a chunk before the next chunk).  All layers read the same synthetic inputs, which
    changes nothing in the work done."""
    wl = st1.wl
    streams = [st1] + [Stream(wl, st1.inp, torch) for _ in range(layers - 1)]
    plan = wl.step_starts()

    def run():
        built = [0] * layers
        for past, n in plan:
            for li, st in enumerate(streams):
                built[li] = st.step(past, n, built[li])
    ms = time_steps(torch, run, steps, warmup)
    hbm = sum(sum(t.numel() * t.element_size() for t in (s_.mem.k, s_.mem.v, s_.mem.unit_ksum, s_.mem.repr_idx,
                                                           s_.mem.qprefix, s_.mem.rpart)) for s_ in streams)
    return {"workload": f"{wl.name} x {layers} layers", "layers": layers, "seq_len": wl.seq_len, "ms_per_step": ms,
            "ctx_tok_per_s": wl.seq_len / (ms / 1e3), "memory_resident_gb": hbm / 1e9}


def decode_varlen_leg(st, steps, warmup, torch, spacing=6144):
    """Serving-style decode: the 16 sequences at different depths (128K, 122K, ..., 38K prior tokens),
    stepped together by infllm_step_varlen.  Each sequence's memory is first rebuilt alone to its
    own length (untimed); the step inputs, gathered from each sequence's own position, are made
    before timing."""
    F, wl = st.F, st.wl
    B, S, D = wl.batch, wl.seq_len, wl.head_dim
    lens = [wl.prefill_len - spacing * b for b in range(B)]
    built = []
    for b in range(B):
        built.append(st.prefill_view(b, lens[b]))
    torch.cuda.synchronize()
    T = wl.decode_steps
    pos = torch.tensor(lens, device="cuda")
    ar = torch.arange(B, device="cuda")

    def gather(x, t):
        return x[ar, :, pos + t].unsqueeze(2).contiguous()  # [B][H][1][D]
    qs = [gather(st.inp["q"], t) for t in range(T)]
    ks = [gather(st.inp["k"], t) for t in range(T)]
    vs = [gather(st.inp["v"], t) for t in range(T)]
    pasts = [[lens[b] + t for b in range(B)] for t in range(T)]
    builts = [built] + [[F.infllm_partition(st.p, pp)[1] for pp in pasts[t]] for t in range(T - 1)]
    out = torch.zeros((B, wl.n_q_heads, 1, D), dtype=st.out.dtype, device="cuda")
    lse = torch.zeros((B, wl.n_q_heads, 1), dtype=torch.float32, device="cuda")
    scores = torch.zeros((B, wl.n_kv_heads, st.max_units), dtype=torch.float32, device="cuda")

    def run():
        for t in range(T):
            F.infllm_step_varlen(st.p, st.mem.struct, qs[t], D, ks[t], vs[t], D, 1, pasts[t], builts[t], scores,
                                 st.idx, out, D, lse, st.ws)
    ms = time_steps(torch, run, steps, warmup)
    return {"workload": wl.name + "+varlen", "decode_steps": T, "batch": B, "prior_tokens": [min(lens), max(lens)],
            "us_per_step": ms * 1e3 / T, "tok_per_s": B * T / (ms / 1e3)}


def _ordinal(n):
    return f"{n}{'nd' if n == 2 else 'rd' if n == 3 else 'th'}"


def _oracle_threads():
    """Host cores this process may run on, and the BLAS threads the oracle's matrix products use."""
    cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        blas = None
    return cores, blas


def _oracle_head(wl, synth, b, g, p1):
    """The oracle over one (sequence, kv head) of a workload: inputs [0, p1) of its G query heads."""
    from oracle import infllm_oracle as O
    G = wl.group
    q = np.stack([synth.q(b, g * G + h, 0, p1) for h in range(G)])[None]
    k = synth.k(b, g, 0, p1)[None, None]
    v = synth.v(b, g, 0, p1)[None, None]
    op = O.Params(G, 1, wl.head_dim, wl.n_init, wl.n_local, wl.block_size, wl.n_repr, wl.topk)
    return O, O.StreamOracle(q, k, v, op), op


def _oracle_stream(wl, synth, plan, stride, b=0):
    """Oracle seconds for one kv head: every unit the plan builds, then every `stride`-th step of the
    plan scored, looked up and attended.  Returns (unit seconds, step seconds, steps timed, units)."""
    O, so, op = _oracle_head(wl, synth, b, 0, plan[-1][0] + plan[-1][1])
    last_units = O.partition(plan[-1][0], op).n_units
    t0 = time.time()
    so.group_query_sum(0, 0)
    for u in range(last_units):
        so.repr_offsets(0, 0, u)
    t_units = time.time() - t0
    sample = plan[stride - 1::stride] if stride > 1 else plan
    t0 = time.time()
    for past, n in sample:
        so.step(0, past, n)
    return t_units, time.time() - t0, len(sample), last_units


def cpu_baseline(synth, n_chunk_samples=64, extra=True):
    """The oracle, unchanged, on bounded samples, timed on this host's cores.

    Headline (128K encode): kv head 0 (of 8) with its 4 query heads; all of that head's units are
    built and every 4th chunk is scored, looked up and attended; extrapolated linearly to all chunks
    and all kv heads.  With `extra`: the 16 x 128K decode (sequence 0, kv head 0: its 991 units, then
    every 64th of the 256 steps; per step x16 sequences x8 kv heads) and the 1M encode (kv head 0:
    all 8,155 units, every 128th chunk; extrapolated over chunks and kv heads)."""
    from workload import WORKLOADS, Synth
    cores, blas = _oracle_threads()
    wl = synth.wl
    plan = wl.step_starts()
    stride = max(1, len(plan) // n_chunk_samples)
    t_units, t_steps, n_s, nu = _oracle_stream(wl, synth, plan, stride)
    t_full = wl.n_kv_heads * (t_units + t_steps * len(plan) / n_s)
    out = {"value": wl.seq_len / t_full, "unit": "ctx tok/s", "cores": cores, "blas_threads": blas,
           "kind": "oracle",
           "sample": f"kv head 0 of {wl.n_kv_heads}: all {nu} units built, {n_s} of {len(plan)} chunks (every "
                     f"{_ordinal(stride)}) scored/selected/attended; extrapolated x{len(plan) / n_s:g} over "
                     f"chunks and x{wl.n_kv_heads} over kv heads",
           "sample_seconds": t_units + t_steps}
    if not extra:
        return out
    # 16 x 128K decode: oracle microseconds per decode step (16 tokens)
    wd = WORKLOADS["llama3-8b-decode-16x128k"]
    sd = Synth(wd, synth.seed)
    dplan = wd.step_starts()[-wd.decode_steps:]
    t_u, t_s, n_d, nu_d = _oracle_stream(wd, sd, dplan, 64)
    per_step = t_s / n_d * wd.batch * wd.n_kv_heads  # the units were built before the steps (prior context)
    out["decode_16x128k"] = {"us_per_step": per_step * 1e6, "unit": "us per decode step (16 tokens)",
                             "sample": f"sequence 0, kv head 0: its {nu_d} units built ({t_u:.1f} s, not counted: "
                                       f"prior context), {n_d} of {len(dplan)} steps timed; x{wd.batch} sequences "
                                       f"x{wd.n_kv_heads} kv heads",
                             "sample_seconds": t_u + t_s}
    # 1M encode, extrapolated from every 128th chunk
    w1 = WORKLOADS["llama3-8b-1m"]
    s1 = Synth(w1, synth.seed)
    p1 = w1.step_starts()
    t_u, t_s, n_1, nu_1 = _oracle_stream(w1, s1, p1, 128)
    t1 = w1.n_kv_heads * (t_u + t_s * len(p1) / n_1)
    out["encode_1m"] = {"value": w1.seq_len / t1, "unit": "ctx tok/s", "extrapolated": True,
                        "sample": f"kv head 0 of {w1.n_kv_heads}: all {nu_1} units built, {n_1} of {len(p1)} chunks "
                                  f"(every 128th) scored/selected/attended; extrapolated x{len(p1) / n_1:g} over "
                                  f"chunks and x{w1.n_kv_heads} over kv heads",
                        "sample_seconds": t_u + t_s}
    return out


# Memory settings of the paper's studies of them: representative tokens r_k, selected units
# k_m, and unit size l_bs with the total context held at 12K (4K local + 8K selected).
SWEEP = ([{"n_repr": r} for r in (1, 2, 4, 8)]
         + [{"topk": k} for k in (2, 4, 8, 16, 32, 64, 96, 128)]
         + [{"block_size": b, "topk": 8192 // b} for b in (32, 64, 128, 256)])


def sweep(seed, steps, warmup, torch):
    """128K stream under each memory setting of SWEEP (same inputs): one JSON line per setting."""
    base, _, st = encode_leg("llama3-8b-128k", seed, steps, warmup, torch)
    inputs = st.inp
    del st
    for m in SWEEP:
        r, _, s2 = encode_leg("llama3-8b-128k", seed, steps, warmup, torch, inputs=inputs, **m)
        del s2
        torch.cuda.empty_cache()
        a = r["attention"]
        print(json.dumps({"sweep": r["method"], "ms_per_step": r["ms_per_step"], "ctx_tok_per_s": r["ctx_tok_per_s"],
                          "attention_us_per_launch": a["avg_ms"] * 1e3, "attention_tflops": a["tflops"],
                          "attention_ms_per_step": a["total_ms"]}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--legs", default="32k,1m,1m-paper,32l-1m,decode,remap,mean,mass",
                    help="extra legs: comma list of 32k, 1m, 1m-paper, 32l-1m, decode, remap, mean, mass (or 'none')")
    ap.add_argument("--sweep", action="store_true",
                    help="only time the 128K stream under the paper's memory settings (r_k, k_m, l_bs)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run the plain-copy calibration dispatch of MIB MiB (for the traffic counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this path runs on one GPU: the whole context memory lives in one "
                                   "MI355X's HBM and no step exchanges data between GPUs; run with --gpus 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch
    if args.copy_calibration > 0:
        torch.cuda.set_device(0)
        copy_calibration(args.copy_calibration, torch)
        return
    from paper_2402_04617_amd import infllm as F
    F.lib()
    torch.cuda.set_device(0)
    if args.sweep:
        sweep(args.seed, args.steps, args.warmup, torch)
        return

    main_res, synth, st = encode_leg("llama3-8b-128k", args.seed, args.steps, args.warmup, torch)
    log(f"128K: {main_res['ms_per_step']:.2f} ms/step, {main_res['ctx_tok_per_s'] / 1e6:.2f}M ctx tok/s; "
        f"attention {main_res['attention']['tflops']:.0f} TFLOP/s")
    extra = {}
    kernels = list(main_res.get("kernels", []))
    legs = [] if args.legs == "none" else [x.strip() for x in args.legs.split(",") if x.strip()]
    if "remap" in legs:
        # the same 128K stream with the positional remap (Llama-3 rotary frequencies), same inputs
        rr, _, st_r = encode_leg("llama3-8b-128k", args.seed, args.steps, args.warmup, torch, remap=True,
                                 inputs=st.inp)
        del st_r
        extra["encode_128k_remap"] = rr
        log(f"128K remap: {rr['ms_per_step']:.2f} ms/step, {rr['ctx_tok_per_s'] / 1e6:.2f}M ctx tok/s; "
            f"attention {rr['attention']['tflops']:.0f} TFLOP/s")
    if "mean" in legs:
        # the same 128K stream with units represented by their mean key
        rm, _, st_m = encode_leg("llama3-8b-128k", args.seed, args.steps, args.warmup, torch, mean_repr=True,
                                 inputs=st.inp)
        del st_m
        extra["encode_128k_mean_repr"] = rm
        log(f"128K mean repr: {rm['ms_per_step']:.2f} ms/step, {rm['ctx_tok_per_s'] / 1e6:.2f}M ctx tok/s")
    if "mass" in legs:
        # the same 128K stream with the attention mass / frequency score after every step
        rs, _, st_s = encode_leg("llama3-8b-128k", args.seed, args.steps, args.warmup, torch, want_roofline=False,
                                 inputs=st.inp, mass=True)
        del st_s
        rs["added_us_per_step"] = (rs["ms_per_step"] - main_res["ms_per_step"]) * 1e3 / len(st.wl.step_starts())
        rs["decay"] = MASS_DECAY
        rs["entry"] = "infllm_step_mass"
        extra["encode_128k_unit_mass"] = rs
        log(f"128K with unit mass: {rs['ms_per_step']:.2f} ms/step (+{rs['added_us_per_step']:.1f} us per chunk)")
    del st
    torch.cuda.empty_cache()
    if "32k" in legs:
        # the Mistral-7B-shaped 32K stream (k_m 16)
        r2, _, st2 = encode_leg("mistral7b-32k", args.seed, args.steps, args.warmup, torch)
        del st2
        torch.cuda.empty_cache()
        extra["encode_32k"] = r2
        log(f"32K: {r2['ms_per_step']:.2f} ms/step, {r2['ctx_tok_per_s'] / 1e6:.2f}M ctx tok/s; "
            f"attention {r2['attention']['tflops']:.0f} TFLOP/s")
    if "1m" in legs or "1m-paper" in legs or "32l-1m" in legs:
        r1, _, st1 = encode_leg("llama3-8b-1m", args.seed, max(1, min(args.steps, 2)), 1, torch)
        if "1m" in legs:
            extra["encode_1m"] = r1
            kernels += r1.get("kernels", [])
            log(f"1M: {r1['ms_per_step']:.1f} ms/step, {r1['ctx_tok_per_s'] / 1e6:.2f}M ctx tok/s")
        if "1m-paper" in legs:
            # the paper's settings for its 1,024K run: 2048-token chunks, one representative token
            rp, _, st2 = encode_leg("llama3-8b-1m", args.seed, max(1, min(args.steps, 2)), 1, torch,
                                    inputs=st1.inp, chunk=2048, n_repr=1)
            del st2
            extra["encode_1m_paper_settings"] = rp
            log(f"1M (chunk 2048, r_k 1): {rp['ms_per_step']:.1f} ms/step, "
                f"{rp['ctx_tok_per_s'] / 1e6:.2f}M ctx tok/s")
        if "32l-1m" in legs:
            try:
                rl = multilayer_leg(st1, 32, 1, 1, torch)
                extra["encode_1m_32_layers"] = rl
                log(f"1M x 32 layers: {rl['ms_per_step'] / 1e3:.2f} s/pass, {rl['ctx_tok_per_s'] / 1e3:.0f}K ctx tok/s "
                    f"through all layers, {rl['memory_resident_gb']:.0f} GB of memory resident")
            except torch.cuda.OutOfMemoryError as e:  # report, keep the rest of the line
                extra["encode_1m_32_layers"] = {"error": f"out of device memory: {e}"[:200]}
            torch.cuda.empty_cache()
        del st1
        torch.cuda.empty_cache()
    if "decode" in legs:
        rd, st_d = decode_leg(args.seed, max(1, min(args.steps, 3)), 1, torch)
        extra["decode_16x128k"] = rd
        kernels += rd.get("kernels", [])
        log(f"decode: {rd['us_per_step']:.1f} us/step (16 seqs)")
        rv = decode_varlen_leg(st_d, max(1, min(args.steps, 3)), 1, torch)
        extra["decode_16_varlen"] = rv
        log(f"decode, lengths {rv['prior_tokens'][0]}..{rv['prior_tokens'][1]}: {rv['us_per_step']:.1f} us/step")
        del st_d
        torch.cuda.empty_cache()

    att = main_res["attention"]
    achieved = att["tflops"]
    line = {
        "metric": "chunk-encode context tok/s at 128K & 1M; decode µs/token; % MFMA/HBM peak",
        "value": main_res["ctx_tok_per_s"],
        "unit": "ctx tok/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": main_res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "llama3-8b-128k", "seq_len": 131072, "batch": 1, "q_heads": 32, "kv_heads": 8,
                   "head_dim": 128, "n_init": 128, "n_local": 4096, "block_size": 128, "n_repr": 4, "topk": 32,
                   "chunk": 512, "parallelism": "single-gpu"},
        "roofline": {"bound": "mfma", "kernel": "attend_mfma_kernel<128, 0, false>", "achieved": achieved,
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                     "traffic": kernel_traffic_bytes("attend_mfma_llama3-8b-128k"), "traffic_unit": "B/launch",
                     "algorithmic_bytes": att["algorithmic_bytes_per_launch"],
                     "split_partial_bytes": att["split_partial_bytes_per_launch"], "avg_launch_ms": att["avg_ms"],
                     "launches_per_step": att["launches"], "kernels": kernels},
        "extra": extra,
    }
    peaks = measured_peaks()
    if peaks is not None:
        line["roofline"]["measured_peaks"] = peaks
        line["roofline"]["frac_of_measured"] = achieved / peaks["mfma_bf16_tflops"]
        log(f"measured peaks: {peaks}")
    if not args.no_cpu_baseline:
        t = time.time()
        line["cpu_baseline"] = cpu_baseline(synth)
        log(f"cpu baseline: {line['cpu_baseline']['value']:.1f} ctx tok/s ({time.time() - t:.1f}s)")
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
