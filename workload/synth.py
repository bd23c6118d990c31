"""Seeded, streamable synthetic Q/K/V for single-layer long-context attention.

Inputs stand in for the paper's long-document and passkey workloads (Section 4:
InfiniteBench averages ~145K tokens; the passkey runs reach 1,024K): Gaussian
queries/keys/values with a few planted "needle" blocks whose keys lean along a
per-(sequence, kv-head) random unit direction u that is also added to every 8th
query of the kv head's query group.

Every value is a pure function of (seed, workload, tensor, sequence, head,
position), drawn from NumPy's counter-based Philox generator in spans of
``SPAN`` tokens, so a 1M-token sequence can be produced piecewise and in
parallel, and any span can be re-drawn alone.  Draws are float32, scaled, then
planted, then rounded once (round-to-nearest-even) to the workload's dtype.
"""
from __future__ import annotations

import dataclasses
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, Optional

import numpy as np

SPAN = 1024  # tokens per independent random stream

_TENSOR_ID = {"q": 1, "k": 2, "v": 3, "dir": 4, "needle": 5}


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and method parameters of one synthetic single-layer workload."""

    name: str
    wid: int                 # stable id mixed into the random keys
    batch: int               # independent sequences
    seq_len: int             # tokens per sequence (prior context + steps)
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    dtype: str               # "f32" or "bf16"
    n_init: int              # l_I
    n_local: int             # l_L
    block_size: int          # l_bs
    n_repr: int              # r_k
    topk: int                # k_m
    chunk: int               # l_X while encoding
    qk_std: float            # std of the Gaussian part of q and k
    v_std: float
    n_needles: int           # planted blocks per (sequence, kv head)
    decode_steps: int = 0    # > 0: the last `decode_steps` tokens arrive one per step
    needle_shift: float = 2.0
    needle_query_every: int = 8

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def prefill_len(self) -> int:
        """Tokens encoded chunk by chunk before any single-token step."""
        return self.seq_len - self.decode_steps

    def step_starts(self):
        """(past_len, n_q) of every step, in order: chunked encode, then decode."""
        steps = []
        p = 0
        while p < self.prefill_len:
            n = min(self.chunk, self.prefill_len - p)
            steps.append((p, n))
            p += n
        for t in range(self.decode_steps):
            steps.append((self.prefill_len + t, 1))
        return steps


def _wl(**kw) -> Workload:
    return Workload(**kw)


WORKLOADS: Dict[str, Workload] = {
    w.name: w
    for w in [
        # Tiny fp32 case: 2 query heads on 1 kv head, head_dim 64.
        _wl(name="tiny-2k-f32", wid=1, batch=1, seq_len=2048, n_q_heads=2, n_kv_heads=1,
            head_dim=64, dtype="f32", n_init=16, n_local=256, block_size=32, n_repr=4,
            topk=4, chunk=64, qk_std=1.0 / 8.0, v_std=1.0, n_needles=4),
        # Mistral-7B layer shape, 32K tokens, bf16, GQA 4:1.
        _wl(name="mistral7b-32k", wid=2, batch=1, seq_len=32768, n_q_heads=32, n_kv_heads=8,
            head_dim=128, dtype="bf16", n_init=128, n_local=4096, block_size=128, n_repr=4,
            topk=16, chunk=512, qk_std=128 ** -0.5, v_std=128 ** -0.5, n_needles=2),
        # Llama-3-8B layer shape, 128K tokens.
        _wl(name="llama3-8b-128k", wid=3, batch=1, seq_len=131072, n_q_heads=32, n_kv_heads=8,
            head_dim=128, dtype="bf16", n_init=128, n_local=4096, block_size=128, n_repr=4,
            topk=32, chunk=512, qk_std=128 ** -0.5, v_std=128 ** -0.5, n_needles=4),
        # Llama-3-8B layer shape, 1M tokens streamed.
        _wl(name="llama3-8b-1m", wid=4, batch=1, seq_len=1048576, n_q_heads=32, n_kv_heads=8,
            head_dim=128, dtype="bf16", n_init=128, n_local=4096, block_size=128, n_repr=4,
            topk=32, chunk=512, qk_std=128 ** -0.5, v_std=128 ** -0.5, n_needles=8),
        # Batched decode: 16 sequences x 128K prior tokens, then 256 single-token steps.
        _wl(name="llama3-8b-decode-16x128k", wid=5, batch=16, seq_len=131072 + 256,
            n_q_heads=32, n_kv_heads=8, head_dim=128, dtype="bf16", n_init=128, n_local=4096,
            block_size=128, n_repr=4, topk=32, chunk=512, qk_std=128 ** -0.5,
            v_std=128 ** -0.5, n_needles=4, decode_steps=256),
    ]
}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns the uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _stream(seed: int, wid: int, tensor: str, b: int, h: int, span: int) -> np.random.Generator:
    ss = np.random.SeedSequence([seed, wid, _TENSOR_ID[tensor], b, h, span])
    key = int.from_bytes(ss.generate_state(2, np.uint64).tobytes(), "little")
    return np.random.Generator(np.random.Philox(key=key))


class Synth:
    """Draws the inputs of one workload for one seed, span by span."""

    def __init__(self, wl: Workload, seed: int = 0):
        self.wl = wl
        self.seed = seed
        # Needle blocks: block-aligned spans starting at n_init, taken among the
        # blocks that lie wholly before the last step's local window and chunk.
        last_past = wl.step_starts()[-1][0]
        avail = max(0, (last_past - wl.n_init - wl.n_local) // wl.block_size)
        self._needles = {}
        self._dirs = {}
        for b in range(wl.batch):
            for g in range(wl.n_kv_heads):
                rng = _stream(seed, wl.wid, "needle", b, g, 0)
                n = min(wl.n_needles, avail)
                self._needles[(b, g)] = np.sort(rng.choice(avail, size=n, replace=False)) if n else \
                    np.zeros(0, dtype=np.int64)
                d = _stream(seed, wl.wid, "dir", b, g, 0).standard_normal(wl.head_dim)
                self._dirs[(b, g)] = (d / np.linalg.norm(d)).astype(np.float32)

    # -- structure --------------------------------------------------------
    def needle_blocks(self, b: int, g: int) -> np.ndarray:
        """Indices j of planted blocks: tokens [n_init + j*block_size, ... + block_size)."""
        return self._needles[(b, g)]

    def direction(self, b: int, g: int) -> np.ndarray:
        return self._dirs[(b, g)]

    # -- raw draws ----------------------------------------------------------
    def _gauss(self, tensor: str, b: int, h: int, p0: int, p1: int) -> np.ndarray:
        D = self.wl.head_dim
        out = np.empty((p1 - p0, D), dtype=np.float32)
        s0, s1 = p0 // SPAN, (p1 - 1) // SPAN
        for s in range(s0, s1 + 1):
            a, e = max(p0, s * SPAN), min(p1, (s + 1) * SPAN)
            x = _stream(self.seed, self.wl.wid, tensor, b, h, s).standard_normal(
                (SPAN, D), dtype=np.float32)
            out[a - p0:e - p0] = x[a - s * SPAN:e - s * SPAN]
        return out

    def _round(self, x: np.ndarray) -> np.ndarray:
        if self.wl.dtype == "bf16":
            return bf16_bits_to_f32(f32_to_bf16_bits(x))
        return x

    # -- public draws (float32 values exactly representable in wl.dtype) -----
    def q(self, b: int, h: int, p0: int, p1: int) -> np.ndarray:
        wl = self.wl
        x = self._gauss("q", b, h, p0, p1) * np.float32(wl.qk_std)
        g = h // wl.group
        pos = np.arange(p0, p1)
        sel = (pos % wl.needle_query_every) == 0
        x[sel] += self._dirs[(b, g)]
        return self._round(x)

    def k(self, b: int, g: int, p0: int, p1: int) -> np.ndarray:
        wl = self.wl
        x = self._gauss("k", b, g, p0, p1) * np.float32(wl.qk_std)
        shift = np.float32(wl.needle_shift) * self._dirs[(b, g)]
        for j in self._needles[(b, g)]:
            a = wl.n_init + int(j) * wl.block_size
            e = a + wl.block_size
            lo, hi = max(a, p0), min(e, p1)
            if lo < hi:
                x[lo - p0:hi - p0] += shift
        return self._round(x)

    def v(self, b: int, g: int, p0: int, p1: int) -> np.ndarray:
        return self._round(self._gauss("v", b, g, p0, p1) * np.float32(self.wl.v_std))

    # -- whole tensors -----------------------------------------------------
    def full(self, tensor: str, p0: int = 0, p1: Optional[int] = None, threads: int = 8) -> np.ndarray:
        """float32 [batch][heads][p1-p0][D] for tensor in {"q","k","v"}."""
        wl = self.wl
        p1 = wl.seq_len if p1 is None else p1
        H = wl.n_q_heads if tensor == "q" else wl.n_kv_heads
        out = np.empty((wl.batch, H, p1 - p0, wl.head_dim), dtype=np.float32)
        fn = getattr(self, tensor)
        jobs = [(b, h) for b in range(wl.batch) for h in range(H)]

        def run(bh):
            b, h = bh
            out[b, h] = fn(b, h, p0, p1)

        if threads > 1 and len(jobs) > 1:
            with ThreadPoolExecutor(threads) as ex:
                list(ex.map(run, jobs))
        else:
            for j in jobs:
                run(j)
        return out
