"""Helpers for the GPU parity tests: device tensors, a stream runner over the C ABI, comparisons.

The runner drives the library only through paper_2402_04617_amd.infllm (the C
ABI); expected values always come from oracle/ on the same seeded inputs.
"""
from __future__ import annotations

import sys
from typing import Dict, Iterable, Optional

import numpy as np
import torch

from oracle import infllm_oracle as O
from paper_2402_04617_amd import infllm as F


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def dev(x: np.ndarray, dtype: str) -> torch.Tensor:
    """Upload float32 values (exactly representable in `dtype`)."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    return t.cuda()


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy() if t.dtype in (torch.bfloat16, torch.float16) else t.detach().cpu().numpy()


def oparams(p: F.Params) -> O.Params:
    freqs = tuple(float(p.rope_inv_freq[i]) for i in range(p.head_dim // 2)) if p.remap else None
    return O.Params(p.n_q_heads, p.n_kv_heads, p.head_dim, p.n_init, p.n_local, p.block_size, p.n_repr,
                    p.topk, float(p.sm_scale), rope_inv_freq=freqs, mean_repr=p.mean_repr)


class Layer:
    """One layer's device memory plus step buffers, driven through infllm_step."""

    def __init__(self, p: F.Params, batch: int, capacity: int, chunk: int, ring: Optional[int] = None):
        self.p = p
        self.batch = batch
        self.capacity = capacity
        self.chunk = chunk
        op = oparams(p)
        self.max_units = max(1, O.partition(capacity, op).n_units)
        self.ring = ring if ring is not None else F.recommended_ring(p, chunk)
        self.mem = F.alloc_memory(p, batch, capacity, self.max_units, self.ring)
        ws = max(F.infllm_workspace_bytes(p, batch, chunk), F.infllm_workspace_bytes(p, batch, 1))
        self.ws = torch.zeros(ws, dtype=torch.uint8, device="cuda")
        dt = torch.bfloat16 if p.dtype == F.INFLLM_BF16 else torch.float32
        self.dt = dt
        self.esize = 2 if dt == torch.bfloat16 else 4
        self.out = torch.zeros((batch, p.n_q_heads, chunk, p.head_dim), dtype=dt, device="cuda")
        self.lse = torch.zeros((batch, p.n_q_heads, chunk), dtype=torch.float32, device="cuda")
        self.scores = torch.zeros((batch * p.n_kv_heads * self.max_units,), dtype=torch.float32, device="cuda")
        self.idx = torch.zeros((batch, p.n_kv_heads, max(1, p.topk)), dtype=torch.int32, device="cuda")
        self.units_built = 0

    def step(self, q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, past: int, n: int) -> None:
        """q [B][Hq][S][D], k/v [B][Hkv][S][D] device inputs for the whole sequence."""
        S, D = q.shape[2], q.shape[3]
        off = past * D * self.esize
        F.infllm_step(self.p, self.mem.struct, q.data_ptr() + off, S * D, k.data_ptr() + off,
                      v.data_ptr() + off, S * D, n, past, self.units_built, self.scores, self.idx, self.out,
                      self.chunk * D, self.lse, self.ws)
        self.units_built = O.partition(past, oparams(self.p)).n_units

    def step_mass(self, q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, past: int, n: int, decay: float,
                  mass: torch.Tensor, freq: Optional[torch.Tensor]) -> None:
        """The same step through infllm_step_mass: also the unit masses and frequency scores."""
        S, D = q.shape[2], q.shape[3]
        off = past * D * self.esize
        F.infllm_step_mass(self.p, self.mem.struct, q.data_ptr() + off, S * D, k.data_ptr() + off,
                           v.data_ptr() + off, S * D, n, past, self.units_built, self.scores, self.idx, self.out,
                           self.chunk * D, self.lse, decay, mass, freq, self.ws)
        self.units_built = O.partition(past, oparams(self.p)).n_units

    def capture(self, n: int, n_units: int) -> Dict[str, np.ndarray]:
        torch.cuda.synchronize()
        B, Hq, Hkv = self.batch, self.p.n_q_heads, self.p.n_kv_heads
        return {
            "out": host(self.out[:, :, :n]).astype(np.float64),
            # lse is written compact, [batch][Hq][n] (no head stride), also for a short last chunk
            "lse": host(self.lse.reshape(-1)[: B * Hq * n].reshape(B, Hq, n)).astype(np.float64),
            "scores": host(self.scores[: B * Hkv * n_units]).reshape(B, Hkv, n_units).astype(np.float64),
            "idx": host(self.idx).astype(np.int64),
        }


def gap_rel(scores_row: np.ndarray, k: int) -> float:
    """(s_(k) - s_(k+1)) / max(|s_(k)|, rms(row)) of the sorted row; inf when nothing is left out."""
    n = scores_row.shape[0]
    k_eff = min(k, n)
    if k_eff == 0 or k_eff == n:
        return float("inf")
    s = np.sort(scores_row)[::-1]
    scale = max(abs(s[k_eff - 1]), float(np.sqrt(np.mean(scores_row ** 2))), 1e-30)
    return float((s[k_eff - 1] - s[k_eff]) / scale)


def check_selection(gpu_row: np.ndarray, oracle_row: np.ndarray, oracle_scores: np.ndarray, k: int,
                    rel: float = 1e-3) -> bool:
    """Index sets must match exactly where the k-th/(k+1)-th gap exceeds `rel`; inside a near-tie the
    GPU's set must still be a valid top-k (every chosen unit within the tie band).  Returns True when
    the sets are identical."""
    n = oracle_scores.shape[0]
    k_eff = min(k, n)
    g = gpu_row[:k_eff]
    assert np.all(gpu_row[k_eff:] == -1)
    assert np.all(np.diff(g) > 0) and (k_eff == 0 or (g[0] >= 0 and g[-1] < n)), gpu_row
    if np.array_equal(g, oracle_row[:k_eff]):
        return True
    gr = gap_rel(oracle_scores, k)
    assert gr <= rel, f"index sets differ with gap {gr:.3g} > {rel}: gpu {g} oracle {oracle_row[:k_eff]}"
    s_sorted = np.sort(oracle_scores)[::-1]
    band = rel * max(abs(s_sorted[k_eff - 1]), float(np.sqrt(np.mean(oracle_scores ** 2))))
    assert np.all(oracle_scores[g] >= s_sorted[k_eff - 1] - band)
    return False


def conditioned_step(so: "O.StreamOracle", b: int, past: int, n: int, gpu_repr_idx: np.ndarray) -> dict:
    """The oracle's step for sequence b, conditioned on the device's unit representatives.

    Representative sets are an integer decision on r_m; where the device's set differs from the
    oracle's, it must lie inside the r_m near-tie band (the same 1e-3 rule as the lookup), and the
    oracle then scores that unit with the device's set (a conditioned oracle: scores, lookup and
    attention all follow from it).  gpu_repr_idx: [Hkv][>= n_units][r_k] offsets of sequence b.
    Returns the step dict with the conditioned scores and lookup, plus "rep_ties": units that
    differed."""
    p = so.p
    G = p.group
    nu = O.partition(past, p).n_units
    if p.mean_repr or nu == 0:
        r = so.step(b, past, n)
        r["rep_ties"] = 0
        return r
    scores = np.zeros((p.n_kv_heads, nu))
    ties = 0
    for g in range(p.n_kv_heads):
        reps = []
        for u in range(nu):
            mine = so.repr_offsets(b, g, u)
            dev_off = np.sort(np.asarray(gpu_repr_idx[g, u], dtype=np.int64))
            if not np.array_equal(mine, dev_off):
                check_selection(np.asarray(gpu_repr_idx[g, u], dtype=np.int64), mine, so.repr_scores(b, g, u),
                                p.n_repr)
                ties += 1
            reps.append(O.unit_start(u, p) + dev_off)
        qx = so.q[b, g * G:(g + 1) * G, past:past + n]
        scores[g] = O.unit_relevance(qx, so.k[b, g], np.stack(reps), p)
    sel = np.stack([O.select_units(scores[g], p) for g in range(p.n_kv_heads)])
    r = so.step(b, past, n, sel=sel)
    r["scores"] = scores
    r["rep_ties"] = ties
    return r
