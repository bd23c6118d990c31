"""Plain CPU reference for InfLLM's block-memory attention step (arXiv 2402.04617, Section 3).

TEST INFRASTRUCTURE ONLY.  This module is the oracle that the device library is
checked against.  Only the tests, the package smoke check and the benchmark's
CPU-baseline leg may import it; the product path never does.  It shares no code
with the HIP library and computes everything in float64 from the exact input
values (bf16/fp32 inputs widen to float64 without rounding).

Notation follows the paper: past length l_P, initial tokens l_I, local window
l_L, unit (block) size l_bs, representative tokens per unit r_k, units loaded per
step k_m, current tokens l_X.  For grouped-query attention the paper is silent;
the readings used here are listed with each function.

Positional remap (Section 3.2, "Positional Encoding"; Appendix "Positional
Encoding"), optional: with rotary frequencies given, q and k arrive without
positions and the oracle applies them.  Tokens beyond the local window (I and the
memory units) sit at the fixed distance l_L from every current token; L and X
keep their true positions.  Without frequencies the inputs carry their positions
already and no rotation is applied.

Every function has a pin in tests/test_oracle_pins.py (brute force, closed
forms, special cases reducing to library attention, invariants).
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np


@dataclasses.dataclass(frozen=True)
class Params:
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    n_init: int       # l_I
    n_local: int      # l_L
    block_size: int   # l_bs
    n_repr: int       # r_k
    topk: int         # k_m
    sm_scale: float = 1.0
    # Rotary angular frequencies theta_i (radians per position) of the D/2 dimension
    # pairs (2i, 2i+1) for the positional remap; None: positions pre-applied.
    rope_inv_freq: Optional[Tuple[float, ...]] = None
    # Units represented by the mean of their keys (the "Mean Repr" alternative of
    # Section 4) instead of r_k representative tokens.
    mean_repr: bool = False

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads


@dataclasses.dataclass(frozen=True)
class Partition:
    n_init: int       # |I| (fewer than l_I while the past is short)
    n_units: int      # whole units formed from the evicted tokens E
    local_begin: int  # first position of L; L = [local_begin, l_P)


def rotate(x: np.ndarray, positions, inv_freq: Sequence[float]) -> np.ndarray:
    """Rotary position encoding R(p) x: dimension pair i = (2i, 2i+1) turned by the angle p * theta_i.

    x: [..., S, D] (or [..., D] with a scalar position); positions: [S] or a scalar.
    The pairing is the interleaved one; a model trained with the half-split
    pairing (i, i + D/2) is the same model after one fixed permutation of the
    head dimensions applied to q and k alike, which leaves every q . k unchanged.
    Angles are formed in float64.  Returns float64.
    """
    x = np.asarray(x, dtype=np.float64)
    ang = np.multiply.outer(np.asarray(positions, dtype=np.float64), np.asarray(inv_freq, dtype=np.float64))
    c, s = np.cos(ang), np.sin(ang)
    out = np.empty_like(x)
    out[..., 0::2] = x[..., 0::2] * c - x[..., 1::2] * s
    out[..., 1::2] = x[..., 0::2] * s + x[..., 1::2] * c
    return out


def partition(past_len: int, p: Params) -> Partition:
    """Split of the past key-values P (Section 3.1, "Overall Framework").

    I = the first l_I tokens, L = the last l_L tokens, E = the tokens between.
    E is cut into consecutive units of l_bs tokens (Section 3.2).  Reading where
    the paper is silent: only whole units are formed; a trailing remainder of
    fewer than l_bs evicted tokens stays attended as part of L, so L holds
    between l_L and l_L + l_bs - 1 tokens once eviction has begun.
    """
    n_init = min(p.n_init, past_len)
    evicted = past_len - p.n_init - p.n_local
    n_units = evicted // p.block_size if evicted > 0 else 0
    return Partition(n_init, n_units, n_init + n_units * p.block_size)


def unit_start(unit: int, p: Params) -> int:
    """First position of memory unit `unit`; units tile E starting right after I (Section 3.2)."""
    return p.n_init + unit * p.block_size


def representative_scores(q_group: np.ndarray, k_head: np.ndarray, unit: int, p: Params,
                          q_summed: Optional[np.ndarray] = None) -> np.ndarray:
    """Representative score r_m of every token m of one unit (Section 3.2, "Block-Level Memory Units").

    r_m = (1/l_L) * sum_{j=1..l_L} q_{m+j} . k_m : the mean dot product of token m's
    key with the queries of the l_L tokens that follow it.  GQA reading: the
    query side is also averaged over the G query heads that share the kv head, so
    r_m = 1/(l_L*G) * sum_h sum_j q^h_{m+j} . k_m.

    q_group: [G][S][D] queries of the group's heads (positions up to m + l_L must
    exist); k_head: [S][D] keys of the kv head.  q_summed, if given, is the same
    group's query sum sum_h q^h as float64 [S][D], precomputed once per sequence
    (q_group then only supplies G).  With the positional remap, q_{m+j} and k_m
    are rotated to their own positions (the local window keeps true distances).
    Returns float64 [l_bs].
    """
    G = q_group.shape[0]
    m0 = unit_start(unit, p)
    lbs, lL = p.block_size, p.n_local
    # Window queries of all tokens of the unit: positions m0+1 .. m0+l_bs-1+l_L,
    # summed over the group's heads (sum_h q^h . k = (sum_h q^h) . k).
    if q_summed is None:
        qw = np.asarray(q_group[:, m0 + 1: m0 + lbs + lL, :], dtype=np.float64).sum(axis=0)
    else:
        qw = q_summed[m0 + 1: m0 + lbs + lL]
    ku = np.asarray(k_head[m0: m0 + lbs, :], dtype=np.float64)
    if p.rope_inv_freq is not None:
        # Positional remap: while token m is in the local window its queries see it
        # at the true distance j, so both sides keep their own positions.
        qw = rotate(qw, np.arange(m0 + 1, m0 + lbs + lL), p.rope_inv_freq)
        ku = rotate(ku, np.arange(m0, m0 + lbs), p.rope_inv_freq)
    dots = ku @ qw.T  # dots[t, a] = k_{m0+t} . q~_{m0+1+a}
    r = np.empty(lbs)
    for t in range(lbs):
        # j = 1..l_L  <->  window index a = t + j - 1 = t .. t + l_L - 1
        r[t] = dots[t, t: t + lL].sum()
    return r / (lL * G)


def top_indices(values: np.ndarray, count: int) -> np.ndarray:
    """The `count` largest entries of `values`, returned as ascending indices.

    Ties go to the lower index (reading: the paper does not say).  Done as
    repeated arg-max, which returns the first (lowest) index among equal maxima.
    """
    vals = np.array(values, dtype=np.float64, copy=True)
    count = min(count, vals.shape[0])
    chosen = []
    for _ in range(count):
        i = int(np.argmax(vals))
        chosen.append(i)
        vals[i] = -np.inf
    return np.array(sorted(chosen), dtype=np.int64)


def representatives(r: np.ndarray, p: Params) -> np.ndarray:
    """R(B): the r_k tokens of a unit with the highest r_m (Section 3.2), as ascending offsets in the unit."""
    return top_indices(r, p.n_repr)


def unit_relevance(q_chunk_group: np.ndarray, k_head: np.ndarray, rep_pos: np.ndarray,
                   p: Optional[Params] = None) -> np.ndarray:
    """sim(X, B) = sum_{i=1..l_X} sum_{j=1..r_k} q_{i+l_P} . k^B_{b_j} for every unit B (Section 3.2).

    No normalisation (the formula has none).  GQA reading: one score per kv head,
    summed over the query heads of its group as well.  With the positional remap
    (p given with frequencies) every memory key sits at distance l_L from every
    current token: the queries are rotated by R(l_L), the keys not at all.
    q_chunk_group: [G][l_X][D]; rep_pos: [n_units][r_k] absolute key positions.
    Returns float64 [n_units].
    """
    if rep_pos.shape[0] == 0:
        return np.zeros(0)
    D = k_head.shape[1]
    qx = np.asarray(q_chunk_group, dtype=np.float64).reshape(-1, D)        # every (head, i)
    if p is not None and p.rope_inv_freq is not None:
        qx = rotate(qx, float(p.n_local), p.rope_inv_freq)
    keys = np.asarray(k_head[rep_pos.reshape(-1)], dtype=np.float64)        # every (unit, j)
    dots = qx @ keys.T                                                        # all q_i . k_{b_j}
    return dots.reshape(qx.shape[0], rep_pos.shape[0], rep_pos.shape[1]).sum(axis=(0, 2))


def mean_relevance(q_chunk_group: np.ndarray, k_head: np.ndarray, n_units: int, p: Params) -> np.ndarray:
    """sim(X, B) = sum_{i=1..l_X} q_{i+l_P} . mean_{j=1..l_bs} k^B_j for every unit B: the unit
    represented by the mean of its keys (the "Mean Repr" alternative evaluated in Section 4),
    summed over the query heads of the group like unit_relevance, and with the positional
    remap taken the same way.  Returns float64 [n_units]."""
    if n_units == 0:
        return np.zeros(0)
    pos = np.stack([np.arange(unit_start(u, p), unit_start(u, p) + p.block_size) for u in range(n_units)])
    return unit_relevance(q_chunk_group, k_head, pos, p) / p.block_size


def select_units(sim: np.ndarray, p: Params, k: Optional[int] = None) -> np.ndarray:
    """Memory lookup f(X, E): the k_m units with the highest sim (Section 3.2, "memory lookup").

    Returns k_m entries: the min(k_m, n_units) chosen unit ids ascending, then -1.
    """
    k = p.topk if k is None else k
    out = np.full(k, -1, dtype=np.int64)
    chosen = top_indices(sim, k) if k > 0 else np.zeros(0, dtype=np.int64)
    out[: chosen.shape[0]] = chosen
    return out


def context_positions(past_len: int, sel: np.ndarray, p: Params) -> np.ndarray:
    """Positions of the current key-value cache C = Concat(I, f(X, E), L) (Section 3.1)."""
    part = partition(past_len, p)
    pos = [np.arange(part.n_init)]
    for b in sel:
        if b >= 0:
            s = unit_start(int(b), p)
            pos.append(np.arange(s, s + p.block_size))
    pos.append(np.arange(part.local_begin, past_len))
    return np.concatenate(pos).astype(np.int64)


def attention_logits(q_chunk: np.ndarray, k: np.ndarray, past_len: int, sel_g: np.ndarray, p: Params,
                     g: int) -> Tuple[np.ndarray, np.ndarray]:
    """Logits of kv group g's G query heads over Concat(C, X) (Section 3.1).

    z[hh][i][t] = sm_scale * q . k for key t of C (I, the looked-up units in the
    order of sel_g, L) followed by the current tokens X, -inf where X is causally
    hidden (query i sees X positions up to its own).  Under the positional remap
    (Section 3.2) I and the units are met by the query turned by R(l_L) with the
    key unrotated, L and X at their true positions.
    Returns z float64 [G][l_X][|C| + l_X] and the keys' positions [|C| + l_X].
    """
    nq = q_chunk.shape[1]
    G = p.group
    causal = np.tril(np.ones((nq, nq), dtype=bool))
    remap = p.rope_inv_freq is not None
    part = partition(past_len, p)
    pos = context_positions(past_len, sel_g, p)
    kc = np.asarray(k[g, pos], dtype=np.float64)
    kx = np.asarray(k[g, past_len: past_len + nq], dtype=np.float64)
    n_mem = pos.shape[0] - (past_len - part.local_begin)
    if remap:
        kc[n_mem:] = rotate(kc[n_mem:], pos[n_mem:], p.rope_inv_freq)
        kx = rotate(kx, np.arange(past_len, past_len + nq), p.rope_inv_freq)
    z = np.empty((G, nq, pos.shape[0] + nq))
    for hh in range(G):
        qh = np.asarray(q_chunk[g * G + hh], dtype=np.float64)
        if remap:
            q_mem = rotate(qh, float(p.n_local), p.rope_inv_freq)
            q_loc = rotate(qh, np.arange(past_len, past_len + nq), p.rope_inv_freq)
            zc = np.concatenate([q_mem @ kc[:n_mem].T, q_loc @ kc[n_mem:].T], axis=1)
            zx = q_loc @ kx.T
        else:
            zc, zx = qh @ kc.T, qh @ kx.T
        z[hh] = np.concatenate([p.sm_scale * zc, np.where(causal, p.sm_scale * zx, -np.inf)], axis=1)
    return z, np.concatenate([pos, np.arange(past_len, past_len + nq)])


def attend(q_chunk: np.ndarray, k: np.ndarray, v: np.ndarray, past_len: int,
           sel: np.ndarray, p: Params) -> Tuple[np.ndarray, np.ndarray]:
    """O = Attn[Q X, Concat(C_k, K X), Concat(C_v, V X)] (Section 3.1).

    One softmax per query over the union of C and the current tokens X, causal
    inside X (query i sees X positions up to its own).  Logits are
    sm_scale * q . k; sm_scale = 1 when the inputs come pre-scaled.
    q_chunk: [Hq][l_X][D]; k, v: [Hkv][S][D]; sel: [Hkv][k] unit ids (-1 = none).
    Returns O float64 [Hq][l_X][D] and natural-log lse [Hq][l_X].
    """
    Hq, nq, D = q_chunk.shape
    G = p.group
    O = np.empty((Hq, nq, D))
    lse = np.empty((Hq, nq))
    for g in range(p.n_kv_heads):
        z, keys = attention_logits(q_chunk, k, past_len, sel[g], p, g)
        vk = np.asarray(v[g, keys], dtype=np.float64)
        for hh in range(G):
            zmax = z[hh].max(axis=1, keepdims=True)
            w = np.exp(z[hh] - zmax)
            s = w.sum(axis=1, keepdims=True)
            O[g * G + hh] = (w / s) @ vk
            lse[g * G + hh] = (zmax + np.log(s))[:, 0]
    return O, lse


def unit_mass(q_chunk: np.ndarray, k: np.ndarray, past_len: int, sel: np.ndarray, p: Params) -> np.ndarray:
    """Attention mass of each looked-up unit (Section 3.2, "Cache Management"; the
    appendix's frequency score adds it up).

    The attention score of a key for a query is its softmax probability in the
    step's attention (the logits and key set of `attend`); a unit's mass sums it
    over the unit's l_bs keys, the chunk's queries and the G query heads of the
    kv group.  sel: [Hkv][k] unit ids (-1 = none, mass 0).  Returns float64 [Hkv][k].
    """
    n_units = partition(past_len, p).n_units
    mass = np.zeros(np.shape(sel), dtype=np.float64)
    for g in range(p.n_kv_heads):
        z, keys = attention_logits(q_chunk, k, past_len, sel[g], p, g)
        prob = np.exp(z - z.max(axis=2, keepdims=True))
        prob /= prob.sum(axis=2, keepdims=True)
        for j, b in enumerate(sel[g]):
            if 0 <= b < n_units:
                s0 = unit_start(int(b), p)
                in_unit = (keys >= s0) & (keys < s0 + p.block_size)
                mass[g, j] = prob[:, :, in_unit].sum()
    return mass


def frequency_update(freq: np.ndarray, sel: np.ndarray, mass: np.ndarray, n_units: int,
                     decay: float) -> np.ndarray:
    """The frequency score after one step (appendix on cache management):
    s_b <- s_b * d + (mass of b this step), for every built unit b < n_units, the
    mass being 0 for a unit that was not looked up.  freq: [Hkv][>= n_units]."""
    f = np.array(freq, dtype=np.float64, copy=True)
    f[:, :n_units] *= decay
    for g in range(f.shape[0]):
        for j, b in enumerate(sel[g]):
            if 0 <= b < n_units:
                f[g, b] += mass[g, j]
    return f


def lse_merge(outs: Sequence[np.ndarray], lses: Sequence[np.ndarray]) -> Tuple[np.ndarray, np.ndarray]:
    """Combine softmax-normalised partial attentions over disjoint key sets into the single softmax.

    LSE = log sum_s exp(lse_s);  O = sum_s exp(lse_s - LSE) O_s.  A part with no
    keys has lse_s = -inf and weight 0.  This is what the single Attn of
    Section 3.1 equals when its key set is split.
    """
    L = np.stack([np.asarray(x, dtype=np.float64) for x in lses])
    M = L.max(axis=0)
    Ms = np.where(np.isfinite(M), M, 0.0)
    w = np.exp(L - Ms)
    tot = w.sum(axis=0)
    lse = Ms + np.log(tot)
    O = sum(w[s][..., None] * np.asarray(outs[s], dtype=np.float64) for s in range(len(outs)))
    return O / tot[..., None], lse


class StreamOracle:
    """Runs the per-step lookup + attention of one layer over a stream of steps.

    q: [B][Hq][S][D], k, v: [B][Hkv][S][D] (float32 or float64 arrays holding the
    exact input values).  Units are a pure function of Q and K, so each unit's
    representatives are computed once on first use and cached; any step can be
    evaluated alone.
    """

    def __init__(self, q: np.ndarray, k: np.ndarray, v: np.ndarray, p: Params):
        self.q, self.k, self.v, self.p = q, k, v, p
        self._rep: Dict[Tuple[int, int, int], np.ndarray] = {}
        self._rscore: Dict[Tuple[int, int, int], np.ndarray] = {}
        self._qsum: Dict[Tuple[int, int], np.ndarray] = {}

    def group_query_sum(self, b: int, g: int) -> Optional[np.ndarray]:
        """sum_h q^h over kv head g's query group, float64 [S][D] (cached; None for very long inputs)."""
        if self.q.shape[2] > (1 << 18):
            return None
        if (b, g) not in self._qsum:
            G = self.p.group
            self._qsum[(b, g)] = np.asarray(self.q[b, g * G:(g + 1) * G], dtype=np.float64).sum(axis=0)
        return self._qsum[(b, g)]

    def repr_scores(self, b: int, g: int, unit: int) -> np.ndarray:
        key = (b, g, unit)
        if key not in self._rscore:
            G = self.p.group
            self._rscore[key] = representative_scores(self.q[b, g * G:(g + 1) * G], self.k[b, g], unit, self.p,
                                                      self.group_query_sum(b, g))
        return self._rscore[key]

    def repr_offsets(self, b: int, g: int, unit: int) -> np.ndarray:
        key = (b, g, unit)
        if key not in self._rep:
            self._rep[key] = representatives(self.repr_scores(b, g, unit), self.p)
        return self._rep[key]

    def rep_positions(self, b: int, g: int, n_units: int) -> np.ndarray:
        if n_units == 0:
            return np.zeros((0, self.p.n_repr), dtype=np.int64)
        return np.stack([unit_start(u, self.p) + self.repr_offsets(b, g, u) for u in range(n_units)])

    def scores(self, b: int, past_len: int, n_q: int) -> np.ndarray:
        """sim for every (kv head, unit) at this step: float64 [Hkv][n_units]."""
        p = self.p
        G = p.group
        nu = partition(past_len, p).n_units
        out = np.zeros((p.n_kv_heads, nu))
        for g in range(p.n_kv_heads):
            qx = self.q[b, g * G:(g + 1) * G, past_len:past_len + n_q]
            if p.mean_repr:
                out[g] = mean_relevance(qx, self.k[b, g], nu, p)
            else:
                out[g] = unit_relevance(qx, self.k[b, g], self.rep_positions(b, g, nu), p)
        return out

    def step(self, b: int, past_len: int, n_q: int, sel: Optional[np.ndarray] = None) -> dict:
        """One step of sequence b: scores, selection, output and lse.

        `sel` overrides the lookup (used by tests that fix the selection).
        """
        p = self.p
        sim = self.scores(b, past_len, n_q)
        if sel is None:
            sel = np.stack([select_units(sim[g], p) for g in range(p.n_kv_heads)])
        qx = self.q[b, :, past_len:past_len + n_q]
        O, lse = attend(qx, self.k[b], self.v[b], past_len, sel, p)
        return {"scores": sim, "idx": sel, "out": O, "lse": lse,
                "n_units": partition(past_len, p).n_units}
