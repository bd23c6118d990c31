"""Checks that pin the CPU oracle to things other than itself.

Each check raises AssertionError on failure.  They are plain functions so that
tests/test_oracle_pins.py can run them against the oracle as written and also
against deliberately broken copies of it (to show each plausible mistake is
caught by at least one pin).

Independent references used here: hand-worked values from the paper's formulas
(tests/golden/hand_worked_tiny.yaml), brute-force pure-Python loops on tiny
inputs, algebraic identities (prefix differences, linearity), and PyTorch's
scaled_dot_product_attention in float64 on the CPU as the textbook softmax
attention it must reduce to in special cases.
"""
from __future__ import annotations

import math
import os

import numpy as np
import torch
import yaml

from oracle import infllm_oracle as O

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _params(**kw) -> O.Params:
    base = dict(n_q_heads=4, n_kv_heads=2, head_dim=8, n_init=4, n_local=16, block_size=8,
                n_repr=2, topk=2, sm_scale=1.0)
    base.update(kw)
    return O.Params(**base)


def _rand_qkv(rng, p: O.Params, S: int, B: int = 1):
    q = rng.standard_normal((B, p.n_q_heads, S, p.head_dim))
    k = rng.standard_normal((B, p.n_kv_heads, S, p.head_dim))
    v = rng.standard_normal((B, p.n_kv_heads, S, p.head_dim))
    return q, k, v


# --------------------------------------------------------------------------- P1
def brute_partition(past_len: int, l_I: int, l_L: int, l_bs: int):
    """Label positions 1..l_P as the paper writes them (1-based): I = [1, l_I],
    E = [l_I+1, l_P-l_L], L = the rest; E tokens of an incomplete trailing unit
    stay in L.  Returns (|I|, n_units, first L position 0-based, labels)."""
    labels = []
    for pos in range(1, past_len + 1):
        if pos <= l_I:
            labels.append(("I", None))
        elif pos <= past_len - l_L:
            labels.append(("E", (pos - l_I - 1) // l_bs))
        else:
            labels.append(("L", None))
    counts = {}
    for lab, u in labels:
        if lab == "E":
            counts[u] = counts.get(u, 0) + 1
    whole = {u for u, c in counts.items() if c == l_bs}
    labels = [(lab, u) if lab != "E" or u in whole else ("L", None) for lab, u in labels]
    n_i = sum(1 for lab, _ in labels if lab == "I")
    first_l = next((i for i, (lab, _) in enumerate(labels) if lab == "L"), past_len)
    return n_i, len(whole), first_l, labels


def check_partition():
    for l_I in (0, 1, 4, 16):
        for l_L in (1, 3, 16):
            for l_bs in (1, 2, 5, 8):
                p = _params(n_init=l_I, n_local=l_L, block_size=l_bs)
                for past in range(0, l_I + l_L + 4 * l_bs + 3):
                    part = O.partition(past, p)
                    n_i, n_u, first_l, labels = brute_partition(past, l_I, l_L, l_bs)
                    assert (part.n_init, part.n_units, part.local_begin) == (n_i, n_u, first_l), \
                        (past, l_I, l_L, l_bs, part, (n_i, n_u, first_l))
                    # L is contiguous up to l_P and sizes add up
                    assert all(lab == "L" for lab, _ in labels[first_l:])
                    assert part.n_init + part.n_units * l_bs + (past - part.local_begin) == past
                    if part.n_units:
                        assert l_L <= past - part.local_begin < l_L + l_bs


# --------------------------------------------------------------------------- P2
def brute_repr_scores(q, k, g, unit, p):
    """Literal r_m with pure-Python loops: 1/(l_L G) sum_h sum_{j=1..l_L} sum_d q^h_{m+j,d} k_{m,d}."""
    G = p.group
    m0 = p.n_init + unit * p.block_size
    out = []
    for m in range(m0, m0 + p.block_size):
        tot = 0.0
        for h in range(g * G, (g + 1) * G):
            for j in range(1, p.n_local + 1):
                for d in range(p.head_dim):
                    tot += float(q[h, m + j, d]) * float(k[g, m, d])
        out.append(tot / (p.n_local * G))
    return np.array(out)


def check_repr_scores_bruteforce():
    rng = np.random.default_rng(11)
    p = _params(n_q_heads=4, n_kv_heads=2, head_dim=3, n_init=2, n_local=3, block_size=4)
    q, k, _ = _rand_qkv(rng, p, S=2 + 3 * 4 + 3 + 1)
    for g in range(2):
        for unit in range(3):
            got = O.representative_scores(q[0, g * 2:(g + 1) * 2], k[0, g], unit, p)
            ref = brute_repr_scores(q[0], k[0], g, unit, p)
            assert np.allclose(got, ref, rtol=1e-12, atol=1e-12), (g, unit, got, ref)


def check_repr_scores_prefix_identity():
    """W_m = sum_{j=1..l_L} q~_{m+j} = Pi_{m+l_L+1} - Pi_{m+1} with Pi_t = sum_{p<t} q~_p."""
    rng = np.random.default_rng(12)
    p = _params(n_q_heads=8, n_kv_heads=2, head_dim=16, n_init=3, n_local=64, block_size=16)
    S = 3 + 6 * 16 + 64 + 1
    q, k, _ = _rand_qkv(rng, p, S)
    G = p.group
    for g in range(2):
        qt = q[0, g * G:(g + 1) * G].sum(axis=0)
        Pi = np.concatenate([np.zeros((1, p.head_dim)), np.cumsum(qt, axis=0)])
        for unit in range(6):
            m = p.n_init + unit * p.block_size + np.arange(p.block_size)
            W = Pi[m + p.n_local + 1] - Pi[m + 1]
            ref = (W * k[0, g, m]).sum(axis=1) / (p.n_local * G)
            got = O.representative_scores(q[0, g * G:(g + 1) * G], k[0, g], unit, p)
            assert np.allclose(got, ref, rtol=1e-12, atol=1e-12)


def check_repr_scores_presummed_queries():
    """Passing the group's query sum precomputed gives the same r_m as summing per call."""
    rng = np.random.default_rng(23)
    p = _params(n_q_heads=6, n_kv_heads=2, head_dim=5, n_init=2, n_local=7, block_size=4)
    q, k, _ = _rand_qkv(rng, p, S=2 + 5 * 4 + 8)
    for g in range(2):
        qs = q[0, 3 * g:3 * g + 3].sum(axis=0)
        for unit in range(5):
            a = O.representative_scores(q[0, 3 * g:3 * g + 3], k[0, g], unit, p)
            b = O.representative_scores(q[0, 3 * g:3 * g + 3], k[0, g], unit, p, qs)
            assert np.allclose(a, b, rtol=1e-13, atol=1e-13)


def check_repr_scores_window_one():
    """l_L = 1: r_m is the group-mean of q_{m+1} . k_m."""
    rng = np.random.default_rng(13)
    p = _params(n_q_heads=6, n_kv_heads=2, head_dim=5, n_init=1, n_local=1, block_size=3)
    q, k, _ = _rand_qkv(rng, p, S=1 + 4 * 3 + 2)
    G = p.group
    for g in range(2):
        for unit in range(4):
            m = p.n_init + unit * 3 + np.arange(3)
            ref = np.einsum("hmd,md->m", q[0][g * G:(g + 1) * G][:, m + 1], k[0, g, m]) / G
            got = O.representative_scores(q[0, g * G:(g + 1) * G], k[0, g], unit, p)
            assert np.allclose(got, ref, rtol=1e-13, atol=1e-13)


def check_repr_scores_window_support():
    """Only queries at m+1..m+l_L matter: perturbing q at position m (or past the last
    window) leaves r_m unchanged; perturbing q_{m+l_L} changes it."""
    rng = np.random.default_rng(14)
    p = _params(n_q_heads=2, n_kv_heads=1, head_dim=4, n_init=2, n_local=5, block_size=4)
    q, k, _ = _rand_qkv(rng, p, S=40)
    base = O.representative_scores(q[0], k[0, 0], 1, p)
    m0 = p.n_init + 1 * p.block_size
    for pos, expect_change in ((m0, False), (m0 + p.block_size - 1 + p.n_local + 1, False),
                               (m0 + p.n_local, True), (m0 + 1, True)):
        q2 = q.copy()
        q2[0, :, pos] += 3.0
        r2 = O.representative_scores(q2[0], k[0, 0], 1, p)
        changed = not np.allclose(r2, base, rtol=0, atol=1e-14)
        assert changed == expect_change, (pos, expect_change)
    # first token's score moves with its last window query, not the next one
    q3 = q.copy()
    q3[0, :, m0 + p.n_local] += 3.0
    r3 = O.representative_scores(q3[0], k[0, 0], 1, p)
    assert not np.isclose(r3[0], base[0])
    q4 = q.copy()
    q4[0, :, m0 + p.n_local + 1] += 3.0
    r4 = O.representative_scores(q4[0], k[0, 0], 1, p)
    assert np.isclose(r4[0], base[0], rtol=0, atol=1e-14)


# --------------------------------------------------------------------------- P3
def brute_topk(values, k):
    order = sorted(range(len(values)), key=lambda i: (-float(values[i]), i))
    return sorted(order[:k])


def check_top_indices():
    rng = np.random.default_rng(15)
    for n in (0, 1, 2, 5, 17, 100):
        for kind in ("gauss", "ties", "const", "neg"):
            if kind == "gauss":
                vals = rng.standard_normal(n)
            elif kind == "ties":
                vals = rng.integers(0, 4, n).astype(float)
            elif kind == "const":
                vals = np.full(n, 0.5)
            else:
                vals = -np.abs(rng.standard_normal(n)) - 1.0
            for k in sorted({0, 1, 3, n, n + 2}):
                got = list(O.top_indices(vals, k))
                assert got == brute_topk(vals, k), (n, kind, k, got)


# --------------------------------------------------------------------------- P4/P5
def check_unit_relevance_linearity():
    """sim = sum_i sum_j q_i . k_{b_j} = (sum_i q_i) . (sum_j k_{b_j})."""
    rng = np.random.default_rng(16)
    G, nq, D, S = 3, 7, 9, 60
    q = rng.standard_normal((G, nq, D))
    k = rng.standard_normal((S, D))
    rep = np.stack([np.sort(rng.choice(S, 4, replace=False)) for _ in range(10)])
    got = O.unit_relevance(q, k, rep)
    ref = np.array([q.sum(axis=(0, 1)) @ k[r].sum(axis=0) for r in rep])
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-12)
    # literal loops on a smaller slice
    lit = []
    for r in rep[:3]:
        t = 0.0
        for h in range(G):
            for i in range(nq):
                for j in r:
                    t += sum(float(q[h, i, d]) * float(k[j, d]) for d in range(D))
        lit.append(t)
    assert np.allclose(got[:3], lit, rtol=1e-12, atol=1e-12)


def check_mean_repr_special_case():
    """r_k = l_bs makes every token representative: sim(X,B) = l_bs * Qbar . mean(K_B)
    (the paper's "Mean Repr" representation scaled by l_bs), independent of r_m."""
    rng = np.random.default_rng(17)
    p = _params(n_q_heads=4, n_kv_heads=2, head_dim=6, n_init=3, n_local=8, block_size=4,
                n_repr=4, topk=2)
    S = 60
    q, k, v = _rand_qkv(rng, p, S)
    so = O.StreamOracle(q, k, v, p)
    past, nq = 40, 5
    sim = so.scores(0, past, nq)
    nu = (past - p.n_init - p.n_local) // p.block_size
    assert sim.shape == (2, nu)
    for g in range(2):
        qbar = q[0, g * 2:(g + 1) * 2, past:past + nq].sum(axis=(0, 1))
        for u in range(nu):
            s = p.n_init + u * p.block_size
            ref = p.block_size * qbar @ k[0, g, s:s + p.block_size].mean(axis=0)
            assert math.isclose(sim[g, u], ref, rel_tol=1e-12, abs_tol=1e-12)


# --------------------------------------------------------------------------- P6-P9
def _sdpa(q, k, v, mask, scale):
    """float64 textbook attention from PyTorch; q [H][n][D], k/v [H][S][D], mask [H or 1][n][S] (True = attend).
    Returns O and lse (lse via logsumexp of the masked logits)."""
    qt, kt, vt = (torch.from_numpy(np.ascontiguousarray(x)).double() for x in (q, k, v))
    mt = torch.from_numpy(mask)
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mt, scale=scale)
    z = torch.matmul(qt, kt.transpose(-1, -2)) * scale
    z = z.masked_fill(~mt, float("-inf"))
    return o.numpy(), torch.logsumexp(z, dim=-1).numpy()


def _expand(kv, G):
    return np.repeat(kv, G, axis=0)


def check_full_attention_when_everything_selected():
    """k_m >= n_units at every step: InfLLM attends every past token, i.e. causal attention."""
    rng = np.random.default_rng(18)
    p = _params(n_q_heads=4, n_kv_heads=2, head_dim=8, n_init=3, n_local=8, block_size=4,
                n_repr=2, topk=100, sm_scale=0.7)
    S, chunk = 64, 6
    q, k, v = _rand_qkv(rng, p, S)
    mask = np.tril(np.ones((S, S), dtype=bool))[None]
    ref_o, ref_l = _sdpa(q[0], _expand(k[0], 2), _expand(v[0], 2), mask, 0.7)
    so = O.StreamOracle(q, k, v, p)
    for past in range(0, S, chunk):
        nq = min(chunk, S - past)
        r = so.step(0, past, nq)
        assert np.allclose(r["out"], ref_o[:, past:past + nq], rtol=1e-12, atol=1e-12), past
        assert np.allclose(r["lse"], ref_l[:, past:past + nq], rtol=1e-12, atol=1e-12), past


def check_full_attention_when_window_covers():
    """l_L >= S: nothing is ever evicted, so the result is causal attention for any k_m."""
    rng = np.random.default_rng(19)
    p = _params(n_q_heads=2, n_kv_heads=1, head_dim=8, n_init=2, n_local=64, block_size=4,
                n_repr=1, topk=0)
    S = 40
    q, k, v = _rand_qkv(rng, p, S)
    mask = np.tril(np.ones((S, S), dtype=bool))[None]
    ref_o, ref_l = _sdpa(q[0], _expand(k[0], 2), _expand(v[0], 2), mask, 1.0)
    so = O.StreamOracle(q, k, v, p)
    for past in (0, 7, 33):
        r = so.step(0, past, 7 if past < 33 else 7)
        assert np.allclose(r["out"], ref_o[:, past:past + 7], rtol=1e-12, atol=1e-12)
        assert np.allclose(r["lse"], ref_l[:, past:past + 7], rtol=1e-12, atol=1e-12)


def _visible_mask(past, nq, S, p, sel_g):
    """Mask from the brute-force labelling: key t is visible to query i iff t is in I, in a
    selected whole unit, in L, or in X at or before the query."""
    _, _, _, labels = brute_partition(past, p.n_init, p.n_local, p.block_size)
    m = np.zeros((nq, S), dtype=bool)
    for t, (lab, u) in enumerate(labels):
        if lab in ("I", "L") or (lab == "E" and u in set(int(x) for x in sel_g if x >= 0)):
            m[:, t] = True
    for i in range(nq):
        m[i, past:past + i + 1] = True
    return m


def check_streaming_llm_when_no_lookup():
    """k_m = 0 (f returns the empty set): initial tokens + local window + causal X,
    the LM-Infinite / StreamingLLM pattern the paper says InfLLM degenerates to."""
    rng = np.random.default_rng(20)
    p = _params(n_q_heads=4, n_kv_heads=2, head_dim=8, n_init=3, n_local=9, block_size=4,
                n_repr=2, topk=0, sm_scale=0.9)
    S = 72
    q, k, v = _rand_qkv(rng, p, S)
    so = O.StreamOracle(q, k, v, p)
    for past, nq in ((0, 5), (11, 5), (30, 8), (55, 1), (63, 9)):
        r = so.step(0, past, nq)
        for g in range(2):
            mask = _visible_mask(past, nq, S, p, [])[None]
            o, l = _sdpa(q[0, 2 * g:2 * g + 2, past:past + nq], k[0, g:g + 1].repeat(2, 0),
                         v[0, g:g + 1].repeat(2, 0), mask, 0.9)
            assert np.allclose(r["out"][2 * g:2 * g + 2], o, rtol=1e-12, atol=1e-12), (past, g)
            assert np.allclose(r["lse"][2 * g:2 * g + 2], l, rtol=1e-12, atol=1e-12), (past, g)


def check_sparse_equals_masked_dense():
    """General case: gathering I, the selected units, L and causal X equals dense attention
    over all l_P + l_X keys masked to that set."""
    rng = np.random.default_rng(21)
    p = _params(n_q_heads=6, n_kv_heads=2, head_dim=8, n_init=2, n_local=7, block_size=3,
                n_repr=1, topk=3, sm_scale=1.3)
    S = 80
    q, k, v = _rand_qkv(rng, p, S)
    for past, nq in ((25, 6), (50, 4), (70, 10)):
        nu = O.partition(past, p).n_units
        sel = np.full((2, 3), -1)
        for g in range(2):
            c = np.sort(rng.choice(nu, min(3, nu), replace=False))
            sel[g, :c.size] = c
        out, lse = O.attend(q[0, :, past:past + nq], k[0], v[0], past, sel, p)
        for g in range(2):
            mask = _visible_mask(past, nq, S, p, sel[g])[None]
            o, l = _sdpa(q[0, 3 * g:3 * g + 3, past:past + nq], k[0, g:g + 1].repeat(3, 0),
                         v[0, g:g + 1].repeat(3, 0), mask, 1.3)
            assert np.allclose(out[3 * g:3 * g + 3], o, rtol=1e-12, atol=1e-12), (past, g)
            assert np.allclose(lse[3 * g:3 * g + 3], l, rtol=1e-12, atol=1e-12), (past, g)


def check_lse_merge():
    """Any split of the key set into parts (one of them empty), each softmax-normalised,
    merges back to the single softmax over all keys."""
    rng = np.random.default_rng(22)
    n, S, D = 5, 40, 6
    q = rng.standard_normal((1, n, D))
    k = rng.standard_normal((1, S, D)) * 2
    v = rng.standard_normal((1, S, D))
    full_mask = np.ones((1, n, S), dtype=bool)
    ref_o, ref_l = _sdpa(q, k, v, full_mask, 1.0)
    cuts = [0, 3, 3, 17, 29, 40]  # includes an empty part [3, 3)
    outs, lses = [], []
    for a, b in zip(cuts[:-1], cuts[1:]):
        if a == b:
            outs.append(np.zeros((1, n, D)))
            lses.append(np.full((1, n), -np.inf))
            continue
        o, l = _sdpa(q, k[:, a:b], v[:, a:b], np.ones((1, n, b - a), dtype=bool), 1.0)
        outs.append(o)
        lses.append(l)
    mo, ml = O.lse_merge(outs, lses)
    assert np.allclose(mo, ref_o, rtol=1e-13, atol=1e-13)
    assert np.allclose(ml, ref_l, rtol=1e-13, atol=1e-13)


# --------------------------------------------------------------------------- positional remap
def _rot_complex(x, pos, freqs):
    """R(p) x written as complex arithmetic: pair (x_2i, x_2i+1) is the number
    x_2i + i x_2i+1, multiplied by e^{i p theta_i}.  pos: scalar or one per row."""
    x = np.asarray(x, float)
    z = (x[..., 0::2] + 1j * x[..., 1::2]) * np.exp(1j * np.multiply.outer(np.asarray(pos, float), freqs))
    out = np.empty(x.shape)
    out[..., 0::2] = z.real
    out[..., 1::2] = z.imag
    return out


def _rope_params(**kw):
    rng = np.random.default_rng(kw.pop("seed", 30))
    p = _params(**kw)
    freqs = tuple(float(f) for f in rng.uniform(0.05, 1.5, p.head_dim // 2))
    return O.Params(**{**p.__dict__, "rope_inv_freq": freqs})


def check_rotation_is_complex_multiplication():
    """The rotary map against complex multiplication, at small and at 2^20-scale positions;
    it preserves norms and composes additively, R(a) R(b) = R(a + b)."""
    rng = np.random.default_rng(31)
    freqs = rng.uniform(0.0, 2.0, 5)
    x = rng.standard_normal((3, 7, 10))
    for pos in (np.arange(7), np.arange(7) * 149_999 + 3, 12.0):
        got = O.rotate(x, pos, freqs)
        ref = _rot_complex(x, pos, freqs)
        assert np.allclose(got, ref, rtol=1e-12, atol=1e-12), pos
        assert np.allclose(np.linalg.norm(got, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)
    ab = O.rotate(O.rotate(x, 5.0, freqs), 9.0, freqs)
    assert np.allclose(ab, O.rotate(x, 14.0, freqs), rtol=1e-12, atol=1e-12)


def check_remap_zero_frequencies_is_identity():
    """All angles zero: the remap changes nothing (every rotation is the identity)."""
    rng = np.random.default_rng(32)
    p0 = _params(n_q_heads=4, n_kv_heads=2, head_dim=8, n_init=3, n_local=8, block_size=4, n_repr=2,
                 topk=2, sm_scale=0.9)
    pz = O.Params(**{**p0.__dict__, "rope_inv_freq": (0.0,) * 4})
    q, k, v = _rand_qkv(rng, p0, 70)
    a, b = O.StreamOracle(q, k, v, p0), O.StreamOracle(q, k, v, pz)
    for past, nq in ((30, 5), (61, 9)):
        ra, rb = a.step(0, past, nq), b.step(0, past, nq)
        for key in ("scores", "out", "lse"):
            assert np.allclose(ra[key], rb[key], rtol=1e-14, atol=1e-14), (past, key)
        assert (ra["idx"] == rb["idx"]).all()


def check_remap_attention_effective_positions():
    """Brute force of the remap as the paper states it: for query i at position P the key of a
    token in I or in a selected unit is placed at position P - l_L (distance l_L), a key of L or X
    at its own position; each logit is sm_scale (R(P) q) . (R(e) k) with its own rotation
    (complex arithmetic, per query and key)."""
    rng = np.random.default_rng(33)
    p = _rope_params(seed=34, n_q_heads=4, n_kv_heads=2, head_dim=6, n_init=3, n_local=5,
                     block_size=3, n_repr=1, topk=2, sm_scale=0.8)
    f = np.array(p.rope_inv_freq)
    S, G = 60, 2
    q, k, v = _rand_qkv(rng, p, S)
    for past, nq in ((20, 4), (47, 6)):
        part = O.partition(past, p)
        sel = np.stack([np.sort(rng.choice(part.n_units, 2, replace=False)) for _ in range(2)])
        out, lse = O.attend(q[0, :, past:past + nq], k[0], v[0], past, sel, p)
        for h in range(p.n_q_heads):
            g = h // G
            mem = list(range(part.n_init))
            for b in sel[g]:
                s0 = p.n_init + int(b) * p.block_size
                mem += list(range(s0, s0 + p.block_size))
            for i in range(nq):
                P = past + i
                keys = [(t, P - p.n_local) for t in mem] + [(t, t) for t in range(part.local_begin, P + 1)]
                qr = _rot_complex(q[0, h, P], P, f)
                z = np.array([p.sm_scale * float(qr @ _rot_complex(k[0, g, t], e, f)) for t, e in keys])
                w = np.exp(z - z.max())
                o = sum(w[j] * v[0, g, t] for j, (t, _) in enumerate(keys)) / w.sum()
                assert np.allclose(out[h, i], o, rtol=1e-11, atol=1e-11), (past, h, i)
                assert math.isclose(lse[h, i], z.max() + math.log(w.sum()), rel_tol=1e-11, abs_tol=1e-11)


def check_remap_relevance_effective_positions():
    """sim with the remap, literal triple sum: query i at its position P, every representative key
    at P - l_L, each rotated on its own."""
    rng = np.random.default_rng(35)
    f = rng.uniform(0.05, 1.5, 3)
    p = O.Params(n_q_heads=2, n_kv_heads=1, head_dim=6, n_init=2, n_local=5, block_size=4, n_repr=2,
                 topk=2, rope_inv_freq=tuple(f))
    G, nq, S, past = 2, 4, 50, 37
    q = rng.standard_normal((G, S, 6))
    k = rng.standard_normal((S, 6))
    rep = np.stack([np.sort(rng.choice(30, 2, replace=False)) for _ in range(6)])
    got = O.unit_relevance(q[:, past:past + nq], k, rep, p)
    ref = []
    for r in rep:
        t = 0.0
        for h in range(G):
            for i in range(nq):
                P = past + i
                for j in r:
                    t += float(_rot_complex(q[h, P], P, f) @ _rot_complex(k[j], P - p.n_local, f))
        ref.append(t)
    assert np.allclose(got, ref, rtol=1e-11, atol=1e-11)


def check_remap_repr_scores_bruteforce():
    """r_m with the remap, literal loops: window query m+j at position m+j, key m at position m."""
    rng = np.random.default_rng(36)
    p = _rope_params(seed=37, n_q_heads=4, n_kv_heads=2, head_dim=4, n_init=2, n_local=3, block_size=4)
    f = np.array(p.rope_inv_freq)
    q, k, _ = _rand_qkv(rng, p, S=2 + 3 * 4 + 3 + 1)
    so = O.StreamOracle(q, k, k, p)
    for g in range(2):
        for unit in range(3):
            m0 = p.n_init + unit * p.block_size
            ref = []
            for m in range(m0, m0 + p.block_size):
                km = _rot_complex(k[0, g, m], m, f)
                tot = 0.0
                for h in range(2 * g, 2 * g + 2):
                    for j in range(1, p.n_local + 1):
                        tot += float(_rot_complex(q[0, h, m + j], m + j, f) @ km)
                ref.append(tot / (p.n_local * 2))
            got = O.representative_scores(q[0, 2 * g:2 * g + 2], k[0, g], unit, p)
            assert np.allclose(got, ref, rtol=1e-12, atol=1e-12), (g, unit)
            assert np.allclose(so.repr_scores(0, g, unit), ref, rtol=1e-12, atol=1e-12), (g, unit)


def check_remap_reduces_to_rotary_attention():
    """No initial tokens and a window longer than the sequence: nothing is ever beyond the local
    window, so the remap is plain causal attention over rotary-encoded q and k (PyTorch's
    scaled_dot_product_attention in float64 on the rotated inputs)."""
    rng = np.random.default_rng(38)
    p = _rope_params(seed=39, n_q_heads=4, n_kv_heads=2, head_dim=8, n_init=0, n_local=64,
                     block_size=4, n_repr=1, topk=3, sm_scale=0.6)
    f = np.array(p.rope_inv_freq)
    S = 40
    q, k, v = _rand_qkv(rng, p, S)
    pos = np.arange(S)
    qr, kr = _rot_complex(q[0], pos, f), _rot_complex(k[0], pos, f)
    mask = np.tril(np.ones((S, S), dtype=bool))[None]
    ref_o, ref_l = _sdpa(qr, _expand(kr, 2), _expand(v[0], 2), mask, 0.6)
    so = O.StreamOracle(q, k, v, p)
    for past in (0, 9, 31):
        r = so.step(0, past, 9)
        assert np.allclose(r["out"], ref_o[:, past:past + 9], rtol=1e-12, atol=1e-12), past
        assert np.allclose(r["lse"], ref_l[:, past:past + 9], rtol=1e-12, atol=1e-12), past


# --------------------------------------------------------------------------- Mean Repr
def check_mean_repr_mode():
    """Units represented by their mean key: literal loops sum_h sum_i sum_d q[d] * (1/l_bs) sum_j k_j[d];
    equal to the representative-token scores with r_k = l_bs divided by l_bs; and, with the
    remap, the literal loops with every query turned by R(l_L) (complex arithmetic)."""
    rng = np.random.default_rng(40)
    base = dict(n_q_heads=4, n_kv_heads=2, head_dim=6, n_init=3, n_local=8, block_size=4, n_repr=2, topk=2)
    pm = _params(**base, mean_repr=True)
    pt = _params(**{**base, "n_repr": 4})
    S, past, nq = 60, 40, 5
    q, k, v = _rand_qkv(rng, pm, S)
    nu = O.partition(past, pm).n_units
    sm = O.StreamOracle(q, k, v, pm).scores(0, past, nq)
    st = O.StreamOracle(q, k, v, pt).scores(0, past, nq)
    assert np.allclose(sm, st / pm.block_size, rtol=1e-12, atol=1e-12)
    f = rng.uniform(0.05, 1.5, 3)
    pr = O.Params(**{**pm.__dict__, "rope_inv_freq": tuple(f)})
    sr = O.StreamOracle(q, k, v, pr).scores(0, past, nq)
    for g in range(2):
        for u in range(nu):
            s0 = pm.n_init + u * pm.block_size
            lit = lit_r = 0.0
            for h in range(2 * g, 2 * g + 2):
                for i in range(past, past + nq):
                    qr = _rot_complex(q[0, h, i], pm.n_local, f)
                    for d in range(pm.head_dim):
                        kd = sum(float(k[0, g, s0 + j, d]) for j in range(pm.block_size)) / pm.block_size
                        lit += float(q[0, h, i, d]) * kd
                        lit_r += float(qr[d]) * kd
            assert math.isclose(sm[g, u], lit, rel_tol=1e-12, abs_tol=1e-12), (g, u)
            assert math.isclose(sr[g, u], lit_r, rel_tol=1e-11, abs_tol=1e-11), (g, u)


# --------------------------------------------------------------------------- golden
def load_golden():
    with open(os.path.join(GOLDEN, "hand_worked_tiny.yaml")) as f:
        return yaml.safe_load(f)


def check_hand_worked_example():
    gd = load_golden()
    p = O.Params(**gd["params"])
    q = np.stack([np.array(gd["q_a"], float), np.array(gd["q_b"], float)])[None]
    k = np.array(gd["k"], float)[None, None]
    v = np.array(gd["v"], float)[None, None]
    so = O.StreamOracle(q, k, v, p)
    for rs in gd["repr_scores"]:
        assert np.allclose(so.repr_scores(0, 0, rs["unit"]), rs["r"], rtol=1e-14, atol=1e-14)
        assert list(so.repr_offsets(0, 0, rs["unit"])) == rs["offsets"]
    for st in gd["steps"]:
        part = O.partition(st["past_len"], p)
        assert (part.n_init, part.n_units, part.local_begin) == (
            st["partition"]["n_init"], st["partition"]["n_units"], st["partition"]["local_begin"])
        r = so.step(0, st["past_len"], st["n_q"])
        assert np.allclose(r["scores"][0], st["scores"], rtol=1e-14, atol=1e-14)
        assert list(r["idx"][0]) == st["idx"]
        assert np.allclose(r["out"], st["out"], rtol=1e-13, atol=1e-13)
        assert np.allclose(r["lse"], st["lse"], rtol=1e-13, atol=1e-13)


def check_unit_mass_uniform_closed_form():
    """q = 0 makes every logit 0: query i spreads its attention evenly over its |T_i| keys, so a
    looked-up unit's mass is G * sum_i l_bs / |T_i| with |T_i| = l_I + k_eff*l_bs + |L| + i + 1."""
    rng = np.random.default_rng(61)
    p = _params(n_q_heads=6, n_kv_heads=2, head_dim=4, n_init=3, n_local=7, block_size=5, topk=3)
    S, G = 80, 3
    _, k, v = _rand_qkv(rng, p, S)
    for past, nq in ((40, 5), (63, 1), (71, 9)):
        q = np.zeros((p.n_q_heads, nq, p.head_dim))
        part = O.partition(past, p)
        sel = np.stack([np.sort(rng.choice(part.n_units, 3, replace=False)) for _ in range(2)])
        sel[1, 2] = -1  # an empty slot: mass 0, and one unit fewer in the key set
        m = O.unit_mass(q, k[0], past, sel, p)
        for g in range(2):
            k_eff = int((sel[g] >= 0).sum())
            n_t = part.n_init + k_eff * p.block_size + (past - part.local_begin) + np.arange(1, nq + 1)
            want = G * float(np.sum(p.block_size / n_t))
            for j in range(3):
                assert math.isclose(m[g, j], want if sel[g, j] >= 0 else 0.0, rel_tol=1e-12), (past, g, j)


def check_unit_mass_bruteforce():
    """Softmax probabilities formed key by key (explicit attended-position list, per-key logits,
    math.exp), summed over each looked-up unit, every query and every head of the group; with and
    without the positional remap (complex-number rotations, memory keys at distance l_L)."""
    rng = np.random.default_rng(62)
    for remap in (False, True):
        p = _rope_params(seed=63, n_q_heads=4, n_kv_heads=2, head_dim=6, n_init=2, n_local=5,
                         block_size=3, n_repr=1, topk=2, sm_scale=0.7)
        if not remap:
            import dataclasses
            p = dataclasses.replace(p, rope_inv_freq=None)
        f = None if p.rope_inv_freq is None else np.array(p.rope_inv_freq)
        S, G = 50, 2
        q, k, _ = _rand_qkv(rng, p, S)
        for past, nq in ((22, 4), (38, 1)):
            part = O.partition(past, p)
            sel = np.stack([np.sort(rng.choice(part.n_units, 2, replace=False)) for _ in range(2)])
            m = O.unit_mass(q[0, :, past:past + nq], k[0], past, sel, p)
            for g in range(2):
                units = {int(b): set(range(p.n_init + int(b) * p.block_size,
                                           p.n_init + (int(b) + 1) * p.block_size)) for b in sel[g]}
                mem = list(range(part.n_init)) + sorted(t for u in units.values() for t in u)
                want = {b: 0.0 for b in units}
                for h in range(g * G, (g + 1) * G):
                    for i in range(nq):
                        P = past + i
                        keys = [(t, P - p.n_local if f is not None else t) for t in mem] + \
                               [(t, t) for t in range(part.local_begin, P + 1)]
                        qr = q[0, h, P] if f is None else _rot_complex(q[0, h, P], P, f)
                        z = [p.sm_scale * float(qr @ (k[0, g, t] if f is None else _rot_complex(k[0, g, t], e, f)))
                             for t, e in keys]
                        zm = max(z)
                        tot = sum(math.exp(x - zm) for x in z)
                        for (t, _), x in zip(keys, z):
                            for b, pos in units.items():
                                if t in pos and t < past:
                                    want[b] += math.exp(x - zm) / tot
                for j, b in enumerate(sel[g]):
                    assert math.isclose(m[g, j], want[int(b)], rel_tol=1e-11, abs_tol=1e-14), (remap, past, g, j)


def check_frequency_update_recurrence():
    """The decayed sum in closed form: a unit looked up every step with mass c reaches
    c (1 - d^n) / (1 - d) after n steps; one never looked up keeps s_0 d^n; units not yet
    built stay untouched."""
    d, c, n = 0.1, 2.5, 7
    freq = np.array([[4.0, 1.0, 9.0]])
    for _ in range(n):
        freq = O.frequency_update(freq, np.array([[0, -1]]), np.array([[c, 0.0]]), 2, d)
    assert math.isclose(freq[0, 0], 4.0 * d ** n + c * (1 - d ** n) / (1 - d), rel_tol=1e-13)
    assert math.isclose(freq[0, 1], 1.0 * d ** n, rel_tol=1e-13)
    assert freq[0, 2] == 9.0


ALL_CHECKS = [
    check_partition,
    check_repr_scores_bruteforce,
    check_repr_scores_prefix_identity,
    check_repr_scores_presummed_queries,
    check_repr_scores_window_one,
    check_repr_scores_window_support,
    check_top_indices,
    check_unit_relevance_linearity,
    check_mean_repr_special_case,
    check_full_attention_when_everything_selected,
    check_full_attention_when_window_covers,
    check_streaming_llm_when_no_lookup,
    check_sparse_equals_masked_dense,
    check_lse_merge,
    check_hand_worked_example,
    check_rotation_is_complex_multiplication,
    check_remap_zero_frequencies_is_identity,
    check_remap_attention_effective_positions,
    check_remap_relevance_effective_positions,
    check_remap_repr_scores_bruteforce,
    check_remap_reduces_to_rotary_attention,
    check_mean_repr_mode,
    check_unit_mass_uniform_closed_form,
    check_unit_mass_bruteforce,
    check_frequency_update_recurrence,
]
