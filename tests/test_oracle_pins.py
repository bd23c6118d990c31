"""The CPU oracle against its pins, plus planted-mistake checks showing the pins bite.

CPU only.  Each mutant below is a plausible slip in writing the oracle from the
paper (a window off by one, a dropped 1/G, ties broken the other way, causal
mask dropped, ...).  The mutant replaces the oracle function for the duration
of one test, and at least one pin must then fail.
"""
import numpy as np
import pytest

from oracle import infllm_oracle as O
from tests import oracle_pins as P


@pytest.mark.parametrize("check", P.ALL_CHECKS, ids=lambda c: c.__name__)
def test_pin(check):
    check()


# ------------------------------------------------------------------ mutants
_orig = {name: getattr(O, name) for name in
         ("partition", "representative_scores", "top_indices", "unit_relevance", "attend",
          "lse_merge", "context_positions", "select_units", "unit_start", "rotate", "mean_relevance",
          "unit_mass", "frequency_update")}


def _mut_partition_drop_remainder(past_len, p):
    # remainder of E discarded instead of kept in L
    part = _orig["partition"](past_len, p)
    if part.n_units:
        return O.Partition(part.n_init, part.n_units, max(part.local_begin, past_len - p.n_local))
    return part


def _mut_partition_ceil_units(past_len, p):
    ev = past_len - p.n_init - p.n_local
    n = -(-ev // p.block_size) if ev > 0 else 0
    n_init = min(p.n_init, past_len)
    return O.Partition(n_init, n, min(past_len, n_init + n * p.block_size))


def _mut_repr_window_shift(q_group, k_head, unit, p, q_summed=None):
    # j = 0 .. l_L-1 instead of 1 .. l_L
    G = q_group.shape[0]
    m0 = O.unit_start(unit, p)
    qw = np.asarray(q_group[:, m0: m0 + p.block_size + p.n_local - 1, :], float).sum(axis=0)
    dots = qw @ np.asarray(k_head[m0:m0 + p.block_size], float).T
    return np.array([dots[t:t + p.n_local, t].sum() for t in range(p.block_size)]) / (p.n_local * G)


def _mut_repr_no_group_mean(q_group, k_head, unit, p, q_summed=None):
    return _orig["representative_scores"](q_group, k_head, unit, p) * q_group.shape[0]


def _mut_repr_first_head_only(q_group, k_head, unit, p, q_summed=None):
    return _orig["representative_scores"](q_group[:1], k_head, unit, p)


def _mut_topk_high_index_ties(values, count):
    vals = np.array(values, float)
    order = sorted(range(len(vals)), key=lambda i: (-vals[i], -i))
    return np.array(sorted(order[:min(count, len(vals))]), dtype=np.int64)


def _mut_topk_smallest(values, count):
    return _orig["top_indices"](-np.asarray(values, float), count)


def _mut_relevance_sign(q, k, rep, p=None):
    return -_orig["unit_relevance"](q, k, rep, p)


def _mut_relevance_one_rep(q, k, rep, p=None):
    return _orig["unit_relevance"](q, k, rep[:, :1], p)


# ---- positional remap slips
def _mut_rotate_half_split(x, positions, inv_freq):
    # pairs (i, i + D/2) instead of (2i, 2i+1)
    x = np.asarray(x, float)
    h = x.shape[-1] // 2
    ang = np.multiply.outer(np.asarray(positions, float), np.asarray(inv_freq, float))
    c, s = np.cos(ang), np.sin(ang)
    out = np.empty_like(x)
    out[..., :h] = x[..., :h] * c - x[..., h:] * s
    out[..., h:] = x[..., :h] * s + x[..., h:] * c
    return out


def _mut_rotate_backwards(x, positions, inv_freq):
    return _orig["rotate"](x, -np.asarray(positions, float), inv_freq)


def _mut_relevance_true_positions(q, k, rep, p=None):
    # memory keys scored without the remap (no R(l_L) on the queries)
    import dataclasses
    return _orig["unit_relevance"](q, k, rep, None if p is None else dataclasses.replace(p, rope_inv_freq=None))


def _mut_repr_unrotated(q_group, k_head, unit, p, q_summed=None):
    import dataclasses
    return _orig["representative_scores"](q_group, k_head, unit, dataclasses.replace(p, rope_inv_freq=None),
                                          q_summed)


def _mut_attend_memory_negative_distance(q_chunk, k, v, past_len, sel, p):
    # memory queries turned by R(-l_L) instead of R(l_L)
    import dataclasses
    if p.rope_inv_freq is None:
        return _orig["attend"](q_chunk, k, v, past_len, sel, p)
    real_rotate = O.rotate

    def rot(x, positions, f):
        if np.ndim(positions) == 0 and float(positions) == float(p.n_local):
            positions = -float(p.n_local)
        return real_rotate(x, positions, f)
    O.rotate = rot
    try:
        return _orig["attend"](q_chunk, k, v, past_len, sel, p)
    finally:
        O.rotate = real_rotate


def _mut_mean_sum_not_mean(q, k, n_units, p):
    # the key sum instead of the mean
    return _orig["mean_relevance"](q, k, n_units, p) * p.block_size


def _mut_mean_skips_last_key(q, k, n_units, p):
    # l_bs - 1 keys averaged (an off-by-one in the unit's span)
    if n_units == 0:
        return np.zeros(0)
    pos = np.stack([np.arange(O.unit_start(u, p), O.unit_start(u, p) + p.block_size - 1) for u in range(n_units)])
    return O.unit_relevance(q, k, pos, p) / (p.block_size - 1)


def _mut_attend_init_true_positions(q_chunk, k, v, past_len, sel, p):
    # initial tokens kept at their true positions (only the units remapped)
    if p.rope_inv_freq is None:
        return _orig["attend"](q_chunk, k, v, past_len, sel, p)
    Hq, nq, D = q_chunk.shape
    G = p.group
    f = p.rope_inv_freq
    part = O.partition(past_len, p)
    out, lse = np.empty((Hq, nq, D)), np.empty((Hq, nq))
    for g in range(p.n_kv_heads):
        pos = O.context_positions(past_len, sel[g], p)
        for h in range(g * G, (g + 1) * G):
            for i in range(nq):
                P = past_len + i
                keys = np.concatenate([pos, np.arange(past_len, P + 1)])
                qr = O.rotate(q_chunk[h, i], float(P), f)
                z = []
                for t in keys:
                    e = t if (t < part.n_init or t >= part.local_begin) else P - p.n_local
                    z.append(p.sm_scale * float(qr @ O.rotate(k[g, t], float(e), f)))
                z = np.array(z)
                w = np.exp(z - z.max())
                out[h, i] = (w[:, None] * v[g, keys]).sum(0) / w.sum()
                lse[h, i] = z.max() + np.log(w.sum())
    return out, lse


def _mut_attend_no_causal(q_chunk, k, v, past_len, sel, p):
    # current tokens fully visible to each other
    Hq, nq, D = q_chunk.shape
    G = p.group
    out, lse = np.empty((Hq, nq, D)), np.empty((Hq, nq))
    for g in range(p.n_kv_heads):
        pos = np.concatenate([O.context_positions(past_len, sel[g], p),
                              np.arange(past_len, past_len + nq)])
        for h in range(g * G, (g + 1) * G):
            z = p.sm_scale * q_chunk[h] @ k[g, pos].T
            m = z.max(axis=1, keepdims=True)
            w = np.exp(z - m)
            out[h] = (w / w.sum(1, keepdims=True)) @ v[g, pos]
            lse[h] = (m + np.log(w.sum(1, keepdims=True)))[:, 0]
    return out, lse


def _mut_attend_no_scale(q_chunk, k, v, past_len, sel, p):
    import dataclasses
    return _orig["attend"](q_chunk, k, v, past_len, sel, dataclasses.replace(p, sm_scale=1.0))


def _mut_attend_log2_lse(q_chunk, k, v, past_len, sel, p):
    o, l = _orig["attend"](q_chunk, k, v, past_len, sel, p)
    return o, l / np.log(2.0)


def _mut_merge_unnormalised(outs, lses):
    # weights exp(lse_s - max) applied but never divided by their sum
    L = np.stack(lses)
    M = L.max(axis=0)
    w = np.exp(L - M)
    return sum(w[s][..., None] * outs[s] for s in range(len(outs))), M + np.log(w.sum(axis=0))


def _mut_unit_start_off_by_one(unit, p):
    return p.n_init + unit * p.block_size + 1


def _mut_context_drop_init(past_len, sel, p):
    pos = _orig["context_positions"](past_len, sel, p)
    return pos[O.partition(past_len, p).n_init:]


def _mut_select_top_km_minus_1(sim, p, k=None):
    k = p.topk if k is None else k
    out = _orig["select_units"](sim, p, k)
    c = (out >= 0).sum()
    if c:
        out[c - 1] = -1
    return out


# ---- attention mass and frequency score slips
def _mut_mass_unnormalised(q_chunk, k, past_len, sel, p):
    # exp(z - max) summed without dividing by the row's total
    n_units = O.partition(past_len, p).n_units
    mass = np.zeros(np.shape(sel))
    for g in range(p.n_kv_heads):
        z, keys = O.attention_logits(q_chunk, k, past_len, sel[g], p, g)
        w = np.exp(z - z.max(axis=2, keepdims=True))
        for j, b in enumerate(sel[g]):
            if 0 <= b < n_units:
                s0 = O.unit_start(int(b), p)
                mass[g, j] = w[:, :, (keys >= s0) & (keys < s0 + p.block_size)].sum()
    return mass


def _mut_mass_first_head_only(q_chunk, k, past_len, sel, p):
    G = p.group
    return _orig["unit_mass"](q_chunk, k, past_len, sel, p) / G


def _mut_mass_span_short(q_chunk, k, past_len, sel, p):
    # the unit's last key left out
    n_units = O.partition(past_len, p).n_units
    mass = np.zeros(np.shape(sel))
    for g in range(p.n_kv_heads):
        z, keys = O.attention_logits(q_chunk, k, past_len, sel[g], p, g)
        prob = np.exp(z - z.max(axis=2, keepdims=True))
        prob /= prob.sum(axis=2, keepdims=True)
        for j, b in enumerate(sel[g]):
            if 0 <= b < n_units:
                s0 = O.unit_start(int(b), p)
                mass[g, j] = prob[:, :, (keys >= s0) & (keys < s0 + p.block_size - 1)].sum()
    return mass


def _mut_mass_no_remap(q_chunk, k, past_len, sel, p):
    import dataclasses
    return _orig["unit_mass"](q_chunk, k, past_len, sel, dataclasses.replace(p, rope_inv_freq=None))


def _mut_freq_add_then_decay(freq, sel, mass, n_units, decay):
    f = np.array(freq, dtype=np.float64, copy=True)
    for g in range(f.shape[0]):
        for j, b in enumerate(sel[g]):
            if 0 <= b < n_units:
                f[g, b] += mass[g, j]
    f[:, :n_units] *= decay
    return f


def _mut_freq_idle_units_kept(freq, sel, mass, n_units, decay):
    # only looked-up units decay
    f = np.array(freq, dtype=np.float64, copy=True)
    for g in range(f.shape[0]):
        for j, b in enumerate(sel[g]):
            if 0 <= b < n_units:
                f[g, b] = f[g, b] * decay + mass[g, j]
    return f


MUTANTS = [
    ("partition", _mut_partition_drop_remainder),
    ("partition", _mut_partition_ceil_units),
    ("representative_scores", _mut_repr_window_shift),
    ("representative_scores", _mut_repr_no_group_mean),
    ("representative_scores", _mut_repr_first_head_only),
    ("top_indices", _mut_topk_high_index_ties),
    ("top_indices", _mut_topk_smallest),
    ("unit_relevance", _mut_relevance_sign),
    ("unit_relevance", _mut_relevance_one_rep),
    ("attend", _mut_attend_no_causal),
    ("attend", _mut_attend_no_scale),
    ("attend", _mut_attend_log2_lse),
    ("lse_merge", _mut_merge_unnormalised),
    ("unit_start", _mut_unit_start_off_by_one),
    ("context_positions", _mut_context_drop_init),
    ("select_units", _mut_select_top_km_minus_1),
    ("unit_mass", _mut_mass_unnormalised),
    ("unit_mass", _mut_mass_first_head_only),
    ("unit_mass", _mut_mass_span_short),
    ("unit_mass", _mut_mass_no_remap),
    ("frequency_update", _mut_freq_add_then_decay),
    ("frequency_update", _mut_freq_idle_units_kept),
    ("rotate", _mut_rotate_half_split),
    ("rotate", _mut_rotate_backwards),
    ("unit_relevance", _mut_relevance_true_positions),
    ("representative_scores", _mut_repr_unrotated),
    ("attend", _mut_attend_memory_negative_distance),
    ("attend", _mut_attend_init_true_positions),
    ("mean_relevance", _mut_mean_sum_not_mean),
    ("mean_relevance", _mut_mean_skips_last_key),
]


@pytest.mark.parametrize("name,mutant", MUTANTS, ids=[m.__name__ for _, m in MUTANTS])
def test_pins_catch_planted_mistake(monkeypatch, name, mutant):
    monkeypatch.setattr(O, name, mutant)
    failed = []
    for check in P.ALL_CHECKS:
        try:
            check()
        except (AssertionError, IndexError, ValueError):
            failed.append(check.__name__)
    assert failed, f"no pin caught mutant {mutant.__name__} of {name}"
