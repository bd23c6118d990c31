"""Parity at the benchmark's full sizes, in the benchmark's launch configuration (GPU).

The device runs whole streams exactly as bench.py does (infllm_step per chunk,
workspace from infllm_workspace_bytes).  The oracle checks what it can compute
one by one: sampled steps end to end at 128K; at 1M and for the 16 x 128K
decode batch, the whole lookup of sampled (sequence, kv head) pairs (the
oracle builds the representatives of every unit, scores every unit and takes
the top-k; the device's lookup must match outside the near-tie band, and its
attention output at that lookup must match the oracle's), plus sampled units
(representatives and key sums), the selection as the exact top-k of the
device's own scores (a property that holds at any size), and attention with a
test-chosen unit set on sampled heads.
"""
import numpy as np
import pytest
import torch

from oracle import infllm_oracle as O
from paper_2402_04617_amd import infllm as F
from tests.gpu_util import Layer, check_selection, conditioned_step, dev, host, log, oparams
from workload import WORKLOADS, Synth

pytestmark = pytest.mark.gpu


def wl_params(wl):
    return F.params(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.n_init, wl.n_local, wl.block_size,
                    wl.n_repr, wl.topk, wl.dtype)


def upload_streamed(synth, name, threads=16):
    """Device tensor [B][H][S][D] bf16, drawn head by head in parallel (the host keeps nothing)."""
    from concurrent.futures import ThreadPoolExecutor
    wl = synth.wl
    H = wl.n_q_heads if name == "q" else wl.n_kv_heads
    t = torch.empty((wl.batch, H, wl.seq_len, wl.head_dim), dtype=torch.bfloat16, device="cuda")
    fn = getattr(synth, name)
    jobs = [(b, h) for b in range(wl.batch) for h in range(H)]
    with ThreadPoolExecutor(threads) as ex:
        for (b, h), x in zip(jobs, ex.map(lambda bh: fn(bh[0], bh[1], 0, wl.seq_len), jobs)):
            t[b, h].copy_(torch.from_numpy(x).to(torch.bfloat16))
    return t


def topk_property(scores_row, idx_row, k):
    """idx is exactly the top-k (ties to the lower index) of the given float32 scores, ascending."""
    exp = O.select_units(scores_row.astype(np.float64), O.Params(1, 1, 64, 0, 1, 1, 1, k))
    assert np.array_equal(idx_row, exp), (idx_row, exp)


def check_units_sampled(synth, L, units, b=0):
    """Representatives and key sums of sampled units against the oracle, from slices drawn on demand.

    The oracle sees the slice [m0, m0 + l_bs + l_L) of one unit's keys and its group's queries, with
    l_I = 0 so that the unit starts at local position 0."""
    wl = synth.wl
    p = oparams(L.p)
    G = wl.group
    pl = O.Params(p.n_q_heads, p.n_kv_heads, p.head_dim, 0, p.n_local, p.block_size, p.n_repr, p.topk)
    ridx = host(L.mem.repr_idx)
    ksum = host(L.mem.unit_ksum)
    for g, u in units:
        lo = wl.n_init + u * wl.block_size
        hi = lo + wl.block_size + wl.n_local
        qg = np.stack([synth.q(b, g * G + h, lo, hi) for h in range(G)])
        kh = synth.k(b, g, lo, hi)
        r = O.representative_scores(qg, kh, 0, pl)
        exp = O.representatives(r, pl)
        got = ridx[b, g, u]
        if not np.array_equal(got, exp):
            srt = np.sort(r)[::-1]
            assert (srt[wl.n_repr - 1] - srt[wl.n_repr]) <= 1e-9 * max(1.0, abs(srt[wl.n_repr - 1])), \
                (g, u, got, exp)
        ks = kh[got].astype(np.float64).sum(axis=0)
        assert np.allclose(ksum[b, g, :, u, :].reshape(-1), ks, rtol=1e-6, atol=1e-6), (g, u)


@pytest.mark.parametrize("mode", ["plain", "remap", "mean"])
def test_encode_128k_sampled_steps(mode):
    """The benchmark's 128K legs: plain, with the positional remap (Llama-3 rotary frequencies,
    inputs read as unrotated) and with Mean Repr."""
    wl = WORKLOADS["llama3-8b-128k"]
    synth = Synth(wl, 0)
    log(f"[128k {mode}] generating inputs")
    q, k, v = synth.full("q", threads=16), synth.full("k", threads=16), synth.full("v", threads=16)
    p = F.params(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.n_init, wl.n_local, wl.block_size, wl.n_repr,
                 wl.topk, wl.dtype, rope_inv_freq=F.rope_frequencies(wl.head_dim) if mode == "remap" else None,
                 repr_mode="mean" if mode == "mean" else "tokens")
    op = oparams(p)
    L = Layer(p, 1, wl.seq_len, chunk=wl.chunk)
    qd, kd, vd = dev(q, "bf16"), dev(k, "bf16"), dev(v, "bf16")
    so = O.StreamOracle(q, k, v, op)
    steps = wl.step_starts()
    check = {100, len(steps) - 1} if mode == "plain" else {len(steps) - 1}
    lse_tol = 1e-2 if mode == "remap" else 1e-3  # rotated q and k enter the MFMA rounded to bf16
    G = wl.group
    n_checked = 0
    mass = torch.zeros((1, wl.n_kv_heads, wl.topk), dtype=torch.float32, device="cuda")
    mass_rel = 2e-2 if mode == "remap" else 2e-3  # twice the lse tolerance (p = exp(z - lse))
    for si, (past, n) in enumerate(steps):
        L.step(qd, kd, vd, past, n)
        if si not in check:
            continue
        log(f"[128k] checking step {si} past={past}")
        # the looked-up units' attention mass at the benchmark's shape (its unit-mass leg)
        F.infllm_unit_mass(p, L.mem.struct, qd.data_ptr() + past * wl.head_dim * 2, wl.seq_len * wl.head_dim, n,
                           past, L.idx, wl.topk, L.lse, 0.1, mass)
        nu = O.partition(past, op).n_units
        got = L.capture(n, nu)
        gm = host(mass)
        r = conditioned_step(so, 0, past, n, host(L.mem.repr_idx)[0])
        same = [check_selection(got["idx"][0, g], r["idx"][g], r["scores"][g], wl.topk) for g in range(wl.n_kv_heads)]
        # where the device's lookup differs inside the near-tie band it is a valid lookup too: the
        # oracle then attends over the device's units, so every kv head is compared
        if not all(same):
            r_dev = so.step(0, past, n, sel=np.array(got["idx"][0]))
            for key in ("out", "lse"):
                r[key] = r_dev[key]
        sel_dev = np.array(got["idx"][0])
        om = O.unit_mass(q[0, :, past:past + n], k[0], past, sel_dev, op)
        for g in range(wl.n_kv_heads):
            assert np.all(np.abs(gm[0, g] - om[g]) <= mass_rel * om[g] + 1e-6 * G * n), (si, g)
        for g in range(wl.n_kv_heads):
            es = r["scores"][g]
            scale = max(np.abs(es).max(), np.sqrt(np.mean(es ** 2)))
            assert np.abs(got["scores"][0, g] - es).max() <= 1e-3 * scale, (si, g)
            topk_property(got["scores"][0, g].astype(np.float32), got["idx"][0, g], wl.topk)
            hs = slice(g * G, (g + 1) * G)
            assert np.abs(got["out"][0, hs] - r["out"][hs]).max() <= 2e-2, (si, g)
            assert np.abs(got["lse"][0, hs] - r["lse"][hs]).max() <= lse_tol, (si, g)
            n_checked += 1
    assert n_checked == len(check) * wl.n_kv_heads


def oracle_lookup_head(synth, op, b, g, past, n, dev_repr):
    """The oracle's whole lookup for one (sequence, kv head) at the step (past, n), from slices drawn
    on demand: the representatives of every unit built by then, the relevance of every unit and the
    top-k_m.  Where the device's representative set of a unit differs from the oracle's, it must lie
    inside the 1e-3 near-tie band of r_m, and that unit is then scored with the device's set (the
    conditioned oracle, as in the stream tests).  dev_repr: [>= n_units][r_k] device offsets.
    Returns (scores float64 [n_units], sel [k_m], q chunk [G][n][D], keys [past + n][D], r_m ties)."""
    from concurrent.futures import ThreadPoolExecutor
    wl = synth.wl
    G = wl.group
    nu = O.partition(past, op).n_units
    q_sum = np.zeros((past + n, wl.head_dim))
    qx = np.empty((G, n, wl.head_dim), dtype=np.float32)
    with ThreadPoolExecutor(G) as ex:
        for h, x in enumerate(ex.map(lambda h: synth.q(b, g * G + h, 0, past + n), range(G))):
            q_sum += x
            qx[h] = x[past:]
    kh = synth.k(b, g, 0, past + n)
    dummy = np.zeros((G, 1, wl.head_dim))
    reps = np.empty((nu, wl.n_repr), dtype=np.int64)
    ties = 0
    for u in range(nu):
        r = O.representative_scores(dummy, kh, u, op, q_summed=q_sum)
        mine = O.representatives(r, op)
        dev_off = np.sort(np.asarray(dev_repr[u], dtype=np.int64))
        if not np.array_equal(mine, dev_off):
            check_selection(np.asarray(dev_repr[u], dtype=np.int64), mine, r, wl.n_repr)
            ties += 1
        reps[u] = O.unit_start(u, op) + dev_off
    scores = O.unit_relevance(qx, kh, reps, op)
    return scores, O.select_units(scores, op), qx, kh, ties


def check_lookup_and_attention(synth, L, op, got, b, g, past, n, lse_tol=1e-3):
    """Full lookup parity for one (sequence, kv head): every unit's score against the oracle, the
    lookup bit-exact outside the near-tie band, and O / lse at the device's own (validated) lookup."""
    wl = synth.wl
    G = wl.group
    log(f"[full lookup] b={b} g={g} past={past}: oracle over every unit")
    es, sel, qx, kh, ties = oracle_lookup_head(synth, op, b, g, past, n, host(L.mem.repr_idx)[b, g])
    scale = max(np.abs(es).max(), np.sqrt(np.mean(es ** 2)))
    err = np.abs(got["scores"][b, g] - es).max()
    assert err <= 1e-3 * scale, (b, g, err / scale)
    dev_idx = got["idx"][b, g]
    same = check_selection(dev_idx, sel, es, wl.topk)
    # attention at the device's lookup: identical to the oracle's, or a valid set inside the tie band
    vv = synth.v(b, g, 0, past + n)
    og = O.Params(G, 1, wl.head_dim, op.n_init, op.n_local, op.block_size, op.n_repr, op.topk, op.sm_scale)
    eo, el = O.attend(qx, kh[None], vv[None], past, dev_idx[None], og)
    hs = slice(g * G, (g + 1) * G)
    assert np.abs(got["out"][b, hs] - eo).max() <= 2e-2, (b, g)
    assert np.abs(got["lse"][b, hs] - el).max() <= lse_tol, (b, g)
    return same, ties


def _attend_with_chosen_units(synth, L, past, heads, rng, b=0):
    """The device's attention at this step with a test-chosen unit set, against the oracle's attend on
    the given kv heads (all of their query heads and rows)."""
    wl = synth.wl
    p = L.p
    op = oparams(p)
    nu = O.partition(past, op).n_units
    sel = np.full((wl.batch, wl.n_kv_heads, wl.topk), -1, dtype=np.int64)
    for bb in range(wl.batch):
        for g in range(wl.n_kv_heads):
            sel[bb, g, :min(wl.topk, nu)] = np.sort(rng.choice(nu, min(wl.topk, nu), replace=False))
    n_q = wl.chunk if wl.decode_steps == 0 else 1
    S, D, G = wl.seq_len, wl.head_dim, wl.group
    idx = torch.from_numpy(sel.astype(np.int32)).cuda()
    out = torch.zeros((wl.batch, wl.n_q_heads, n_q, D), dtype=torch.bfloat16, device="cuda")
    lse = torch.zeros((wl.batch, wl.n_q_heads, n_q), device="cuda")
    F.infllm_chunk_attend(p, L.mem.struct, L.q_dev.data_ptr() + past * D * 2, S * D, n_q, past, idx, wl.topk,
                          out, n_q * D, lse, L.ws)
    torch.cuda.synchronize()
    got_o, got_l = host(out).astype(np.float64), host(lse).astype(np.float64)
    og = O.Params(G, 1, D, p.n_init, p.n_local, p.block_size, p.n_repr, p.topk, float(p.sm_scale))
    for g in heads:
        kk = synth.k(b, g, 0, past + n_q)[None]
        vv = synth.v(b, g, 0, past + n_q)[None]
        qx = np.stack([synth.q(b, g * G + h, past, past + n_q) for h in range(G)])
        eo, el = O.attend(qx, kk, vv, past, sel[b, g][None], og)
        err = np.abs(got_o[b, g * G:(g + 1) * G] - eo).max()
        assert err <= 2e-2, (g, err)
        assert np.abs(got_l[b, g * G:(g + 1) * G] - el).max() <= 1e-3, g


def test_encode_1m_sampled():
    wl = WORKLOADS["llama3-8b-1m"]
    synth = Synth(wl, 0)
    p = wl_params(wl)
    op = oparams(p)
    log("[1m] uploading inputs")
    qd, kd, vd = upload_streamed(synth, "q"), upload_streamed(synth, "k"), upload_streamed(synth, "v")
    L = Layer(p, 1, wl.seq_len, chunk=wl.chunk)
    L.q_dev = qd
    steps = wl.step_starts()
    log(f"[1m] running {len(steps)} steps")
    for si, (past, n) in enumerate(steps):
        L.step(qd, kd, vd, past, n)
    past, n = steps[-1]
    nu = O.partition(past, op).n_units
    got = L.capture(n, nu)
    rng = np.random.default_rng(7)
    # units: early, middle, late, needles
    units = [(g, int(u)) for g in range(wl.n_kv_heads) for u in rng.choice(nu, 3, replace=False)]
    units += [(g, int(u)) for g in (0, 5) for u in synth.needle_blocks(0, g)[:2]]
    log(f"[1m] checking {len(units)} units")
    check_units_sampled(synth, L, units)
    # scores of sampled units at the last step: sim = Qbar . Kbar with the oracle's own representatives
    G = wl.group
    pl = O.Params(p.n_q_heads, p.n_kv_heads, p.head_dim, 0, p.n_local, p.block_size, p.n_repr, p.topk)
    for g in (0, 3, 7):
        qx = np.stack([synth.q(0, g * G + h, past, past + n) for h in range(G)])
        for u in rng.choice(nu, 16, replace=False):
            m0 = wl.n_init + int(u) * wl.block_size
            qg = np.stack([synth.q(0, g * G + h, m0, m0 + wl.block_size + wl.n_local) for h in range(G)])
            kh = synth.k(0, g, m0, m0 + wl.block_size + wl.n_local)
            reps = O.representatives(O.representative_scores(qg, kh, 0, pl), pl)
            exp = O.unit_relevance(qx, kh, reps[None])[0]
            scale = max(abs(exp), np.sqrt(np.mean(got["scores"][0, g] ** 2)))
            assert abs(got["scores"][0, g, u] - exp) <= 1e-3 * scale, (g, u)
        topk_property(got["scores"][0, g].astype(np.float32), got["idx"][0, g], wl.topk)
        needles = set(int(x) for x in synth.needle_blocks(0, g) if x < nu)
        assert needles <= set(got["idx"][0, g].tolist()), "planted needle blocks must be looked up"
    # the whole lookup of the last chunk on two kv heads: all 8,155 units scored by the oracle
    for g in (2, 5):
        check_lookup_and_attention(synth, L, op, got, 0, g, past, n)
    log("[1m] attention with chosen units")
    _attend_with_chosen_units(synth, L, past, heads=(0, 6), rng=rng)


def test_decode_16x128k_sampled():
    wl = WORKLOADS["llama3-8b-decode-16x128k"]
    synth = Synth(wl, 0)
    p = wl_params(wl)
    op = oparams(p)
    log("[decode] uploading inputs")
    qd, kd, vd = upload_streamed(synth, "q"), upload_streamed(synth, "k"), upload_streamed(synth, "v")
    L = Layer(p, wl.batch, wl.seq_len, chunk=wl.chunk)
    L.q_dev = qd
    S, D = wl.seq_len, wl.head_dim
    log("[decode] building memory of the prior context")
    for past in range(0, wl.prefill_len, wl.chunk):
        nu = O.partition(past, op).n_units
        if nu > L.units_built:
            F.infllm_build_units(p, L.mem.struct, L.units_built, nu - L.units_built, past)
            L.units_built = nu
        F.infllm_append(p, L.mem.struct, qd.data_ptr() + past * D * 2, S * D, kd.data_ptr() + past * D * 2,
                        vd.data_ptr() + past * D * 2, S * D, wl.chunk, past)
    steps = wl.step_starts()[-wl.decode_steps:]
    rng = np.random.default_rng(11)
    # step 128 is the first with 992 units: unit 991 is built by that step's own construction stage
    assert O.partition(steps[128][0], op).n_units == O.partition(steps[127][0], op).n_units + 1
    for si, (past, n) in enumerate(steps):
        L.step(qd, kd, vd, past, n)
        if si in (0, 128, 200, len(steps) - 1):
            nu = O.partition(past, op).n_units
            got = L.capture(1, nu)
            log(f"[decode] step {si}: top-k property and needles")
            for b in (0, 9, 15):
                for g in (1, 6):
                    topk_property(got["scores"][b, g].astype(np.float32), got["idx"][b, g], wl.topk)
                    if past % wl.needle_query_every == 0:  # only planted queries lean toward the needles
                        needles = set(int(x) for x in synth.needle_blocks(b, g) if x < nu)
                        assert needles <= set(got["idx"][b, g].tolist())
            if si in (0, 128, len(steps) - 1):
                # every unit's score, the lookup and the attention of two (sequence, kv head) pairs
                for b, g in ((2, 3), (13, 6)):
                    check_lookup_and_attention(synth, L, op, got, b, g, past, 1)
    log("[decode] sampled units")
    nu = O.partition(steps[-1][0], op).n_units
    for b in (0, 15):
        check_units_sampled(synth, L, [(g, int(u)) for g in (0, 7) for u in rng.choice(nu, 3, replace=False)]
                            + [(2, nu - 1)], b=b)
    log("[decode] attention with chosen units")
    _attend_with_chosen_units(synth, L, steps[-1][0], heads=(0, 4), rng=rng, b=3)
