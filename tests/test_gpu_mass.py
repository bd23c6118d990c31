"""Attention mass of the looked-up units and the decayed frequency score (GPU).

Each step of a stream runs through infllm_step, then infllm_unit_mass takes the
step's lookup and lse; the masses and the running frequency scores are compared
with the oracle's unit_mass / frequency_update on the same inputs (decay 0.1,
the paper's setting).  Where a lookup legitimately differs inside a near-tie,
the oracle takes the device's valid set for that kv head (the conditioned
oracle), since that set is what the attention used.

Tolerance: a probability exp(z - lse) inherits the error of z - lse, and the
attention's lse is held to 1e-3 (bf16), 1e-2 (bf16 with the remap, whose rotated
queries and keys are rounded to bf16) and 1e-4 (float32) of the oracle's; the
mass is compared to that relative bound, doubled, plus 1e-6 * G * n_q.
"""
import numpy as np
import pytest
import torch

from oracle import infllm_oracle as O
from paper_2402_04617_amd import infllm as F
from tests.gpu_util import Layer, check_selection, conditioned_step, dev, host, log, oparams
from tests.test_gpu_kernels import rand_inputs

pytestmark = pytest.mark.gpu

DECAY = 0.1


def _rel_tol(p):
    if p.dtype == F.INFLLM_F32:
        return 2e-4
    return 2e-2 if p.remap else 2e-3


def _run(p, dtype, q, k, v, steps, chunk, in_step=False):
    op = oparams(p)
    B, G, Hkv = q.shape[0], p.n_q_heads // p.n_kv_heads, p.n_kv_heads
    L = Layer(p, B, q.shape[2], chunk=chunk)
    qd, kd, vd = dev(q, dtype), dev(k, dtype), dev(v, dtype)
    so = O.StreamOracle(q, k, v, op)
    kk = max(1, p.topk)
    mass = torch.zeros((B, Hkv, kk), dtype=torch.float32, device="cuda")
    freq = torch.zeros((B, Hkv, L.max_units), dtype=torch.float32, device="cuda")
    ofreq = np.zeros((B, Hkv, L.max_units))
    esz = 2 if dtype == "bf16" else 4
    S, D = q.shape[2], q.shape[3]
    rel = _rel_tol(p)
    n_checked = 0
    for si, (past, n) in enumerate(steps):
        if in_step:
            L.step_mass(qd, kd, vd, past, n, DECAY, mass, freq)
        else:
            L.step(qd, kd, vd, past, n)
            F.infllm_unit_mass(p, L.mem.struct, qd.data_ptr() + past * D * esz, S * D, n, past, L.idx, p.topk,
                               L.lse, DECAY, mass, freq)
        log(f"[mass] step={si} past={past} n={n} in_step={in_step}")
        nu = O.partition(past, op).n_units
        got = L.capture(n, nu)
        gm, gf = host(mass), host(freq)
        ridx = host(L.mem.repr_idx)
        for b in range(B):
            r = conditioned_step(so, b, past, n, ridx[b])
            sel = np.array(r["idx"])
            for g in range(Hkv):
                if not check_selection(got["idx"][b, g], r["idx"][g], r["scores"][g], p.topk):
                    sel[g] = got["idx"][b, g]  # a valid set inside the tie band: what the attention used
            om = O.unit_mass(q[b, :, past:past + n], k[b], past, sel, op)
            ofreq[b] = O.frequency_update(ofreq[b], sel, om, nu, DECAY)
            floor = 1e-6 * G * n
            for g in range(Hkv):
                if p.topk:
                    err = np.abs(gm[b, g, :p.topk] - om[g])
                    assert np.all(err <= rel * om[g] + floor), (si, b, g, gm[b, g], om[g])
                    n_checked += int((sel[g] >= 0).sum())
                if nu:
                    ferr = np.abs(gf[b, g, :nu] - ofreq[b, g, :nu])
                    assert np.all(ferr <= rel * np.abs(ofreq[b, g, :nu]) + floor), (si, b, g)
                assert np.all(gf[b, g, nu:] == 0.0), (si, b, g)  # units not built yet are untouched
    assert n_checked > 0


def _steps(S, chunk):
    return [(s, min(chunk, S - s)) for s in range(0, S, chunk)]


# (dtype, G, Hkv, D, l_I, l_L, l_bs, r_k, k_m, S, chunk, remap)
CASES = [
    ("bf16", 4, 2, 128, 5, 300, 24, 4, 7, 1500, 128, False),
    ("bf16", 4, 2, 128, 5, 300, 24, 4, 7, 1500, 128, True),
    ("bf16", 2, 1, 64, 0, 256, 256, 2, 3, 1800, 300, False),
    ("bf16", 8, 1, 128, 64, 512, 64, 4, 8, 2600, 256, False),
    ("f32", 2, 2, 64, 3, 200, 40, 2, 5, 1100, 100, False),
    ("f32", 2, 1, 64, 16, 256, 32, 4, 4, 1000, 64, True),
]


@pytest.mark.parametrize("case", CASES)
def test_unit_mass_stream(case):
    dtype, G, Hkv, D, n_init, n_local, lbs, nrep, topk, S, chunk, remap = case
    rng = np.random.default_rng(sum(case[1:11]))
    freqs = F.rope_frequencies(D, 10000.0) if remap else None
    p = F.params(G * Hkv, Hkv, D, n_init, n_local, lbs, nrep, topk, dtype, rope_inv_freq=freqs)
    q, k, v = rand_inputs(rng, G * Hkv, Hkv, S, D, dtype)
    _run(p, dtype, q, k, v, _steps(S, chunk), chunk)


# infllm_step_mass: the first three shapes have l_I and l_bs multiples of 64 (the attention writes
# the per-tile partials while it runs, the masses follow from the merged lse); the last one takes
# the unit-mass kernel after the step.
STEP_CASES = [
    ("bf16", 8, 1, 128, 64, 512, 64, 4, 8, 2600, 256, False),
    ("bf16", 2, 1, 64, 0, 256, 256, 2, 3, 1800, 300, False),
    ("bf16", 4, 2, 128, 128, 512, 128, 4, 6, 3000, 256, True),
    ("bf16", 4, 2, 128, 5, 300, 24, 4, 7, 1500, 128, False),
]


@pytest.mark.parametrize("case", STEP_CASES)
def test_unit_mass_in_step(case):
    dtype, G, Hkv, D, n_init, n_local, lbs, nrep, topk, S, chunk, remap = case
    rng = np.random.default_rng(sum(case[1:11]) + 1)
    freqs = F.rope_frequencies(D, 10000.0) if remap else None
    p = F.params(G * Hkv, Hkv, D, n_init, n_local, lbs, nrep, topk, dtype, rope_inv_freq=freqs)
    q, k, v = rand_inputs(rng, G * Hkv, Hkv, S, D, dtype)
    _run(p, dtype, q, k, v, _steps(S, chunk), chunk, in_step=True)


def test_unit_mass_in_step_long_rows():
    # 64-token units past 65,920 prior tokens: the score rows hold more than 1,024 units (1,035 and
    # 1,051 at the last two steps), where the attention selects with sixteen keys per thread; it
    # writes the same per-tile partials
    p = F.params(2, 1, 64, 64, 256, 64, 2, 4, "bf16")
    S, chunk = 68000, 1024
    assert O.partition(S - chunk, oparams(p)).n_units > 1024
    q, k, v = rand_inputs(np.random.default_rng(1234), 2, 1, S, 64, "bf16")
    _run(p, "bf16", q, k, v, _steps(S, chunk), chunk, in_step=True)


def test_unit_mass_in_step_mean_repr():
    # the Mean Repr units (scored by the mean of their keys): the same attention tiles, so the
    # same partials; 128-token units after a 64-token I, the lookup larger than the unit count
    # in the first steps (every unit looked up) and smaller later
    rng = np.random.default_rng(31)
    G, Hkv, D, S, chunk = 4, 2, 128, 2900, 256
    p = F.params(G * Hkv, Hkv, D, 64, 512, 128, 4, 6, "bf16", repr_mode="mean")
    q, k, v = rand_inputs(rng, G * Hkv, Hkv, S, D, "bf16")
    _run(p, "bf16", q, k, v, _steps(S, chunk), chunk, in_step=True)


def test_unit_mass_in_step_matches_separate_call():
    """infllm_step_mass against infllm_step + infllm_unit_mass on the same stream (Llama-3 layer shape,
    512-token chunks, k_m 32): the same lookup, output and lse bit for bit (the attention's arithmetic
    is unchanged by the partial sums it also writes), masses and frequency scores to float32 rounding
    of the two summation orders."""
    rng = np.random.default_rng(77)
    G, Hkv, D, S, chunk = 4, 2, 128, 4096 + 128 + 40 * 128 + 3 * 512, 512
    p = F.params(G * Hkv, Hkv, D, 128, 4096, 128, 4, 32, "bf16")
    q, k, v = rand_inputs(rng, G * Hkv, Hkv, S, D, "bf16")
    La, Lb = Layer(p, 1, S, chunk=chunk), Layer(p, 1, S, chunk=chunk)
    qd, kd, vd = dev(q, "bf16"), dev(k, "bf16"), dev(v, "bf16")
    ma, mb = (torch.zeros((1, Hkv, 32), device="cuda") for _ in range(2))
    fa, fb = (torch.zeros((1, Hkv, La.max_units), device="cuda") for _ in range(2))
    n_cmp = 0
    for past, n in _steps(S, chunk):
        La.step(qd, kd, vd, past, n)
        F.infllm_unit_mass(p, La.mem.struct, qd.data_ptr() + past * D * 2, S * D, n, past, La.idx, 32, La.lse,
                           DECAY, ma, fa)
        Lb.step_mass(qd, kd, vd, past, n, DECAY, mb, fb)
        nu = O.partition(past, oparams(p)).n_units
        log(f"[mass] in-step vs separate past={past} units={nu}")
        a, b = La.capture(n, nu), Lb.capture(n, nu)
        assert np.array_equal(a["idx"], b["idx"]) and np.array_equal(a["out"], b["out"])
        assert np.array_equal(a["lse"], b["lse"])
        gma, gmb = host(ma), host(mb)
        assert np.all(np.abs(gma - gmb) <= 2e-5 * np.abs(gma) + 1e-5), np.abs(gma - gmb).max()
        gfa, gfb = host(fa), host(fb)
        assert np.all(np.abs(gfa - gfb) <= 2e-5 * np.abs(gfa) + 1e-5)
        n_cmp += int(nu > 0)
    assert n_cmp >= 3


def test_unit_mass_decode():
    # prefill in chunks, then token-by-token decode of two sequences
    rng = np.random.default_rng(8)
    G, Hkv, D, S0, n_dec = 4, 2, 128, 1100, 12
    p = F.params(G * Hkv, Hkv, D, 4, 256, 32, 4, 6, "bf16")
    q, k, v = rand_inputs(rng, G * Hkv, Hkv, S0 + n_dec, D, "bf16", B=2)
    steps = _steps(S0, 220) + [(S0 + i, 1) for i in range(n_dec)]
    _run(p, "bf16", q, k, v, steps, 220)


def test_unit_mass_every_unit_looked_up():
    # l_I = 0, a one-token local window and k_m above the unit count: every built unit is
    # looked up each step (most of the attention lands on units) and the padded slots are 0
    rng = np.random.default_rng(12)
    G, Hkv, D = 2, 1, 64
    p = F.params(G * Hkv, Hkv, D, 0, 1, 16, 2, 64, "bf16")
    S, chunk = 16 * 40 + 1 + 32, 32
    q, k, v = rand_inputs(rng, G * Hkv, Hkv, S, D, "bf16")
    _run(p, "bf16", q, k, v, _steps(S, chunk), chunk)


def test_unit_mass_degenerate_calls():
    # no lookup slots (k = 0): only the decay of every built unit; no queries (n_q = 0): every
    # looked-up unit gets mass 0 and every built unit still decays; units not built stay untouched
    rng = np.random.default_rng(21)
    G, Hkv, D, S, chunk = 2, 2, 64, 700, 100
    p = F.params(G * Hkv, Hkv, D, 4, 128, 32, 2, 4, "bf16")
    q, k, v = rand_inputs(rng, G * Hkv, Hkv, S, D, "bf16")
    L = Layer(p, 1, S, chunk=chunk)
    qd, kd, vd = dev(q, "bf16"), dev(k, "bf16"), dev(v, "bf16")
    for past, n in _steps(S, chunk):
        L.step(qd, kd, vd, past, n)
    past = S - 1  # the last step's past length had units; use the full prefix for the calls below
    nu = O.partition(past, oparams(p)).n_units
    assert nu > 4
    f0 = rng.uniform(0.5, 2.0, (1, Hkv, L.max_units)).astype(np.float32)
    freq = torch.from_numpy(f0).cuda()
    mass = torch.full((1, Hkv, 4), 7.0, device="cuda")
    F.infllm_unit_mass(p, L.mem.struct, None, 0, 0, past, None, 0, None, 0.25, None, freq)
    got = host(freq)
    assert np.allclose(got[0, :, :nu], f0[0, :, :nu] * np.float32(0.25), rtol=0, atol=0)
    assert np.array_equal(got[0, :, nu:], f0[0, :, nu:])
    idx = torch.tensor([[[0, 2, -1, nu - 1], [1, 3, 4, nu + 5]]], dtype=torch.int32, device="cuda")
    F.infllm_unit_mass(p, L.mem.struct, None, 0, 0, past, idx, 4, None, 0.5, mass, freq)
    assert np.array_equal(host(mass), np.zeros((1, Hkv, 4), dtype=np.float32))
    got2 = host(freq)
    assert np.allclose(got2[0, :, :nu], got[0, :, :nu] * np.float32(0.5), rtol=0, atol=0)
    assert np.array_equal(got2[0, :, nu:], f0[0, :, nu:])
