"""Seeded input generator: determinism, piecewise drawing, rounding, planted structure (CPU)."""
import numpy as np
import torch

from oracle import infllm_oracle as O
from workload import WORKLOADS, Synth, bf16_bits_to_f32, f32_to_bf16_bits


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 3,
                        np.array([0.0, -0.0, 1.0, -1.0, 1e-30, 3.4e38, 1.00390625, 1.01171875],
                                 dtype=np.float32)])
    ours = f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    assert np.array_equal(bf16_bits_to_f32(ours), torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_deterministic_and_piecewise():
    wl = WORKLOADS["mistral7b-32k"]
    a, b = Synth(wl, 3), Synth(wl, 3)
    assert np.array_equal(a.q(0, 5, 1000, 3000), b.q(0, 5, 1000, 3000))
    whole = a.k(0, 2, 0, 5000)
    assert np.array_equal(whole[1234:4321], a.k(0, 2, 1234, 4321))
    assert not np.array_equal(a.v(0, 1, 0, 64), Synth(wl, 4).v(0, 1, 0, 64))
    # values are exactly representable in bf16
    x = a.q(0, 0, 0, 700)
    assert np.array_equal(x, bf16_bits_to_f32(f32_to_bf16_bits(x)))


def test_planted_structure():
    wl = WORKLOADS["tiny-2k-f32"]
    s = Synth(wl, 0)
    u = s.direction(0, 0)
    assert abs(np.linalg.norm(u) - 1) < 1e-6
    nb = s.needle_blocks(0, 0)
    assert len(nb) == wl.n_needles and len(set(nb.tolist())) == wl.n_needles
    k = s.k(0, 0, 0, wl.seq_len)
    proj = k @ u
    for j in nb:
        a = wl.n_init + int(j) * wl.block_size
        assert proj[a:a + wl.block_size].mean() > 1.5
    q = s.q(0, 1, 0, 256)
    assert (q[::8] @ u).mean() > 0.8 and abs((q[1::8] @ u).mean()) < 0.3


def test_steps_cover_sequence():
    for wl in WORKLOADS.values():
        steps = wl.step_starts()
        assert steps[0][0] == 0
        assert sum(n for _, n in steps) == wl.seq_len
        for (p0, n0), (p1, _) in zip(steps, steps[1:]):
            assert p1 == p0 + n0


def test_needles_are_looked_up_tiny():
    """Sanity (not parity): on the tiny workload the oracle selects every evicted needle
    block at every step, since every 8th query leans along the needles' direction."""
    wl = WORKLOADS["tiny-2k-f32"]
    s = Synth(wl, 0)
    q, k, v = s.full("q"), s.full("k"), s.full("v")
    p = O.Params(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.n_init, wl.n_local,
                 wl.block_size, wl.n_repr, wl.topk, 1.0)
    so = O.StreamOracle(q, k, v, p)
    needles = s.needle_blocks(0, 0)
    seen = 0
    for past, n in wl.step_starts():
        r = so.step(0, past, n)
        ev = [int(b) for b in needles if b < r["n_units"]]
        assert set(ev) <= set(r["idx"][0].tolist()), past
        seen += len(ev)
    assert seen > 0
