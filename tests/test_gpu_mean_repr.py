"""Parity of the Mean Repr unit representation (the alternative the paper evaluates in Section 4:
a unit scored by the mean of its keys) against the oracle (GPU).

In this mode the library keeps no query ring and forms no representative scores: unit
construction averages the unit's keys and scoring sums the chunk's queries itself.  Expected
values come from oracle/ with mean_repr set; bars as in the other parity tests.
"""
import numpy as np
import pytest
import torch

from oracle import infllm_oracle as O
from paper_2402_04617_amd import infllm as F
from tests.gpu_util import Layer, dev, host, log, oparams
from tests.test_gpu_kernels import rand_inputs
from tests.test_gpu_remap import _stream, freqs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype,G,D,lI,lbs", [("bf16", 4, 128, 128, 128), ("f32", 2, 64, 16, 32),
                                              ("bf16", 2, 64, 5, 24)])
def test_build_units_mean(dtype, G, D, lI, lbs):
    rng = np.random.default_rng(51)
    Hkv, B = 2, 2
    lL = 64
    n_units = 9
    S = lI + n_units * lbs + lL + 1
    p = F.params(G * Hkv, Hkv, D, lI, lL, lbs, 3, 4, dtype, repr_mode="mean")
    q, k, v = rand_inputs(rng, G * Hkv, Hkv, S, D, dtype, B=B)
    L = Layer(p, B, S, chunk=S)
    L.mem.k.copy_(dev(k, dtype))
    log(f"[mean build] {dtype} G={G} D={D} l_bs={lbs}")
    F.infllm_build_units(p, L.mem.struct, 0, n_units, S)
    torch.cuda.synchronize()
    got = host(L.mem.unit_ksum)  # [B][Hkv][D/4][max_units][4]
    got = got[:, :, :, :n_units, :].transpose(0, 1, 3, 2, 4).reshape(B, Hkv, n_units, D)
    for u in range(n_units):
        s0 = lI + u * lbs
        ref = k[:, :, s0:s0 + lbs].astype(np.float64).mean(axis=2)
        assert np.allclose(got[:, :, u], ref, rtol=1e-5, atol=1e-6), u


def test_mean_repr_stream_f32_every_step():
    rng = np.random.default_rng(52)
    D, S, chunk = 64, 1100, 64
    p = F.params(2, 1, D, 16, 256, 32, 4, 4, "f32", repr_mode="mean")
    q, k, v = rand_inputs(rng, 2, 1, S, D, "f32", qk_std=0.5)
    steps = [(s, min(chunk, S - s)) for s in range(0, S, chunk)]
    _stream(p, q, k, v, steps, set(range(len(steps))), chunk, "f32", 1e-5)


@pytest.mark.parametrize("remap", [False, True])
def test_mean_repr_stream_bf16_chunks_then_decode(remap):
    """bf16 chunks of 512 then single-token steps; with and without the positional remap."""
    rng = np.random.default_rng(53)
    D, chunk = 128, 512
    S0 = 9 * chunk
    S = S0 + 6
    p = F.params(8, 2, D, 128, 1024, 128, 4, 8, "bf16", sm_scale=D ** -0.5, repr_mode="mean",
                 rope_inv_freq=F.rope_frequencies(D) if remap else None)
    q, k, v = rand_inputs(rng, 8, 2, S, D, "bf16", qk_std=1.0)
    steps = [(s, chunk) for s in range(0, S0, chunk)] + [(S0 + i, 1) for i in range(6)]
    _stream(p, q, k, v, steps, {2, 5, 8, 9, 12, 14}, chunk, "bf16", 1e-3)
