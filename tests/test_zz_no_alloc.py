"""The allocation-free attention entry point against the workspace one (GPU).

infllm_chunk_attend_noalloc puts the split-key partials in a device array the
library owns instead of a caller workspace.  Called through the C ABI twice in a
row (the second call smaller, so it reads what the first left behind only if it
is wrong), it must reproduce infllm_chunk_attend exactly when both use the same
number of key parts, and the oracle's output within the bf16 / float32 bars.
Calls that need more than the array holds are rejected before anything runs.
"""
import ctypes

import numpy as np
import pytest
import torch

from oracle import infllm_oracle as O
from paper_2402_04617_amd import infllm as F
from tests.gpu_util import Layer, dev, host, log, oparams
from tests.test_gpu_kernels import TOL, rand_inputs

pytestmark = pytest.mark.gpu

CASES = [
    # dtype, G, Hkv, D, lI, lL, lbs, k_m, past, n_q, B, remap
    ("bf16", 4, 8, 128, 128, 4096, 128, 32, 20000, 512, 1, False),  # the 128K step shape, 4 key parts
    ("bf16", 4, 2, 128, 128, 512, 128, 4, 3000, 77, 1, False),      # smaller, ragged rows
    ("bf16", 4, 2, 128, 128, 4096, 128, 32, 13000, 1, 3, False),    # decode
    ("bf16", 4, 2, 128, 5, 300, 16, 7, 2000, 200, 1, True),         # positional remap (two or more parts)
    ("f32", 2, 1, 64, 16, 256, 32, 4, 1000, 64, 1, False),
]


def _run(case, seed):
    dtype, G, Hkv, D, lI, lL, lbs, km, past, n_q, B, remap = case
    rng = np.random.default_rng(seed)
    S = past + n_q
    p = F.params(G * Hkv, Hkv, D, lI, lL, lbs, 2, km, dtype, sm_scale=0.9,
                 rope_inv_freq=F.rope_frequencies(D, 10000.0) if remap else None)
    op = oparams(p)
    q, k, v = rand_inputs(rng, G * Hkv, Hkv, S, D, dtype, B=B)
    nu = O.partition(past, op).n_units
    sel = np.full((B, Hkv, km), -1, dtype=np.int64)
    for b in range(B):
        for g in range(Hkv):
            c = np.sort(rng.choice(nu, min(km, nu), replace=False)) if nu else np.zeros(0, np.int64)
            sel[b, g, :c.size] = c
    # with the remap the whole sequence is appended in one call (the rotated keys the
    # attention reads for L and X): the ring then holds l_L + S slots
    L = Layer(p, B, S, chunk=n_q, ring=(S + lL + 1) if remap else n_q + 1)
    L.mem.k.copy_(dev(k, dtype))
    L.mem.v.copy_(dev(v, dtype))
    if remap:
        F.infllm_append(p, L.mem.struct, dev(q, dtype), S * D, dev(k, dtype), dev(v, dtype), S * D, S, 0)
    qd = dev(q[:, :, past:past + n_q], dtype)
    idx = torch.from_numpy(sel.astype(np.int32)).cuda()
    outs = []
    for noalloc in (False, True):
        out = torch.zeros((B, G * Hkv, n_q, D), dtype=L.dt, device="cuda")
        lse = torch.zeros((B, G * Hkv, n_q), dtype=torch.float32, device="cuda")
        log(f"[noalloc] {case} noalloc={noalloc}")
        if noalloc:
            F.infllm_chunk_attend_noalloc(p, L.mem.struct, qd, n_q * D, n_q, past, idx, km, out, n_q * D, lse)
        else:
            F.infllm_chunk_attend(p, L.mem.struct, qd, n_q * D, n_q, past, idx, km, out, n_q * D, lse, L.ws)
        torch.cuda.synchronize()
        outs.append((out, lse))
    (o1, l1), (o2, l2) = outs
    assert torch.equal(o1, o2) and torch.equal(l1, l2), case
    got_o, got_l = host(o2).astype(np.float64), host(l2).astype(np.float64)
    for b in range(B):
        eo, el = O.attend(q[b, :, past:past + n_q], k[b], v[b], past, sel[b], op)
        assert np.abs(got_o[b] - eo).max() <= TOL[dtype], case
        assert np.abs(got_l[b] - el).max() <= (1e-2 if remap else 1e-3 if dtype == "bf16" else 1e-4), case


@pytest.mark.parametrize("first,second", [(0, 1), (0, 2), (3, 1), (4, 1)])
def test_noalloc_matches_workspace_entry_point(first, second):
    """Two calls in a row, the second with a smaller input."""
    _run(CASES[first], seed=21)
    _run(CASES[second], seed=22)


def test_noalloc_rejects_beyond_scratch():
    """A call whose fewest key parts exceed the scratch array is refused before anything runs."""
    G, Hkv, D = 4, 8, 128
    p = F.params(G * Hkv, Hkv, D, 128, 4096, 128, 4, 32, "bf16", rope_inv_freq=F.rope_frequencies(D))
    n_q, B = 8192, 2  # remap: two parts of 2*32*8192 rows of 264 bytes = 138 MiB > 32 MiB
    L = Layer(p, B, 20000 + n_q, chunk=1, ring=2)
    out = torch.zeros((B, G * Hkv, n_q, D), dtype=torch.bfloat16, device="cuda")
    q = torch.zeros((B, G * Hkv, n_q, D), dtype=torch.bfloat16, device="cuda")
    idx = torch.zeros((B, Hkv, 32), dtype=torch.int32, device="cuda")
    st = F.lib().infllm_chunk_attend_noalloc(ctypes.byref(p), ctypes.byref(L.mem.struct), q.data_ptr(), n_q * D, n_q,
                                             20000, idx.data_ptr(), 32, out.data_ptr(), n_q * D, None,
                                             torch.cuda.current_stream().cuda_stream)
    assert st == 5  # INFLLM_E_WORKSPACE
    assert not out.any()
