"""Batches whose sequences sit at different past lengths (infllm_step_varlen) against the oracle (GPU).

Each sequence is first encoded alone up to its own length (infllm_step on a one-sequence view of
the batch's memory), then the whole batch steps together with per-sequence past lengths: single
tokens (decoding) and 512-token chunks.  Every sequence's scores, lookup, output and lse are
compared with the oracle's step at that sequence's own position, with the near-tie rule of the
other stream tests.
"""
import numpy as np
import pytest
import torch

from oracle import infllm_oracle as O
from paper_2402_04617_amd import infllm as F
from tests.gpu_util import check_selection, conditioned_step, dev, host, log, oparams
from tests.test_gpu_kernels import TOL, rand_inputs

pytestmark = pytest.mark.gpu


def _view(mem, b):
    """The one-sequence memory struct of sequence b of a batch allocation."""
    def ptr(t):
        return None if t is None else t[b].data_ptr()
    s = mem.struct
    return F.Memory(1, s.capacity, mem.k[b].data_ptr(), mem.v[b].data_ptr(), s.max_units, ptr(mem.repr_idx),
                    ptr(mem.unit_ksum), ptr(mem.qprefix), ptr(mem.rpart), s.ring, ptr(mem.k_rot))


def _prefill(p, mem, b, qd, kd, vd, upto, chunk, ws, esize):
    """Encode sequence b alone over [0, upto) in chunks; returns its units built."""
    S, D = qd.shape[2], qd.shape[3]
    view = _view(mem, b)
    out = torch.zeros((1, p.n_q_heads, chunk, D), dtype=qd.dtype, device="cuda")
    sc = torch.zeros(p.n_kv_heads * max(1, mem.struct.max_units), dtype=torch.float32, device="cuda")
    idx = torch.zeros((1, p.n_kv_heads, max(1, p.topk)), dtype=torch.int32, device="cuda")
    built = 0
    op = oparams(p)
    off = lambda t, past: t[b].data_ptr() + past * D * esize  # noqa: E731
    for past in range(0, upto, chunk):
        n = min(chunk, upto - past)
        F.infllm_step(p, view, off(qd, past), S * D, off(kd, past), off(vd, past), S * D, n, past, built, sc, idx,
                      out, chunk * D, None, ws)
        built = O.partition(past, op).n_units
    return built


def _run(dtype, G, Hkv, D, lI, lL, lbs, km, starts, n_q, n_steps, remap=False, mean=False, seed=61):
    rng = np.random.default_rng(seed)
    B = len(starts)
    S = max(starts) + n_steps * n_q
    f = F.rope_frequencies(D) if remap else None
    p = F.params(G * Hkv, Hkv, D, lI, lL, lbs, 4, km, dtype, sm_scale=D ** -0.5, rope_inv_freq=f,
                 repr_mode="mean" if mean else "tokens")
    op = oparams(p)
    q, k, v = rand_inputs(rng, G * Hkv, Hkv, S, D, dtype, qk_std=1.0, B=B)
    chunk = 512
    max_units = max(1, O.partition(S, op).n_units)
    mem = F.alloc_memory(p, B, S, max_units, F.recommended_ring(p, chunk))
    ws = torch.zeros(max(F.infllm_workspace_bytes(p, B, chunk), F.infllm_workspace_bytes(p, B, 1)),
                     dtype=torch.uint8, device="cuda")
    qd, kd, vd = dev(q, dtype), dev(k, dtype), dev(v, dtype)
    esize = 2 if dtype == "bf16" else 4
    built = [_prefill(p, mem, b, qd, kd, vd, starts[b], chunk, ws, esize) for b in range(B)]
    so = O.StreamOracle(q, k, v, op)
    out = torch.zeros((B, G * Hkv, n_q, D), dtype=qd.dtype, device="cuda")
    lse = torch.zeros((B, G * Hkv, n_q), dtype=torch.float32, device="cuda")
    scores = torch.zeros((B, Hkv, max_units), dtype=torch.float32, device="cuda")
    idx = torch.zeros((B, Hkv, max(1, km)), dtype=torch.int32, device="cuda")
    n_checked = n_tie = 0
    for t in range(n_steps):
        pasts = [st + t * n_q for st in starts]
        # the batch's current tokens, gathered from each sequence's own position
        gather = lambda x: torch.stack([x[b, :, pasts[b]:pasts[b] + n_q] for b in range(B)]).contiguous()  # noqa
        qs, ks, vs = gather(qd), gather(kd), gather(vd)
        log(f"[varlen] {dtype} remap={remap} mean={mean} step {t} pasts={pasts} n_q={n_q}")
        F.infllm_step_varlen(p, mem.struct, qs, n_q * D, ks, vs, n_q * D, n_q, pasts, built, scores, idx, out,
                             n_q * D, lse, ws)
        built = [O.partition(pp, op).n_units for pp in pasts]
        torch.cuda.synchronize()
        go, gl, gs, gi = (host(out).astype(np.float64), host(lse).astype(np.float64),
                          host(scores).astype(np.float64), host(idx).astype(np.int64))
        ridx = host(mem.repr_idx)
        for b in range(B):
            r = conditioned_step(so, b, pasts[b], n_q, ridx[b])
            nu = r["n_units"]
            for g in range(Hkv):
                es = r["scores"][g]
                if nu:
                    scale = max(np.abs(es).max(), np.sqrt(np.mean(es ** 2)))
                    tol = 1e-5 if dtype == "f32" else 1e-3
                    assert np.abs(gs[b, g, :nu] - es).max() <= tol * scale, (t, b, g)
                same = check_selection(gi[b, g], r["idx"][g], es, km)
                hs = slice(g * G, (g + 1) * G)
                if same:
                    assert np.abs(go[b, hs] - r["out"][hs]).max() <= TOL[dtype], (t, b, g)
                    lt = 1e-4 if dtype == "f32" else (1e-2 if remap else 1e-3)
                    assert np.abs(gl[b, hs] - r["lse"][hs]).max() <= lt, (t, b, g)
                    n_checked += 1
                else:
                    n_tie += 1
    assert n_checked > 0 and n_tie <= max(1, n_checked // 20), (n_checked, n_tie)


def test_varlen_decode_bf16():
    # four sequences at different depths: no units yet, a few, many (a unit evicted during the run)
    _run("bf16", 4, 2, 128, 128, 1024, 128, 8, [700, 1290, 3000, 5121], n_q=1, n_steps=4)


def test_varlen_decode_bf16_remap_mean():
    _run("bf16", 4, 2, 128, 64, 512, 64, 6, [300, 1500, 2600], n_q=1, n_steps=3, remap=True, mean=True)


def test_varlen_decode_bf16_remap():
    _run("bf16", 8, 1, 64, 16, 256, 32, 5, [100, 900, 2000], n_q=1, n_steps=3, remap=True)


def test_varlen_chunks_bf16():
    _run("bf16", 4, 2, 128, 128, 1024, 128, 8, [0, 1024, 2560], n_q=512, n_steps=2)


def test_varlen_chunks_long_rows_bf16():
    # 16-token units: the deepest sequence's score rows pass 1,024 units (1,178 and more), so the
    # attention selects with sixteen keys per thread, for a batch that also holds a sequence with
    # a short row (490 units) and one with no units yet
    _run("bf16", 4, 2, 128, 128, 1024, 16, 8, [0, 9000, 20000], n_q=512, n_steps=2)


def test_varlen_decode_max_batch():
    # the largest batch a variable-length step takes: 64 sequences, 50 to 1,499 tokens deep
    _run("bf16", 2, 1, 64, 8, 64, 16, 3, [50 + 23 * i for i in range(64)], n_q=1, n_steps=2)


def test_varlen_decode_f32():
    _run("f32", 2, 1, 64, 16, 256, 32, 4, [200, 640, 1100], n_q=1, n_steps=3)
