"""Parity of the positional remap (Section 3.2, "Positional Encoding") against the oracle (GPU).

q and k arrive without positions; the library rotates them: keys of I and of the
memory units unrotated and met by queries turned by R(l_L), keys of L and X at
their own positions (stored rotated in k_rot by the append), representative
scores at true positions, unit relevance at the memory distance.  Expected
values come from oracle/ with the same rotary frequencies.  Bars as elsewhere:
bf16 outputs within 2e-2 max-abs and fp32 within 1e-4 of the float64 oracle;
rotated keys within the rounding of their dtype.  The bf16 lse bar is 1e-2
here (1e-3 without the remap): the rotated query and key enter the matrix cores
rounded to bf16, which moves each logit by up to sm_scale * 2^-8 * sum_d |q_d k_d|
(about 2e-3 for one logit at these input scales, up to ~3e-2 in the worst
case), and a row with few visible keys passes that straight to its lse.
"""
import numpy as np
import pytest
import torch

from oracle import infllm_oracle as O
from paper_2402_04617_amd import infllm as F
from tests.gpu_util import Layer, check_selection, conditioned_step, dev, host, log, oparams
from tests.test_gpu_kernels import TOL, rand_inputs

pytestmark = pytest.mark.gpu

LSE_TOL = {"bf16": 1e-2, "f32": 1e-4}


def freqs(D, base=10000.0):
    # base 10^4 makes theta_0 = 1 rad per position: every pair turns visibly between positions
    return F.rope_frequencies(D, base)


def rounded(x, dtype):
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).float().numpy()
    return x.astype(np.float32)


# ------------------------------------------------------------------ append: k_rot and the rotated ring
@pytest.mark.parametrize("dtype,G,D", [("bf16", 4, 128), ("f32", 2, 64), ("bf16", 1, 64)])
def test_append_remap_store_and_ring(dtype, G, D):
    rng = np.random.default_rng(41)
    Hkv, B, S = 2, 2, 300
    f = freqs(D)
    p = F.params(G * Hkv, Hkv, D, 4, 16, 8, 2, 2, dtype, rope_inv_freq=f)
    q, k, v = rand_inputs(rng, G * Hkv, Hkv, S, D, dtype, qk_std=1.0, B=B)
    L = Layer(p, B, S, chunk=40, ring=97)
    qd, kd, vd = dev(q, dtype), dev(k, dtype), dev(v, dtype)
    es = L.esize
    past = 0
    for n in (40, 1, 33, 17, 40, 3, 8, 5):
        log(f"[remap append] {dtype} G={G} D={D} past={past} n={n}")
        F.infllm_append(p, L.mem.struct, qd.data_ptr() + past * D * es, S * D, kd.data_ptr() + past * D * es,
                        vd.data_ptr() + past * D * es, S * D, n, past)
        past += n
    torch.cuda.synchronize()
    assert np.array_equal(host(L.mem.k)[:, :, :past], k[:, :, :past])
    assert np.array_equal(host(L.mem.v)[:, :, :past], v[:, :, :past])
    pos = np.arange(past)
    kr = O.rotate(k[:, :, :past], pos, f)
    got = host(L.mem.k_rot)[:, :, :past].astype(np.float64)
    ulp = 2.0 ** -8 if dtype == "bf16" else 2.0 ** -22
    assert np.all(np.abs(got - kr) <= ulp * np.abs(kr) + 1e-5), np.abs(got - kr).max()
    ring = host(L.mem.qprefix)
    qt = O.rotate(q.astype(np.float64).reshape(B, Hkv, G, S, D).sum(axis=2)[:, :, :past], pos, f)
    pref = np.cumsum(qt, axis=2)
    for t in range(max(0, past - 97), past):
        assert np.allclose(ring[:, :, t % 97], pref[:, :, t], rtol=1e-5, atol=1e-4), t


# ------------------------------------------------------------------ attention over both regions
REMAP_ATTEND = [
    # dtype, G, Hkv, D, l_I, l_L, l_bs, k_m, past, n_q, batch
    ("bf16", 4, 2, 128, 128, 512, 128, 4, 3000, 512, 1),    # memory length a multiple of the tile
    ("bf16", 4, 2, 128, 5, 300, 16, 7, 2000, 200, 1),       # memory ends inside a tile: both sides mask it
    ("bf16", 4, 8, 128, 128, 4096, 128, 32, 20000, 512, 1),  # real shape
    ("bf16", 2, 2, 64, 3, 100, 24, 5, 900, 77, 2),          # D = 64, ragged rows, batch 2
    ("bf16", 4, 2, 128, 128, 4096, 128, 32, 0, 512, 1),     # first chunk: no memory keys at all
    ("bf16", 4, 2, 128, 128, 4096, 128, 32, 100, 300, 1),   # past inside I: memory is I alone
    ("bf16", 4, 2, 128, 128, 4096, 128, 32, 13000, 1, 3),   # decode
    ("bf16", 8, 2, 64, 16, 300, 32, 5, 1000, 1, 2),         # decode, G = 8, D = 64
    ("bf16", 1, 3, 64, 7, 333, 24, 6, 1200, 1, 1),          # decode, G = 1, memory ends mid-tile
    ("bf16", 3, 1, 128, 16, 300, 32, 5, 1000, 1, 1),        # decode shape on the matrix-core kernel
    ("f32", 2, 1, 64, 16, 256, 32, 4, 1000, 64, 1),
    ("f32", 4, 2, 128, 5, 100, 8, 6, 700, 37, 2),
    ("f32", 2, 1, 64, 16, 256, 32, 4, 1000, 1, 1),
]


def _remap_attend(case, seed=43):
    dtype, G, Hkv, D, lI, lL, lbs, km, past, n_q, B = case
    rng = np.random.default_rng(seed)
    S = past + n_q
    f = freqs(D)
    p = F.params(G * Hkv, Hkv, D, lI, lL, lbs, 2, km, dtype, sm_scale=0.9, rope_inv_freq=f)
    op = oparams(p)
    q, k, v = rand_inputs(rng, G * Hkv, Hkv, S, D, dtype, qk_std=0.3, B=B)
    nu = O.partition(past, op).n_units
    sel = np.full((B, Hkv, km), -1, dtype=np.int64)
    for b in range(B):
        for g in range(Hkv):
            c = np.sort(rng.choice(nu, min(km, nu), replace=False)) if nu else np.zeros(0, np.int64)
            sel[b, g, :c.size] = c
    L = Layer(p, B, S, chunk=n_q, ring=n_q + 1)
    L.mem.k.copy_(dev(k, dtype))
    L.mem.v.copy_(dev(v, dtype))
    # the rotated keys as the append stores them (rounded once to the dtype)
    L.mem.k_rot.copy_(dev(rounded(O.rotate(k, np.arange(S), f), dtype), dtype))
    qd = dev(q[:, :, past:past + n_q], dtype)
    idx = torch.from_numpy(sel.astype(np.int32)).cuda()
    out = torch.zeros((B, G * Hkv, n_q, D), dtype=L.dt, device="cuda")
    lse = torch.zeros((B, G * Hkv, n_q), dtype=torch.float32, device="cuda")
    log(f"[remap attend] {case}")
    parts = F.infllm_attend_partial(p, L.mem.struct, qd, n_q * D, n_q, past, idx, km, out, n_q * D, lse, L.ws)
    if parts > 1:
        F.infllm_lse_merge(p, B, n_q, parts, L.ws, out, n_q * D, lse)
    torch.cuda.synchronize()
    got_o, got_l = host(out).astype(np.float64), host(lse).astype(np.float64)
    for b in range(B):
        eo, el = O.attend(q[b, :, past:past + n_q], k[b], v[b], past, sel[b], op)
        err = np.abs(got_o[b] - eo).max()
        assert err <= TOL[dtype], (case, b, err)
        assert np.abs(got_l[b] - el).max() <= LSE_TOL[dtype], case
    return parts


@pytest.mark.parametrize("case", REMAP_ATTEND, ids=[str(c) for c in REMAP_ATTEND])
def test_remap_attend(case):
    parts = _remap_attend(case)
    dtype, G, Hkv, D, lI, lL, lbs, km, past, n_q, B = case
    if min(lI, past) > 0:
        assert parts >= 2  # memory and local keys never share a part


# ------------------------------------------------------------------ whole steps
def _stream(p, q, k, v, steps, check, chunk, dtype, score_rel):
    op = oparams(p)
    B, G, Hkv = q.shape[0], p.n_q_heads // p.n_kv_heads, p.n_kv_heads
    L = Layer(p, B, q.shape[2], chunk=chunk)
    qd, kd, vd = dev(q, dtype), dev(k, dtype), dev(v, dtype)
    so = O.StreamOracle(q, k, v, op)
    n_checked = n_tie = 0
    for si, (past, n) in enumerate(steps):
        L.step(qd, kd, vd, past, n)
        if si not in check:
            continue
        log(f"[remap stream] step={si} past={past} n={n}")
        nu = O.partition(past, op).n_units
        got = L.capture(n, nu)
        ridx = host(L.mem.repr_idx)
        for b in range(B):
            r = conditioned_step(so, b, past, n, ridx[b])
            for g in range(Hkv):
                es = r["scores"][g]
                if nu:
                    scale = max(np.abs(es).max(), np.sqrt(np.mean(es ** 2)))
                    assert np.abs(got["scores"][b, g] - es).max() <= score_rel * scale, (si, b, g)
                same = check_selection(got["idx"][b, g], r["idx"][g], es, p.topk)
                hs = slice(g * G, (g + 1) * G)
                if same:
                    err = np.abs(got["out"][b, hs] - r["out"][hs]).max()
                    assert err <= TOL[dtype], (si, b, g, err)
                    assert np.abs(got["lse"][b, hs] - r["lse"][hs]).max() <= LSE_TOL[dtype], (si, b, g)
                    n_checked += 1
                else:
                    n_tie += 1
    assert n_checked > 0 and n_tie <= max(1, n_checked // 20), (n_checked, n_tie)


def test_remap_stream_f32_every_step():
    rng = np.random.default_rng(44)
    D, S, chunk = 64, 1100, 64
    p = F.params(2, 1, D, 16, 256, 32, 4, 4, "f32", sm_scale=1.0, rope_inv_freq=freqs(D))
    q, k, v = rand_inputs(rng, 2, 1, S, D, "f32", qk_std=0.5)
    steps = [(s, min(chunk, S - s)) for s in range(0, S, chunk)]
    _stream(p, q, k, v, steps, set(range(len(steps))), chunk, "f32", 1e-5)


def test_remap_stream_bf16_chunks_then_decode():
    """bf16 chunks of 512 (matrix-core attention, fused unit construction), then single-token steps
    (the decode kernel), Llama-3 rotary frequencies."""
    rng = np.random.default_rng(45)
    D, chunk = 128, 512
    S0 = 9 * chunk
    S = S0 + 6
    p = F.params(8, 2, D, 128, 1024, 128, 4, 8, "bf16", sm_scale=D ** -0.5,
                 rope_inv_freq=F.rope_frequencies(D))
    q, k, v = rand_inputs(rng, 8, 2, S, D, "bf16", qk_std=1.0)
    steps = [(s, chunk) for s in range(0, S0, chunk)] + [(S0 + i, 1) for i in range(6)]
    _stream(p, q, k, v, steps, {2, 5, 8, 9, 12, 14}, chunk, "bf16", 1e-3)
