"""C ABI on the host: symbols, partition arithmetic, workspace sizing, argument validation.

No GPU is used.  Every call below either is host-only (partition, workspace
size, status strings) or carries an argument error that the library must
reject before its first HIP call; the fake device pointers are never
dereferenced.  (A call with valid arguments is made only in the E_DEVICE test,
which is skipped wherever a GPU is visible.)
"""
import ctypes
import os
import re

import pytest

from oracle import infllm_oracle as O
from paper_2402_04617_amd import infllm as F

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x7F0000001000  # 16-byte aligned, never dereferenced


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(F._LIB_PATH):
        from paper_2402_04617_amd.build import build
        build()
    return F.lib()


def header_functions():
    txt = open(os.path.join(ROOT, "include", "infllm.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(infllm_\w+)\s*\(", txt)))


def test_exports_every_declared_symbol(L):
    names = header_functions()
    assert len(names) >= 11
    for n in names:
        assert hasattr(L, n), n
    assert sorted(F.EXPORTS) == names


def test_status_strings(L):
    for c in range(8):
        assert L.infllm_status_string(c)
    assert b"unknown" in L.infllm_status_string(99)


def P(**kw):
    base = dict(n_q_heads=32, n_kv_heads=8, head_dim=128, n_init=128, n_local=4096, block_size=128,
                n_repr=4, topk=32, dtype="bf16", sm_scale=1.0)
    base.update(kw)
    return F.params(**base)


def test_partition_matches_oracle(L):
    for l_I, l_L, l_bs in ((128, 4096, 128), (16, 256, 32), (0, 5, 3), (7, 1, 1)):
        p = P(n_init=l_I, n_local=l_L, block_size=l_bs, n_repr=1)
        op = O.Params(32, 8, 128, l_I, l_L, l_bs, 1, 32)
        for past in list(range(0, l_I + l_L + 5 * l_bs + 3)) + [131072, 1 << 20]:
            got = F.infllm_partition(p, past)
            exp = O.partition(past, op)
            assert got == (exp.n_init, exp.n_units, exp.local_begin), (past, got, exp)


def test_partition_errors(L):
    n0, n1, n2 = ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int64()
    assert L.infllm_partition(None, 5, ctypes.byref(n0), ctypes.byref(n1), ctypes.byref(n2)) == 1
    assert L.infllm_partition(ctypes.byref(P()), -1, ctypes.byref(n0), ctypes.byref(n1), ctypes.byref(n2)) == 2
    assert L.infllm_partition(ctypes.byref(P()), 5, None, ctypes.byref(n1), ctypes.byref(n2)) == 1


@pytest.mark.parametrize("kw,code", [
    (dict(n_kv_heads=7), 2), (dict(n_q_heads=0), 2), (dict(head_dim=96), 4), (dict(head_dim=0), 2),
    (dict(n_local=0), 2), (dict(block_size=0), 2), (dict(block_size=512, n_repr=4), 4),
    (dict(n_repr=0), 2), (dict(n_repr=129), 2), (dict(topk=-1), 2), (dict(n_init=-1), 2),
    (dict(sm_scale=float("inf")), 2), (dict(sm_scale=0.0), 2), (dict(sm_scale=-1.0), 2),
])
def test_param_validation(L, kw, code):
    p = P(**kw)
    n0, n1, n2 = ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int64()
    assert L.infllm_partition(ctypes.byref(p), 100, ctypes.byref(n0), ctypes.byref(n1), ctypes.byref(n2)) == code
    assert L.infllm_workspace_bytes(ctypes.byref(p), 1, 512) == 0
    assert L.infllm_attend_workspace_bytes(ctypes.byref(p), 1, 512) == 0


def test_workspace_bytes(L):
    p = P()
    ws = L.infllm_workspace_bytes(ctypes.byref(p), 1, 512)
    rows = 32 * 512
    row_bytes = 2 * 128 + 8  # bf16 inputs: an fp16 partial row, its lse and its exponent
    assert ws >= 2 * rows * row_bytes and ws % 256 == 0
    # decode: room for the most key parts any batch can use, one per 256 keys of the bounded key
    # count l_I + k_m*l_bs + l_L + l_bs - 1 + 1
    wsd = L.infllm_workspace_bytes(ctypes.byref(p), 16, 1)
    assert L.infllm_attend_workspace_bytes(ctypes.byref(p), 16, 1) == wsd
    assert L.infllm_attend_workspace_bytes(ctypes.byref(p), 1, 512) == ws
    nv = 128 + 32 * 128 + 4096 + 127 + 1
    assert wsd >= (nv // 256) * 16 * 32 * row_bytes


def mem(**kw):
    base = dict(batch=1, capacity=1 << 17, k=FAKE, v=FAKE, max_units=2048, repr_idx=FAKE,
                unit_ksum=FAKE, qprefix=FAKE, rpart=FAKE, ring=4096 + 128 + 2 * 512 + 1)
    base.update(kw)
    return F.Memory(**base)


def test_append_validation(L):
    p, m = P(), mem()
    f = L.infllm_append
    bp, bm = ctypes.byref(p), ctypes.byref(m)
    assert f(None, bm, FAKE, 512 * 128, None, None, 0, 512, 0, None) == 1
    assert f(bp, None, FAKE, 512 * 128, None, None, 0, 512, 0, None) == 1
    assert f(bp, bm, None, 512 * 128, None, None, 0, 512, 0, None) == 1
    assert f(bp, bm, FAKE, 100, None, None, 0, 512, 0, None) == 2               # head stride < n_q*D
    assert f(bp, bm, FAKE, 512 * 128, FAKE, None, 512 * 128, 512, 0, None) == 1  # k without v
    assert f(bp, bm, FAKE, 512 * 128, FAKE, FAKE, 512 * 128 + 1, 512, 0, None) == 2  # misaligned stride
    assert f(bp, bm, FAKE, 512 * 128, FAKE + 2, FAKE, 512 * 128, 512, 0, None) == 2  # misaligned ptr
    assert f(bp, bm, FAKE, 512 * 128, None, None, 0, 512, (1 << 17) - 100, None) == 3  # past capacity
    small = mem(ring=512)
    assert f(bp, ctypes.byref(small), FAKE, 512 * 128, None, None, 0, 512, 0, None) == 2  # ring <= n_q
    noq = mem(qprefix=None)
    assert f(bp, ctypes.byref(noq), FAKE, 512 * 128, None, None, 0, 512, 0, None) == 1
    nor = mem(rpart=None)
    assert f(bp, ctypes.byref(nor), FAKE, 512 * 128, None, None, 0, 512, 0, None) == 1
    assert f(bp, bm, FAKE, 512 * 128, None, None, 0, -1, 0, None) == 2
    # streaming past l_L: the ring must keep the running sum of token p - l_L (ring >= l_L + n_q)
    short = mem(ring=4096 + 511)
    assert f(bp, ctypes.byref(short), FAKE, 512 * 128, None, None, 0, 512, 10000, None) == 3
    # a token inside the chunk (l_L < n_q) needs the chunk's keys
    p2 = P(n_local=256)
    assert f(ctypes.byref(p2), bm, FAKE, 512 * 128, None, None, 0, 512, 10000, None) == 1


def test_build_validation(L):
    p, m = P(), mem()
    f = L.infllm_build_units
    bp, bm = ctypes.byref(p), ctypes.byref(m)
    # unit 0 covers [128, 256): its last window ends at 255 + 4096, so it needs past_len >= 4352
    assert f(bp, bm, 0, 1, 4351, None, None) == 3
    assert f(bp, bm, 0, 2, 4479, None, None) == 3
    assert f(bp, bm, 2040, 16, 1 << 17, None, None) == 3     # beyond max_units
    assert f(bp, bm, -1, 1, 10000, None, None) == 2
    # ring too short for the oldest slot: unit 0 starts at 128, ring holds [past-ring, past)
    assert f(bp, bm, 0, 1, 128 + 5249 + 123, None, None) == 3
    nou = mem(unit_ksum=None)
    assert f(bp, ctypes.byref(nou), 0, 1, 4352, None, None) == 1
    nor = mem(rpart=None)
    assert f(bp, ctypes.byref(nor), 0, 1, 4352, None, None) == 1
    assert f(bp, bm, 0, 0, 0, None, None) == 0  # nothing to build: no device needed


def test_score_validation(L):
    p, m = P(), mem()
    f = L.infllm_score_units
    bp, bm = ctypes.byref(p), ctypes.byref(m)
    assert f(bp, bm, FAKE, 512 * 128, 512, 4096, FAKE, FAKE, 1 << 20, None) == 3   # n_units > max_units
    assert f(bp, bm, FAKE, 512 * 128, 512, 100, None, FAKE, 1 << 20, None) == 1
    assert f(bp, bm, FAKE, 512 * 128, 512, 100, FAKE, None, 1 << 20, None) == 1
    assert f(bp, bm, FAKE, 512 * 128, 512, 100, FAKE, FAKE, 16, None) == 5          # workspace
    assert f(bp, bm, FAKE, 512 * 128, 512, 0, None, None, 0, None) == 0             # no units: no-op


def test_topk_validation(L):
    f = L.infllm_select_topk
    assert f(-1, FAKE, 10, 4, FAKE, None) == 2
    assert f(8, FAKE, 10, 4, None, None) == 1
    assert f(8, None, 10, 4, FAKE, None) == 1
    assert f(0, None, 10, 4, None, None) == 0
    assert f(8, None, 10, 0, None, None) == 0


def test_attend_validation(L):
    p, m = P(), mem()
    f = L.infllm_chunk_attend
    bp, bm = ctypes.byref(p), ctypes.byref(m)
    S = 512 * 128
    assert f(bp, bm, FAKE, S, 512, 1 << 17, FAKE, 32, FAKE, S, None, FAKE, 1 << 30, None) == 3  # past+n_q > cap
    assert f(bp, bm, None, S, 512, 8192, FAKE, 32, FAKE, S, None, FAKE, 1 << 30, None) == 1
    assert f(bp, bm, FAKE, S, 512, 8192, None, 32, FAKE, S, None, FAKE, 1 << 30, None) == 1     # idx needed
    assert f(bp, bm, FAKE, S, 512, 8192, FAKE, 32, None, S, None, FAKE, 1 << 30, None) == 1
    assert f(bp, bm, FAKE, S - 8, 512, 8192, FAKE, 32, FAKE, S, None, FAKE, 1 << 30, None) == 2
    assert f(bp, bm, FAKE, S, 512, 8192, FAKE, -1, FAKE, S, None, FAKE, 1 << 30, None) == 2
    parts = ctypes.c_int32()
    assert L.infllm_attend_partial(bp, bm, FAKE, S, 512, 8192, FAKE, 32, FAKE, S, None, FAKE, 1 << 30,
                                   None, None) == 1
    assert L.infllm_lse_merge(bp, 1, 512, 1, FAKE, 1 << 30, FAKE, S, None, None) == 2  # one part: nothing to merge
    assert L.infllm_lse_merge(bp, 1, 512, 4, FAKE, 100, FAKE, S, None, None) == 5
    del parts


def test_step_validation(L):
    p, m = P(), mem()
    f = L.infllm_step
    bp, bm = ctypes.byref(p), ctypes.byref(m)
    S = 512 * 128
    # units_built beyond what the partition allows
    assert f(bp, bm, FAKE, S, None, None, 0, 512, 8192, 100, FAKE, FAKE, FAKE, S, None, FAKE, 1 << 30, None) == 2
    # scores missing while units exist
    assert f(bp, bm, FAKE, S, None, None, 0, 512, 8192, 31, None, FAKE, FAKE, S, None, FAKE, 1 << 30, None) == 1


def test_remap_validation(L):
    """Positional remap: frequencies must be finite and non-negative; the rotated-key store is
    required; memory keys and local keys take separate parts, so attention with I or units
    present needs a workspace; the workspace size leaves room for two parts."""
    S = 512 * 128
    good = F.rope_frequencies(128)
    m = mem()
    for bad in (float("nan"), float("inf"), -1e-3):
        f = list(good)
        f[7] = bad
        p = P(rope_inv_freq=f)
        n0, n1, n2 = ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int64()
        assert L.infllm_partition(ctypes.byref(p), 100, ctypes.byref(n0), ctypes.byref(n1), ctypes.byref(n2)) == 2
    p = P(rope_inv_freq=good)
    bp = ctypes.byref(p)
    # k_rot missing
    assert L.infllm_append(bp, ctypes.byref(m), FAKE, S, FAKE, FAKE, S, 512, 0, None) == 1
    assert L.infllm_chunk_attend(bp, ctypes.byref(m), FAKE, S, 512, 8192, FAKE, 32, FAKE, S, None, FAKE,
                                 1 << 30, None) == 1
    mr = mem(k_rot=FAKE + 8)
    assert L.infllm_append(bp, ctypes.byref(mr), FAKE, S, FAKE, FAKE, S, 512, 0, None) == 2  # misaligned
    mr = mem(k_rot=FAKE)
    bm = ctypes.byref(mr)
    # no workspace while memory keys exist
    assert L.infllm_chunk_attend(bp, bm, FAKE, S, 512, 8192, FAKE, 32, FAKE, S, None, None, 0, None) == 5
    # a one-part workspace is not enough either
    row = 2 * 128 + 8
    assert L.infllm_chunk_attend(bp, bm, FAKE, S, 512, 8192, FAKE, 32, FAKE, S, None, FAKE,
                                 32 * 512 * row, None) == 5
    assert L.infllm_workspace_bytes(bp, 1, 1) >= 2 * 32 * row
    pd = P(rope_inv_freq=good, n_init=0, n_local=64, block_size=16, topk=2)
    assert L.infllm_workspace_bytes(ctypes.byref(pd), 1, 1) >= 2 * 32 * row


def test_step_varlen_validation(L):
    """Variable-length steps: host arrays required, at most 64 sequences, every sequence validated
    as its own step (its own capacity and unit checks) before anything runs."""
    p = P()
    S = 512 * 128
    m = mem(batch=3)
    f = L.infllm_step_varlen
    pl = (ctypes.c_int64 * 3)(8192, 100, 20000)
    ub = (ctypes.c_int32 * 3)(31, 0, 100)
    bp, bm = ctypes.byref(p), ctypes.byref(m)
    args = lambda pl_, ub_: (bp, bm, FAKE, S, None, None, 0, 1, pl_, ub_, FAKE, FAKE, FAKE, 128, None, FAKE,  # noqa
                            1 << 30, None)
    assert f(*args(None, ub)) == 1
    assert f(*args(pl, None)) == 1
    big = mem(batch=65)
    assert f(bp, ctypes.byref(big), FAKE, S, None, None, 0, 1, pl, ub, FAKE, FAKE, FAKE, 128, None, FAKE, 1 << 30,
             None) == 4
    bad = (ctypes.c_int32 * 3)(31, 1, 100)      # sequence 1 has no unit to have built
    assert f(*args(pl, bad)) == 2
    far = (ctypes.c_int64 * 3)(8192, 100, (1 << 17))  # sequence 2 past the capacity
    assert f(*args(far, ub)) == 3
    neg = (ctypes.c_int64 * 3)(8192, -1, 20000)
    assert f(*args(neg, ub)) == 2


def test_mean_repr_validation(L):
    """Mean representation: an unknown mode is a shape error; the query ring, rpart and repr_idx
    are not needed (their absence is not reported, the call reaches the device check)."""
    p = P()
    p.repr_mode = 5
    n0, n1, n2 = ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int64()
    assert L.infllm_partition(ctypes.byref(p), 100, ctypes.byref(n0), ctypes.byref(n1), ctypes.byref(n2)) == 2
    pm = P(repr_mode="mean")
    m = mem(qprefix=None, rpart=None, repr_idx=None, ring=0)
    bp, bm = ctypes.byref(pm), ctypes.byref(m)
    S = 512 * 128
    # argument errors are still found first
    assert L.infllm_append(bp, bm, FAKE, 100, None, None, 0, 512, 0, None) == 2
    assert L.infllm_build_units(bp, bm, 2040, 16, 1 << 17, None, None) == 3
    # the token representation does need them
    pt = P()
    assert L.infllm_append(ctypes.byref(pt), bm, FAKE, S, None, None, 0, 512, 0, None) == 1
    assert L.infllm_build_units(ctypes.byref(pt), bm, 0, 1, 4352, None, None) == 1


def test_unit_mass_validation(L):
    p, m = P(), mem()
    f = L.infllm_unit_mass
    bp, bm = ctypes.byref(p), ctypes.byref(m)
    past = 1 << 16
    ok = (bp, bm, FAKE, 512 * 128, 512, past, FAKE, 32, FAKE, 0.1, FAKE, FAKE, None)

    def call(**kw):
        a = list(ok)
        names = ["p", "m", "q", "qs", "n_q", "past", "idx", "k", "lse", "decay", "mass", "freq", "stream"]
        for key, val in kw.items():
            a[names.index(key)] = val
        return f(*a)
    assert call(p=None) == 1
    assert call(m=None) == 1
    assert call(idx=None) == 1
    assert call(mass=None) == 1
    assert call(lse=None) == 1
    assert call(q=None) == 1
    assert call(qs=100) == 2                   # head stride < n_q*D
    assert call(n_q=-1) == 2
    assert call(k=-1) == 2
    assert call(decay=-0.5) == 2
    assert call(decay=float("nan")) == 2
    assert call(past=(1 << 17) - 100) == 3     # past + n_q beyond capacity
    assert call(k=1025) == 4                   # more lookup slots than the kernel stages
    few = mem(max_units=10)
    assert call(m=ctypes.byref(few)) == 3      # freq rows shorter than the built units


@pytest.mark.skipif(os.path.exists("/dev/kfd") and os.access("/dev/kfd", os.R_OK),
                    reason="a GPU may be present; valid arguments would launch on fake pointers")
def test_valid_arguments_without_gpu_report_device_error(L):
    p, m = P(), mem()
    assert L.infllm_select_topk(8, FAKE, 10, 4, FAKE, None) == 7
    # mean representation without ring buffers: valid, so only the device check fails
    pm = P(repr_mode="mean")
    mm = mem(qprefix=None, rpart=None, repr_idx=None, ring=0)
    assert L.infllm_append(ctypes.byref(pm), ctypes.byref(mm), FAKE, 512 * 128, None, None, 0, 512, 0, None) == 7
    assert L.infllm_build_units(ctypes.byref(pm), ctypes.byref(mm), 0, 1, 4352, None, None) == 7
