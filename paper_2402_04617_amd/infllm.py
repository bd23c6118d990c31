"""ctypes binding of libinfllm.so (the C ABI declared in include/infllm.h).

Argument marshalling only: every function here forwards to the C entry point
of the same name, passing device pointers taken from PyTorch tensors and the
current HIP stream.  PyTorch supplies device memory and streams; all compute
runs in the library's gfx950 kernels.  Loading fails loudly when the library has
not been built, and every call raises on a non-OK status.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional, Tuple

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libinfllm.so")

INFLLM_F32 = 0
INFLLM_BF16 = 1
INFLLM_REPR_TOKENS = 0
INFLLM_REPR_MEAN = 1

STATUS = {0: "INFLLM_OK", 1: "INFLLM_E_NULL", 2: "INFLLM_E_SHAPE", 3: "INFLLM_E_RANGE",
          4: "INFLLM_E_UNSUPPORTED", 5: "INFLLM_E_WORKSPACE", 6: "INFLLM_E_LAUNCH", 7: "INFLLM_E_DEVICE"}

EXPORTS = ["infllm_partition", "infllm_workspace_bytes", "infllm_attend_workspace_bytes", "infllm_append", "infllm_build_units",
           "infllm_score_units", "infllm_select_topk", "infllm_chunk_attend", "infllm_chunk_attend_noalloc",
           "infllm_attend_partial",
           "infllm_lse_merge", "infllm_step", "infllm_step_mass", "infllm_step_varlen", "infllm_unit_mass",
           "infllm_status_string"]


class InfllmError(RuntimeError):
    def __init__(self, fn: str, code: int, text: str):
        super().__init__(f"{fn} -> {STATUS.get(code, code)}: {text}")
        self.code = code


class Params(ctypes.Structure):
    _fields_ = [("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("n_init", ctypes.c_int32), ("n_local", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("n_repr", ctypes.c_int32), ("topk", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("sm_scale", ctypes.c_float), ("rope_inv_freq", ctypes.POINTER(ctypes.c_double)),
                ("repr_mode", ctypes.c_int32)]

    @property
    def remap(self) -> bool:
        """Positional remap on (rotary frequencies given)."""
        return bool(self.rope_inv_freq)

    @property
    def mean_repr(self) -> bool:
        """Units scored by their mean key (no representative tokens, no query ring)."""
        return self.repr_mode == INFLLM_REPR_MEAN


class Memory(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("capacity", ctypes.c_int64), ("k", ctypes.c_void_p),
                ("v", ctypes.c_void_p), ("max_units", ctypes.c_int32), ("repr_idx", ctypes.c_void_p),
                ("unit_ksum", ctypes.c_void_p), ("qprefix", ctypes.c_void_p), ("rpart", ctypes.c_void_p),
                ("ring", ctypes.c_int32), ("k_rot", ctypes.c_void_p)]


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"HIP library not built: {_LIB_PATH} is missing "
                           "(run `python -m paper_2402_04617_amd.build`)")
    L = ctypes.CDLL(_LIB_PATH)
    P, M = ctypes.POINTER(Params), ctypes.POINTER(Memory)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    sig = {
        "infllm_partition": [P, i64, ctypes.POINTER(i64), ctypes.POINTER(i32), ctypes.POINTER(i64)],
        "infllm_append": [P, M, vp, i64, vp, vp, i64, i32, i64, vp],
        "infllm_build_units": [P, M, i32, i32, i64, vp, vp],
        "infllm_score_units": [P, M, vp, i64, i32, i32, vp, vp, sz, vp],
        "infllm_select_topk": [i32, vp, i32, i32, vp, vp],
        "infllm_chunk_attend": [P, M, vp, i64, i32, i64, vp, i32, vp, i64, vp, vp, sz, vp],
        "infllm_chunk_attend_noalloc": [P, M, vp, i64, i32, i64, vp, i32, vp, i64, vp, vp],
        "infllm_attend_partial": [P, M, vp, i64, i32, i64, vp, i32, vp, i64, vp, vp, sz,
                                  ctypes.POINTER(i32), vp],
        "infllm_lse_merge": [P, i32, i32, i32, vp, sz, vp, i64, vp, vp],
        "infllm_step": [P, M, vp, i64, vp, vp, i64, i32, i64, i32, vp, vp, vp, i64, vp, vp, sz, vp],
        "infllm_step_mass": [P, M, vp, i64, vp, vp, i64, i32, i64, i32, vp, vp, vp, i64, vp, ctypes.c_float, vp, vp,
                             vp, sz, vp],
        "infllm_step_varlen": [P, M, vp, i64, vp, vp, i64, i32, ctypes.POINTER(i64), ctypes.POINTER(i32), vp, vp,
                               vp, i64, vp, vp, sz, vp],
        "infllm_unit_mass": [P, M, vp, i64, i32, i64, vp, i32, vp, ctypes.c_float, vp, vp, vp],
    }
    for name, args in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    L.infllm_workspace_bytes.argtypes = [P, i32, i32]
    L.infllm_workspace_bytes.restype = ctypes.c_size_t
    L.infllm_attend_workspace_bytes.argtypes = [P, i32, i32]
    L.infllm_attend_workspace_bytes.restype = ctypes.c_size_t
    L.infllm_status_string.argtypes = [ctypes.c_int]
    L.infllm_status_string.restype = ctypes.c_char_p
    _lib = L
    return L


def _check(fn: str, code: int) -> None:
    if code != 0:
        raise InfllmError(fn, code, lib().infllm_status_string(code).decode())


def _ptr(x) -> Optional[int]:
    """Device pointer of a tensor (or None / a raw int)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


# ------------------------------------------------------------------ entry points
def infllm_partition(p: Params, past_len: int) -> Tuple[int, int, int]:
    a, b, c = ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int64()
    _check("infllm_partition", lib().infllm_partition(ctypes.byref(p), past_len, ctypes.byref(a),
                                                      ctypes.byref(b), ctypes.byref(c)))
    return a.value, b.value, c.value


def infllm_workspace_bytes(p: Params, batch: int, n_q: int) -> int:
    return int(lib().infllm_workspace_bytes(ctypes.byref(p), batch, n_q))


def infllm_append(p, m, q, q_head_stride, k, v, kv_head_stride, n_q, past_len, stream=None):
    _check("infllm_append", lib().infllm_append(ctypes.byref(p), ctypes.byref(m), _ptr(q), q_head_stride,
                                                _ptr(k), _ptr(v), kv_head_stride, n_q, past_len,
                                                _stream(stream)))


def infllm_build_units(p, m, first_unit, n_new, past_len, repr_score=None, stream=None):
    _check("infllm_build_units", lib().infllm_build_units(ctypes.byref(p), ctypes.byref(m), first_unit, n_new,
                                                          past_len, _ptr(repr_score), _stream(stream)))


def infllm_score_units(p, m, q, q_head_stride, n_q, n_units, scores, workspace, workspace_bytes=None,
                       stream=None):
    wb = workspace.numel() * workspace.element_size() if workspace_bytes is None else workspace_bytes
    _check("infllm_score_units", lib().infllm_score_units(ctypes.byref(p), ctypes.byref(m), _ptr(q),
                                                          q_head_stride, n_q, n_units, _ptr(scores),
                                                          _ptr(workspace), wb, _stream(stream)))


def infllm_select_topk(rows, scores, n_units, k, idx, stream=None):
    _check("infllm_select_topk", lib().infllm_select_topk(rows, _ptr(scores), n_units, k, _ptr(idx),
                                                          _stream(stream)))


def infllm_chunk_attend(p, m, q, q_head_stride, n_q, past_len, idx, k, out, out_head_stride, lse=None,
                        workspace=None, workspace_bytes=None, stream=None):
    wb = (0 if workspace is None else workspace.numel() * workspace.element_size()) \
        if workspace_bytes is None else workspace_bytes
    _check("infllm_chunk_attend", lib().infllm_chunk_attend(
        ctypes.byref(p), ctypes.byref(m), _ptr(q), q_head_stride, n_q, past_len, _ptr(idx), k, _ptr(out),
        out_head_stride, _ptr(lse), _ptr(workspace), wb, _stream(stream)))


def infllm_chunk_attend_noalloc(p, m, q, q_head_stride, n_q, past_len, idx, k, out, out_head_stride, lse=None,
                                stream=None):
    _check("infllm_chunk_attend_noalloc", lib().infllm_chunk_attend_noalloc(
        ctypes.byref(p), ctypes.byref(m), _ptr(q), q_head_stride, n_q, past_len, _ptr(idx), k, _ptr(out),
        out_head_stride, _ptr(lse), _stream(stream)))


def infllm_attend_partial(p, m, q, q_head_stride, n_q, past_len, idx, k, out, out_head_stride, lse=None,
                          workspace=None, workspace_bytes=None, stream=None) -> int:
    wb = (0 if workspace is None else workspace.numel() * workspace.element_size()) \
        if workspace_bytes is None else workspace_bytes
    parts = ctypes.c_int32()
    _check("infllm_attend_partial", lib().infllm_attend_partial(
        ctypes.byref(p), ctypes.byref(m), _ptr(q), q_head_stride, n_q, past_len, _ptr(idx), k, _ptr(out),
        out_head_stride, _ptr(lse), _ptr(workspace), wb, ctypes.byref(parts), _stream(stream)))
    return parts.value


def infllm_lse_merge(p, batch, n_q, n_parts, workspace, out, out_head_stride, lse=None, workspace_bytes=None,
                     stream=None):
    wb = workspace.numel() * workspace.element_size() if workspace_bytes is None else workspace_bytes
    _check("infllm_lse_merge", lib().infllm_lse_merge(ctypes.byref(p), batch, n_q, n_parts, _ptr(workspace), wb,
                                                      _ptr(out), out_head_stride, _ptr(lse), _stream(stream)))


def infllm_step(p, m, q, q_head_stride, k, v, kv_head_stride, n_q, past_len, units_built, scores, idx, out,
                out_head_stride, lse=None, workspace=None, workspace_bytes=None, stream=None):
    wb = (0 if workspace is None else workspace.numel() * workspace.element_size()) \
        if workspace_bytes is None else workspace_bytes
    _check("infllm_step", lib().infllm_step(
        ctypes.byref(p), ctypes.byref(m), _ptr(q), q_head_stride, _ptr(k), _ptr(v), kv_head_stride, n_q, past_len,
        units_built, _ptr(scores), _ptr(idx), _ptr(out), out_head_stride, _ptr(lse), _ptr(workspace), wb,
        _stream(stream)))


def infllm_step_mass(p, m, q, q_head_stride, k, v, kv_head_stride, n_q, past_len, units_built, scores, idx, out,
                     out_head_stride, lse, decay, mass, freq=None, workspace=None, workspace_bytes=None, stream=None):
    wb = (0 if workspace is None else workspace.numel() * workspace.element_size()) \
        if workspace_bytes is None else workspace_bytes
    _check("infllm_step_mass", lib().infllm_step_mass(
        ctypes.byref(p), ctypes.byref(m), _ptr(q), q_head_stride, _ptr(k), _ptr(v), kv_head_stride, n_q, past_len,
        units_built, _ptr(scores), _ptr(idx), _ptr(out), out_head_stride, _ptr(lse), float(decay), _ptr(mass),
        _ptr(freq), _ptr(workspace), wb, _stream(stream)))


def infllm_unit_mass(p, m, q, q_head_stride, n_q, past_len, idx, k, lse, decay, mass, freq=None, stream=None):
    _check("infllm_unit_mass", lib().infllm_unit_mass(
        ctypes.byref(p), ctypes.byref(m), _ptr(q), q_head_stride, n_q, past_len, _ptr(idx), k, _ptr(lse),
        float(decay), _ptr(mass), _ptr(freq), _stream(stream)))


def infllm_step_varlen(p, m, q, q_head_stride, k, v, kv_head_stride, n_q, past_lens, units_built, scores, idx, out,
                       out_head_stride, lse=None, workspace=None, workspace_bytes=None, stream=None):
    """past_lens, units_built: sequences of `batch` ints (host)."""
    wb = (0 if workspace is None else workspace.numel() * workspace.element_size()) \
        if workspace_bytes is None else workspace_bytes
    pl = (ctypes.c_int64 * len(past_lens))(*[int(x) for x in past_lens])
    ub = (ctypes.c_int32 * len(units_built))(*[int(x) for x in units_built])
    _check("infllm_step_varlen", lib().infllm_step_varlen(
        ctypes.byref(p), ctypes.byref(m), _ptr(q), q_head_stride, _ptr(k), _ptr(v), kv_head_stride, n_q, pl, ub,
        _ptr(scores), _ptr(idx), _ptr(out), out_head_stride, _ptr(lse), _ptr(workspace), wb, _stream(stream)))


# ------------------------------------------------------------------ allocation plumbing
@dataclasses.dataclass
class LayerMemory:
    """Device tensors of one layer's context memory (allocated with PyTorch) and the
    infllm_memory struct that points at them."""

    k: "object"
    v: "object"
    repr_idx: "object"
    unit_ksum: "object"
    qprefix: "object"
    rpart: "object"
    struct: Memory
    k_rot: "object" = None


def params(n_q_heads, n_kv_heads, head_dim, n_init, n_local, block_size, n_repr, topk, dtype="bf16",
           sm_scale=1.0, rope_inv_freq=None, repr_mode="tokens") -> Params:
    """Method parameters.  rope_inv_freq: None (positions pre-applied) or the D/2 rotary angular
    frequencies of the positional remap.  repr_mode: "tokens" (r_k representative tokens) or
    "mean" (units scored by their mean key)."""
    p = Params(n_q_heads, n_kv_heads, head_dim, n_init, n_local, block_size, n_repr, topk,
               INFLLM_BF16 if dtype == "bf16" else INFLLM_F32, sm_scale)
    p.repr_mode = {"tokens": INFLLM_REPR_TOKENS, "mean": INFLLM_REPR_MEAN}[repr_mode]
    if rope_inv_freq is not None:
        if len(rope_inv_freq) != head_dim // 2:
            raise ValueError(f"rope_inv_freq needs head_dim/2 = {head_dim // 2} entries, got {len(rope_inv_freq)}")
        table = (ctypes.c_double * len(rope_inv_freq))(*[float(x) for x in rope_inv_freq])
        p._rope_table = table  # the struct holds a raw pointer: keep the array alive with it
        p.rope_inv_freq = ctypes.cast(table, ctypes.POINTER(ctypes.c_double))
    return p


def rope_frequencies(head_dim: int, base: float = 500000.0):
    """theta_i = base^(-2i/D), i < D/2 (the usual rotary frequencies; base 500000 as in Llama 3)."""
    return [base ** (-2.0 * i / head_dim) for i in range(head_dim // 2)]


def alloc_memory(p: Params, batch: int, capacity: int, max_units: int, ring: int, device="cuda") -> LayerMemory:
    import torch
    dt = torch.bfloat16 if p.dtype == INFLLM_BF16 else torch.float32
    D = p.head_dim
    k = torch.zeros((batch, p.n_kv_heads, capacity, D), dtype=dt, device=device)
    v = torch.zeros_like(k)
    mu = max(1, max_units)
    repr_idx = torch.zeros((batch, p.n_kv_heads, mu, p.n_repr), dtype=torch.int32, device=device)
    unit_ksum = torch.zeros((batch, p.n_kv_heads, D // 4, mu, 4), dtype=torch.float32, device=device)
    # the query ring and the partial representative scores exist only for representative tokens
    ring_used = not p.mean_repr
    qprefix = torch.zeros((batch, p.n_kv_heads, ring, D), dtype=torch.float64, device=device) if ring_used else None
    rpart = torch.zeros((batch, p.n_kv_heads, D // 8, ring), dtype=torch.float64, device=device) if ring_used else None
    k_rot = torch.zeros_like(k) if p.remap else None
    ptr = lambda t: t.data_ptr() if t is not None else None  # noqa: E731
    st = Memory(batch, capacity, k.data_ptr(), v.data_ptr(), max_units, repr_idx.data_ptr(),
                unit_ksum.data_ptr(), ptr(qprefix), ptr(rpart), ring if ring_used else 0, ptr(k_rot))
    return LayerMemory(k, v, repr_idx, unit_ksum, qprefix, rpart, st, k_rot)


def recommended_ring(p: Params, chunk: int) -> int:
    """Ring slots that cover the oldest window unit construction can still need, plus one chunk, so
    that infllm_step can run unit construction and the append in a single launch."""
    return p.n_local + p.block_size + 2 * chunk + 1
