"""Thin ctypes binding of libcosa.so: the C entry points under the same names.

Argument marshalling only: torch tensors supply device pointers (PyTorch is used for device memory
and streams), every computation runs in the library's HIP kernels. The binding raises if the
library was not built; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
import re
from dataclasses import dataclass
from typing import Optional

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libcosa.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "cosa.h")

COSA_OK, COSA_ERR_INVALID_ARG, COSA_ERR_UNSUPPORTED, COSA_ERR_WORKSPACE, COSA_ERR_HIP = range(5)
SELECT_FRACTION, SELECT_TOP_P, SELECT_ALL = 0, 1, 2
ORDER_KAP, ORDER_ASCENDING = 0, 1
SKIP_NONE, SKIP_ROWMAX = 0, 1
VISIT_COMPUTED, VISIT_SKIPPED = 1, 2


class CosaProblem(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("seq_len", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("block", ctypes.c_int32),
                ("stride", ctypes.c_int32), ("sm_scale", ctypes.c_float),
                ("causal", ctypes.c_int32)]


class CosaSelect(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int), ("value", ctypes.c_float), ("order", ctypes.c_int)]


class CosaSkip(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int), ("delta", ctypes.c_float)]


class CosaWorkspaceLayout(ctypes.Structure):
    _fields_ = [("score", ctypes.c_size_t), ("hrm", ctypes.c_size_t), ("order", ctypes.c_size_t),
                ("count", ctypes.c_size_t), ("keys", ctypes.c_size_t), ("queue", ctypes.c_size_t),
                ("total", ctypes.c_size_t)]


class CosaPagedKv(ctypes.Structure):
    _fields_ = [("k_cache", ctypes.c_void_p), ("v_cache", ctypes.c_void_p),
                ("page_table", ctypes.c_void_p), ("page_size", ctypes.c_int32),
                ("n_pages", ctypes.c_int64)]


class CosaVarlen(ctypes.Structure):
    _fields_ = [("n_seqs", ctypes.c_int32), ("cu_blocks", ctypes.POINTER(ctypes.c_int32))]


MAX_PACKED_SEQS = 128


class CosaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


@dataclass(frozen=True)
class Problem:
    batch: int
    n_q_heads: int
    n_kv_heads: int
    seq_len: int
    head_dim: int = 128
    block: int = 128
    stride: int = 16
    sm_scale: float = 0.0
    causal: int = 1

    @property
    def n_blocks(self) -> int:
        return -(-self.seq_len // self.block) if self.block > 0 else 0

    def c(self) -> CosaProblem:
        return CosaProblem(self.batch, self.n_q_heads, self.n_kv_heads, self.seq_len,
                           self.head_dim, self.block, self.stride, self.sm_scale, self.causal)


_lib = None


def declared_symbols():
    """Names of the functions include/cosa.h declares."""
    text = open(HEADER_PATH).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\*?\s+\*?(cosa_[a-z_0-9]+)\(", text,
                                 re.M)))


def lib():
    """Load libcosa.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2607_25291_amd.build_lib`")
        # The library's HIP calls must bind to the HIP runtime that PyTorch loaded, so that the
        # tensors, streams and events it hands over belong to the same runtime. Importing torch
        # first puts that runtime in the process's global symbol scope, where the dynamic linker
        # resolves the library's HIP symbols; loaded the other way round, the library would start
        # a second HIP runtime of its own, which does not share torch's streams or device state.
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB_PATH)
        P, S, vp = ctypes.POINTER(CosaProblem), ctypes.c_int, ctypes.c_void_p
        L.cosa_status_string.restype = ctypes.c_char_p
        L.cosa_status_string.argtypes = [S]
        L.cosa_last_error.restype = ctypes.c_char_p
        L.cosa_last_error.argtypes = []
        L.cosa_kap_score.restype = S
        L.cosa_kap_score.argtypes = [P, vp, vp, vp, vp, vp]
        L.cosa_kap_select_ordered.restype = S
        L.cosa_kap_select_ordered.argtypes = [P, vp, vp, ctypes.POINTER(CosaSelect), vp, vp, vp]
        L.cosa_osk_attention.restype = S
        L.cosa_osk_attention.argtypes = [P, vp, vp, vp, vp, vp, ctypes.POINTER(CosaSkip), vp, vp,
                                         vp, vp, vp]
        L.cosa_osk_attention_queue_bytes.restype = ctypes.c_size_t
        L.cosa_osk_attention_queue_bytes.argtypes = []
        L.cosa_osk_attention_queued.restype = S
        L.cosa_osk_attention_queued.argtypes = [P, vp, vp, vp, vp, vp, ctypes.POINTER(CosaSkip), vp,
                                                vp, vp, vp, vp, ctypes.c_size_t, vp]
        L.cosa_dense_attention.restype = S
        L.cosa_dense_attention.argtypes = [P, vp, vp, vp, vp, vp]
        L.cosa_prefill_workspace_bytes.restype = ctypes.c_size_t
        L.cosa_prefill_workspace_bytes.argtypes = [P]
        L.cosa_prefill_workspace_layout.restype = S
        L.cosa_prefill_workspace_layout.argtypes = [P, ctypes.POINTER(CosaWorkspaceLayout)]
        L.cosa_prefill.restype = S
        L.cosa_prefill.argtypes = [P, vp, vp, vp, ctypes.POINTER(CosaSelect),
                                   ctypes.POINTER(CosaSkip), vp, ctypes.c_size_t, vp, vp]
        L.cosa_prefill_noalloc.restype = S
        L.cosa_prefill_noalloc.argtypes = [P, vp, vp, vp, ctypes.POINTER(CosaSelect),
                                           ctypes.POINTER(CosaSkip), vp, vp]
        L.cosa_block_mass.restype = S
        L.cosa_block_mass.argtypes = [P, vp, vp, vp, vp]
        L.cosa_masked_attention.restype = S
        L.cosa_masked_attention.argtypes = [P, vp, vp, vp, vp, vp, vp]
        KV = ctypes.POINTER(CosaPagedKv)
        L.cosa_kap_score_paged.restype = S
        L.cosa_kap_score_paged.argtypes = [P, vp, KV, vp, vp, vp]
        L.cosa_osk_attention_paged.restype = S
        L.cosa_osk_attention_paged.argtypes = [P, vp, KV, vp, vp, ctypes.POINTER(CosaSkip), vp, vp,
                                               vp, vp, vp]
        L.cosa_prefill_paged.restype = S
        L.cosa_prefill_paged.argtypes = [P, vp, KV, ctypes.POINTER(CosaSelect),
                                         ctypes.POINTER(CosaSkip), vp, ctypes.c_size_t, vp, vp]
        L.cosa_kap_score_workspace_bytes.restype = ctypes.c_size_t
        L.cosa_kap_score_workspace_bytes.argtypes = [P]
        L.cosa_kap_score_staged.restype = S
        L.cosa_kap_score_staged.argtypes = [P, vp, vp, vp, ctypes.c_size_t, vp, vp, vp]
        VL = ctypes.POINTER(CosaVarlen)
        L.cosa_kap_score_varlen.restype = S
        L.cosa_kap_score_varlen.argtypes = [P, VL, vp, vp, vp, vp, vp]
        L.cosa_kap_select_ordered_varlen.restype = S
        L.cosa_kap_select_ordered_varlen.argtypes = [P, VL, vp, vp, ctypes.POINTER(CosaSelect), vp,
                                                     vp, vp]
        L.cosa_osk_attention_varlen.restype = S
        L.cosa_osk_attention_varlen.argtypes = [P, VL, vp, vp, vp, vp, vp, ctypes.POINTER(CosaSkip),
                                                vp, vp, vp, vp, vp]
        L.cosa_dense_attention_varlen.restype = S
        L.cosa_dense_attention_varlen.argtypes = [P, VL, vp, vp, vp, vp, vp]
        L.cosa_prefill_varlen.restype = S
        L.cosa_prefill_varlen.argtypes = [P, VL, vp, vp, vp, ctypes.POINTER(CosaSelect),
                                          ctypes.POINTER(CosaSkip), vp, ctypes.c_size_t, vp, vp]
        L.cosa_prefill_paged_varlen.restype = S
        L.cosa_prefill_paged_varlen.argtypes = [P, VL, vp, KV, ctypes.POINTER(CosaSelect),
                                                ctypes.POINTER(CosaSkip), vp, ctypes.c_size_t, vp,
                                                vp]
        _lib = L
    return _lib


def _check(status: int):
    if status != COSA_OK:
        raise CosaError(status, lib().cosa_last_error().decode())


def _ptr(t) -> Optional[int]:
    """Device pointer of a tensor (None -> NULL); integers are passed through as raw pointers."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("tensors must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _prob(problem) -> CosaProblem:
    return problem.c() if isinstance(problem, Problem) else problem


def select(mode: int = SELECT_FRACTION, value: float = 1.0, order: int = ORDER_KAP) -> CosaSelect:
    return CosaSelect(mode, value, order)


def skip(mode: int = SKIP_NONE, delta: float = 0.0) -> CosaSkip:
    return CosaSkip(mode, delta)


def cosa_status_string(status: int) -> str:
    return lib().cosa_status_string(status).decode()


def cosa_last_error() -> str:
    return lib().cosa_last_error().decode()


def cosa_kap_score(problem, q, k, score, hrm, stream=None):
    p = _prob(problem)
    _check(lib().cosa_kap_score(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(score), _ptr(hrm),
                                _stream(stream)))


def cosa_kap_score_workspace_bytes(problem) -> int:
    p = _prob(problem)
    return int(lib().cosa_kap_score_workspace_bytes(ctypes.byref(p)))


def cosa_kap_score_staged(problem, q, k, workspace, workspace_bytes: int, score, hrm, stream=None):
    p = _prob(problem)
    _check(lib().cosa_kap_score_staged(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(workspace),
                                       workspace_bytes, _ptr(score), _ptr(hrm), _stream(stream)))


def cosa_kap_select_ordered(problem, score, hrm, sel: CosaSelect, order, count, stream=None):
    p = _prob(problem)
    _check(lib().cosa_kap_select_ordered(ctypes.byref(p), _ptr(score), _ptr(hrm), ctypes.byref(sel),
                                         _ptr(order), _ptr(count), _stream(stream)))


def cosa_osk_attention(problem, q, k, v, order, count, sk: Optional[CosaSkip], o, visit_log=None,
                       margin_log=None, n_computed=None, stream=None):
    p = _prob(problem)
    skp = ctypes.byref(sk) if sk is not None else None
    _check(lib().cosa_osk_attention(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(order),
                                    _ptr(count), skp, _ptr(o), _ptr(visit_log), _ptr(margin_log),
                                    _ptr(n_computed), _stream(stream)))


def cosa_osk_attention_queue_bytes() -> int:
    return int(lib().cosa_osk_attention_queue_bytes())


def cosa_osk_attention_queued(problem, q, k, v, order, count, sk: Optional[CosaSkip], o, queue,
                              queue_bytes: int, visit_log=None, margin_log=None, n_computed=None,
                              stream=None):
    p = _prob(problem)
    skp = ctypes.byref(sk) if sk is not None else None
    _check(lib().cosa_osk_attention_queued(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(order),
                                           _ptr(count), skp, _ptr(o), _ptr(visit_log),
                                           _ptr(margin_log), _ptr(n_computed), _ptr(queue),
                                           queue_bytes, _stream(stream)))


def cosa_dense_attention(problem, q, k, v, o, stream=None):
    p = _prob(problem)
    _check(lib().cosa_dense_attention(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(o),
                                      _stream(stream)))


def cosa_block_mass(problem, q, k, mass, stream=None):
    p = _prob(problem)
    _check(lib().cosa_block_mass(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(mass), _stream(stream)))


def cosa_masked_attention(problem, q, k, v, mask, o, stream=None):
    p = _prob(problem)
    _check(lib().cosa_masked_attention(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(mask),
                                       _ptr(o), _stream(stream)))


def cosa_prefill_workspace_bytes(problem) -> int:
    p = _prob(problem)
    n = lib().cosa_prefill_workspace_bytes(ctypes.byref(p))
    if n == 0 and not (p.batch == 0 or p.seq_len == 0):
        raise CosaError(COSA_ERR_INVALID_ARG, cosa_last_error())
    return n


def cosa_prefill_workspace_layout(problem) -> CosaWorkspaceLayout:
    p = _prob(problem)
    out = CosaWorkspaceLayout()
    _check(lib().cosa_prefill_workspace_layout(ctypes.byref(p), ctypes.byref(out)))
    return out


def cosa_prefill(problem, q, k, v, sel: CosaSelect, sk: Optional[CosaSkip], workspace,
                 workspace_bytes: int, o, stream=None):
    p = _prob(problem)
    skp = ctypes.byref(sk) if sk is not None else None
    _check(lib().cosa_prefill(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), ctypes.byref(sel), skp,
                              _ptr(workspace), workspace_bytes, _ptr(o), _stream(stream)))


NOALLOC_SCRATCH_BYTES = 128 * 1024 * 1024


def cosa_prefill_noalloc(problem, q, k, v, sel: CosaSelect, sk: Optional[CosaSkip], o,
                         stream=None):
    p = _prob(problem)
    skp = ctypes.byref(sk) if sk is not None else None
    _check(lib().cosa_prefill_noalloc(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v),
                                      ctypes.byref(sel), skp, _ptr(o), _stream(stream)))


def _kvref(kv):
    return ctypes.byref(kv) if kv is not None else None


def paged_kv(k_cache, v_cache, page_table, page_size: int, n_pages: int) -> CosaPagedKv:
    """cosa_paged_kv from device tensors (v_cache may be None for the proxy-only call)."""
    return CosaPagedKv(_ptr(k_cache), _ptr(v_cache), _ptr(page_table), page_size, n_pages)


def cosa_kap_score_paged(problem, q, kv: CosaPagedKv, score, hrm, stream=None):
    p = _prob(problem)
    _check(lib().cosa_kap_score_paged(ctypes.byref(p), _ptr(q), _kvref(kv), _ptr(score),
                                      _ptr(hrm), _stream(stream)))


def cosa_osk_attention_paged(problem, q, kv: CosaPagedKv, order, count, sk: Optional[CosaSkip], o,
                             visit_log=None, margin_log=None, n_computed=None, stream=None):
    p = _prob(problem)
    skp = ctypes.byref(sk) if sk is not None else None
    _check(lib().cosa_osk_attention_paged(ctypes.byref(p), _ptr(q), _kvref(kv), _ptr(order),
                                          _ptr(count), skp, _ptr(o), _ptr(visit_log),
                                          _ptr(margin_log), _ptr(n_computed), _stream(stream)))


def cosa_prefill_paged(problem, q, kv: CosaPagedKv, sel: CosaSelect, sk: Optional[CosaSkip],
                       workspace, workspace_bytes: int, o, stream=None):
    p = _prob(problem)
    skp = ctypes.byref(sk) if sk is not None else None
    _check(lib().cosa_prefill_paged(ctypes.byref(p), _ptr(q), _kvref(kv), ctypes.byref(sel),
                                    skp, _ptr(workspace), workspace_bytes, _ptr(o),
                                    _stream(stream)))


def varlen(cu_blocks) -> CosaVarlen:
    """cosa_varlen from host block offsets [0, ..., nb] of the packed sequences (the struct keeps
    its own copy of the array alive)."""
    vals = [int(x) for x in cu_blocks]
    arr = (ctypes.c_int32 * max(len(vals), 1))(*vals)
    v = CosaVarlen(len(vals) - 1, ctypes.cast(arr, ctypes.POINTER(ctypes.c_int32)))
    v._host_offsets = arr
    return v


def _vlref(vl):
    return ctypes.byref(vl) if vl is not None else None


def cosa_kap_score_varlen(problem, vl: CosaVarlen, q, k, score, hrm, stream=None):
    p = _prob(problem)
    _check(lib().cosa_kap_score_varlen(ctypes.byref(p), _vlref(vl), _ptr(q), _ptr(k), _ptr(score),
                                       _ptr(hrm), _stream(stream)))


def cosa_kap_select_ordered_varlen(problem, vl: CosaVarlen, score, hrm, sel: CosaSelect, order,
                                   count, stream=None):
    p = _prob(problem)
    _check(lib().cosa_kap_select_ordered_varlen(ctypes.byref(p), _vlref(vl), _ptr(score), _ptr(hrm),
                                                ctypes.byref(sel), _ptr(order), _ptr(count),
                                                _stream(stream)))


def cosa_osk_attention_varlen(problem, vl: CosaVarlen, q, k, v, order, count,
                              sk: Optional[CosaSkip], o, visit_log=None, margin_log=None,
                              n_computed=None, stream=None):
    p = _prob(problem)
    skp = ctypes.byref(sk) if sk is not None else None
    _check(lib().cosa_osk_attention_varlen(ctypes.byref(p), _vlref(vl), _ptr(q), _ptr(k), _ptr(v),
                                           _ptr(order), _ptr(count), skp, _ptr(o), _ptr(visit_log),
                                           _ptr(margin_log), _ptr(n_computed), _stream(stream)))


def cosa_dense_attention_varlen(problem, vl: CosaVarlen, q, k, v, o, stream=None):
    p = _prob(problem)
    _check(lib().cosa_dense_attention_varlen(ctypes.byref(p), _vlref(vl), _ptr(q), _ptr(k), _ptr(v),
                                             _ptr(o), _stream(stream)))


def cosa_prefill_varlen(problem, vl: CosaVarlen, q, k, v, sel: CosaSelect, sk: Optional[CosaSkip],
                        workspace, workspace_bytes: int, o, stream=None):
    p = _prob(problem)
    skp = ctypes.byref(sk) if sk is not None else None
    _check(lib().cosa_prefill_varlen(ctypes.byref(p), _vlref(vl), _ptr(q), _ptr(k), _ptr(v),
                                     ctypes.byref(sel), skp, _ptr(workspace), workspace_bytes,
                                     _ptr(o), _stream(stream)))


def cosa_prefill_paged_varlen(problem, vl: CosaVarlen, q, kv: CosaPagedKv, sel: CosaSelect,
                              sk: Optional[CosaSkip], workspace, workspace_bytes: int, o,
                              stream=None):
    p = _prob(problem)
    skp = ctypes.byref(sk) if sk is not None else None
    _check(lib().cosa_prefill_paged_varlen(ctypes.byref(p), _vlref(vl), _ptr(q), _kvref(kv),
                                           ctypes.byref(sel), skp, _ptr(workspace),
                                           workspace_bytes, _ptr(o), _stream(stream)))
