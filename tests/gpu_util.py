"""GPU-side helpers for the parity tests: device buffers and calls through the C ABI binding."""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

from paper_2607_25291_amd import binding as B


def torch():
    import torch as _t
    return _t


def dev(a: np.ndarray):
    """Upload uint16/int32/uint8 numpy data to the GPU (bit-identical)."""
    t = torch()
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return t.from_numpy(a).cuda()


def host_bits(t) -> np.ndarray:
    a = t.cpu().numpy()
    return a.view(np.uint16) if a.dtype == np.int16 else a


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


@dataclass
class Run:
    """One problem resident on the GPU."""
    problem: B.Problem
    q: object
    k: object
    v: object

    @classmethod
    def upload(cls, problem: B.Problem, q, k, v):
        return cls(problem, dev(q), dev(k), dev(v))

    def _zeros(self, shape, dtype):
        return torch().zeros(shape, dtype=dtype, device="cuda")

    def kap_score(self):
        p = self.problem
        nb = p.n_blocks
        t = torch()
        score = self._zeros((p.batch, p.n_kv_heads, nb, nb), t.float32)
        hrm = self._zeros((p.batch, p.n_kv_heads, nb, nb), t.uint8)
        B.cosa_kap_score(p, self.q, self.k, score, hrm)
        return score, hrm

    def kap_select(self, score, hrm, sel):
        p = self.problem
        nb = p.n_blocks
        t = torch()
        order = self._zeros((p.batch, p.n_kv_heads, nb, nb), t.int32)
        count = self._zeros((p.batch, p.n_kv_heads, nb), t.int32)
        B.cosa_kap_select_ordered(p, score, hrm, sel, order, count)
        return order, count

    def osk(self, order, count, sk=None, logs=True):
        p = self.problem
        nb = p.n_blocks
        t = torch()
        o = self._zeros((p.batch, p.n_q_heads, p.seq_len, p.head_dim), t.int16)
        visit = self._zeros((p.batch, p.n_q_heads, nb, nb), t.uint8) if logs else None
        margin = self._zeros((p.batch, p.n_q_heads, nb, nb), t.float32) if logs else None
        ncomp = self._zeros((p.batch, p.n_q_heads, nb), t.int32) if logs else None
        B.cosa_osk_attention(p, self.q, self.k, self.v, order, count, sk, o, visit, margin, ncomp)
        return o, visit, margin, ncomp

    def dense(self):
        p = self.problem
        o = self._zeros((p.batch, p.n_q_heads, p.seq_len, p.head_dim), torch().int16)
        B.cosa_dense_attention(p, self.q, self.k, self.v, o)
        return o

    def prefill(self, sel, sk=None):
        p = self.problem
        t = torch()
        nbytes = B.cosa_prefill_workspace_bytes(p)
        ws = self._zeros((nbytes,), t.uint8)
        o = self._zeros((p.batch, p.n_q_heads, p.seq_len, p.head_dim), t.int16)
        B.cosa_prefill(p, self.q, self.k, self.v, sel, sk, ws, nbytes, o)
        lay = B.cosa_prefill_workspace_layout(p)
        nb = p.n_blocks
        shp = (p.batch, p.n_kv_heads, nb, nb)
        cells = p.batch * p.n_kv_heads * nb * nb
        order = ws[lay.order:lay.order + 4 * cells].view(t.int32).view(shp)
        count = ws[lay.count:lay.count + 4 * p.batch * p.n_kv_heads * nb].view(t.int32).view(shp[:3])
        score = ws[lay.score:lay.score + 4 * cells].view(t.float32).view(shp)
        hrm = ws[lay.hrm:lay.hrm + cells].view(shp)
        return o, score, hrm, order, count


def tau_of(delta: float, L: int) -> float:
    return float(np.float32(math.log(float(np.float32(delta)) / L)))
