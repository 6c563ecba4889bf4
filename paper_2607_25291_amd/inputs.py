"""Seeded synthetic prefill-attention inputs (shared by the HIP path's tests/bench and the oracle).

This module only *makes data*: it holds none of the method's arithmetic. Both sides of every parity
check consume the very same bf16 bit patterns produced here.

Inputs stand in for the paper's workloads (Qwen3-8B / Llama-3.1-8B activations on RULER and
LongBench-v2, Sec. 5 "Setup"), which are not available. The structure injected mirrors what the paper
observes in real attention maps: attention sinks and a recent-token window (Sec. 3, Limitation 2.1),
row maxima scattered over the map (Sec. 3, Fig. 3 discussion) and needle-like salient blocks
(Sec. 3, Property 1).

Recipe, per (batch index n, KV head g), from ``numpy.random.default_rng(SeedSequence([seed, n, g]))``
and always drawn in this order:

1. K_g, V_g ~ N(0, 1), shape [L, d] (float32).
2. Sinks: K_g[0:n_sink] *= sink_scale.
3. Local window W: a shared AR(1) component c_g (rho = exp(-1/W), unit stationary variance) over
   tokens; every query head h of the group gets Q_h = (Z_h + c_g) / sqrt(2) with Z_h ~ N(0, 1);
   then K_g[t] += 0.5 * mean_h Q_h[t] ("adding 0.5 q to k").
4. Salient keys: a fraction f_k of the positions in [n_sink, L) (without replacement) get
   K_g += 3 u_g, with u_g a random unit vector of the group. f_k is either fixed or drawn per KV head
   from U[lo, hi].
5. Salient queries: 10 % of the positions of every query head of the group get Q_h += 3 u_g.

Everything is rounded once to bf16 (round-to-nearest-even) and returned as uint16 bit patterns with
layout Q [B, Hq, L, d], K/V [B, Hkv, L, d].
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional, Tuple, Union

import numpy as np
from scipy.signal import lfilter


@dataclasses.dataclass(frozen=True)
class Workload:
    """One attention-layer prefill problem plus the two budgets it is run at."""

    name: str
    batch: int
    n_q_heads: int
    n_kv_heads: int
    seq_len: int
    head_dim: int
    block: int
    stride: int
    kap_budget: float          # stage-1 budget B1 (fraction of causal blocks kept by the proxy)
    osk_budget: float          # overall budget B2 reached by the in-kernel skip
    window: int                # AR(1) correlation length W of the local-window structure
    salient_key_frac: Union[float, Tuple[float, float]]
    salient_query_frac: float = 0.10
    sink_scale: float = 8.0
    n_sink: int = 4
    seed: int = 0

    @property
    def n_blocks(self) -> int:
        return -(-self.seq_len // self.block)


# Named workloads. Shapes follow one Qwen3-8B attention layer (32 query heads, 8 KV heads, d = 128)
# and a wider 8:1 GQA variant; block b = 128 is the paper's setting (appendix, "CoSA settings"), and
# the stride s = b / 8 gives 8 samples per block.
WORKLOADS = {
    "tiny_l2k": Workload("tiny_l2k", 1, 1, 1, 2048, 128, 64, 8, 0.50, 0.25, 256, 0.02),
    "qwen3_8b_l32k": Workload("qwen3_8b_l32k", 1, 32, 8, 32768, 128, 128, 16, 0.20, 0.10, 1024,
                              (0.005, 0.03)),
    "qwen3_8b_l128k": Workload("qwen3_8b_l128k", 1, 32, 8, 131072, 128, 128, 16, 0.10, 0.05, 1024,
                               (0.005, 0.03)),
    "wide_gqa_l64k": Workload("wide_gqa_l64k", 1, 64, 8, 65536, 128, 128, 16, 0.15, 0.075, 1024,
                              (0.005, 0.03)),
}


def sweep_workloads():
    """Budget grid at the 128K shape: B1 in {5,10,20,40}% crossed with B2 = {1, 1/2, 1/4} x B1."""
    base = WORKLOADS["qwen3_8b_l128k"]
    out = []
    for b1 in (0.05, 0.10, 0.20, 0.40):
        for f in (1.0, 0.5, 0.25):
            out.append(dataclasses.replace(base, name=f"sweep_b1_{b1:g}_b2_{b1 * f:g}",
                                           kap_budget=b1, osk_budget=b1 * f))
    return out


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round-to-nearest-even) and return the uint16 bit pattern."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    rounding = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + rounding) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _ar1(rng: np.random.Generator, L: int, d: int, window: int) -> np.ndarray:
    rho = math.exp(-1.0 / window)
    x = rng.standard_normal((L, d), dtype=np.float32)
    c0 = math.sqrt(1.0 - rho * rho)
    x[0] /= np.float32(c0)              # so that c[0] = eps[0] (stationary, unit variance)
    return lfilter(np.array([c0], np.float32), np.array([1.0, -rho], np.float32), x, axis=0)


def _unit(rng: np.random.Generator, d: int) -> np.ndarray:
    u = rng.standard_normal(d)
    return u / np.linalg.norm(u)


def make_group(w: Workload, n: int, g: int, seed: Optional[int] = None):
    """Generate (Q [G, L, d], K [L, d], V [L, d]) float32 for batch index n and KV head g."""
    seed = w.seed if seed is None else seed
    rng = np.random.default_rng(np.random.SeedSequence([seed, n, g]))
    L, d = w.seq_len, w.head_dim
    G = w.n_q_heads // w.n_kv_heads
    k = rng.standard_normal((L, d), dtype=np.float32)
    v = rng.standard_normal((L, d), dtype=np.float32)
    ns = min(w.n_sink, L)
    k[:ns] *= np.float32(w.sink_scale)
    c = _ar1(rng, L, d, w.window)
    q = np.empty((G, L, d), dtype=np.float32)
    for hh in range(G):
        q[hh] = rng.standard_normal((L, d), dtype=np.float32)
        q[hh] += c
        q[hh] *= np.float32(1.0 / math.sqrt(2.0))
    k += np.float32(0.5) * q.mean(axis=0)
    if isinstance(w.salient_key_frac, tuple):
        lo, hi = w.salient_key_frac
        fk = float(rng.uniform(lo, hi))
    else:
        fk = float(w.salient_key_frac)
    u = _unit(rng, d).astype(np.float32)
    n_cand = max(L - ns, 0)
    nk = int(round(fk * n_cand))
    if nk > 0:
        pos = ns + rng.choice(n_cand, size=nk, replace=False)
        k[pos] += np.float32(3.0) * u
    nq = int(round(w.salient_query_frac * L))
    for hh in range(G):
        if nq > 0:
            pos = rng.choice(L, size=nq, replace=False)
            q[hh, pos] += np.float32(3.0) * u
    return q, k, v


def make_inputs(w: Workload, seed: Optional[int] = None):
    """Return bf16 bit patterns (uint16): q [B,Hq,L,d], k [B,Hkv,L,d], v [B,Hkv,L,d]."""
    B, Hq, Hkv, L, d = w.batch, w.n_q_heads, w.n_kv_heads, w.seq_len, w.head_dim
    G = Hq // Hkv
    q = np.empty((B, Hq, L, d), dtype=np.uint16)
    k = np.empty((B, Hkv, L, d), dtype=np.uint16)
    v = np.empty((B, Hkv, L, d), dtype=np.uint16)

    def one(ng):
        n, g = divmod(ng, Hkv)
        qg, kg, vg = make_group(w, n, g, seed)
        q[n, g * G:(g + 1) * G] = f32_to_bf16_bits(qg)
        k[n, g] = f32_to_bf16_bits(kg)
        v[n, g] = f32_to_bf16_bits(vg)

    # groups are independent streams of one seed: generate them concurrently
    workers = max(1, min(B * Hkv, os.cpu_count() or 1, 16))
    with ThreadPoolExecutor(max_workers=workers) as ex:
        list(ex.map(one, range(B * Hkv)))
    return q, k, v


def random_inputs(B: int, Hq: int, Hkv: int, L: int, d: int, seed: int = 0, scale: float = 1.0):
    """Unstructured N(0, scale^2) bf16 inputs for edge-case tests (same layouts as make_inputs)."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 7919]))
    q = f32_to_bf16_bits(scale * rng.standard_normal((B, Hq, L, d), dtype=np.float32))
    k = f32_to_bf16_bits(scale * rng.standard_normal((B, Hkv, L, d), dtype=np.float32))
    v = f32_to_bf16_bits(rng.standard_normal((B, Hkv, L, d), dtype=np.float32))
    return q, k, v
