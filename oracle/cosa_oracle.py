"""CPU oracle for CoSA prefill attention (KAP proxy + ordered-skipping kernel + dense attention).

TEST INFRASTRUCTURE ONLY. This module is the plain, slow, float64 statement of what the HIP path
computes. Only the test-suite, the smoke check and the CPU-baseline leg of the benchmark may import
it; the library and its Python binding never do, and it shares no code with them (it does not import
the package at all: inputs arrive as uint16 bf16 bit patterns).

Everything follows the paper "CoSA: Accelerating Long-Context Inference via Proxy-Kernel Co-Designed
Sparse Attention" (arXiv 2607.25291):

* KAP scoring, Sec. 4.2 "Block ranking" and Eq. (score); Algorithm A, proxy stage.
* Flag-grouped sort and the ordered mask M_KAP, Sec. 4.2 "Flag-grouped sorting", Eq. (mkap).
* OSK list walk with in-kernel skip, Sec. 4.3 and Algorithm A, attention loop; skip rule Eq. (skip).
* Dense attention, Sec. 3.1 (tiled online softmax = ordinary causal softmax attention).
* Exact block attention mass (the ground truth of the proxy-fidelity comparison), Sec. 3.2.
* Packed variable-length batches: every packed sequence is its own problem (the definition; the
  paper treats one sequence at a time), with N in ln(Delta/N) the sequence's own length.

Readings of points where the paper is silent or loose (all indices 0-based):

* Stride sampling takes the first token of every stride group: Q~[r] = Q[r s], K~[c] = K[c s].
* Logits are scaled by sm_scale (1/sqrt(d) by default) in both the proxy and the kernel; the skip
  threshold tau = ln(Delta/N) is in natural-log units of those scaled logits, N = seq_len.
* The proxy applies the causal mask over sampled positions (key c visible to row r iff c <= r).
* GQA: one ordered list per KV head; the block score sums over the sampled rows of all query heads of
  the group and the HRM flag is an OR over them. The skip vote stays per (query head, query block).
* K_i under a fractional budget is min(i+1, max(1, ceil(B1 (i+1)))) over the i+1 causal
  candidates, with B1 taken at 1e-6 resolution and the product formed in integers; top-p keeps the
  shortest prefix of the HRM-first order whose score mass reaches p of the row total, both sums in
  float64 taken term by term (the total over ascending block index, the running mass in list
  order). Equal sort keys are ordered by ascending block index.
* HRM is exact equality with the row maximum in the working precision.
* tau is computed in float64 from the float32 Delta and rounded once to float32.
* A ragged last block (seq_len not a multiple of b) has fewer rows/keys; nothing else changes.

Parity pinning status: every function here is pinned by the CPU tests (closed forms, invariants,
brute force on tiny inputs, independent library routines); the paper prints no worked example
(its illustrative KAP figure carries no values), so nothing is pinned to printed paper numbers.
The conventions listed above have no paper value to pin against.
"""
from __future__ import annotations

import math
from typing import Dict, Iterable, List, Optional, Sequence, Tuple

import numpy as np

SELECT_FRACTION = 0
SELECT_TOP_P = 1
SELECT_ALL = 2
ORDER_KAP = 0
ORDER_ASCENDING = 1
SKIP_NONE = 0
SKIP_ROWMAX = 1

VISIT_COMPUTED = 1
VISIT_SKIPPED = 2


# ----------------------------------------------------------------------------------------------
# inputs
# ----------------------------------------------------------------------------------------------
def widen(bits: np.ndarray) -> np.ndarray:
    """Exact value of bf16 bit patterns (uint16) as float64 (Algorithm A input Q, K, V)."""
    u = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


class _Heads:
    """Per-(batch, head) float64 values of a [B, H, L, d] bf16 tensor, widened on first use."""

    def __init__(self, bits: np.ndarray):
        self.bits = bits
        self.shape = bits.shape
        self._cache: Dict[Tuple[int, int], np.ndarray] = {}

    def __call__(self, n: int, h: int) -> np.ndarray:
        key = (n, h)
        if key not in self._cache:
            self._cache[key] = widen(self.bits[n, h])
        return self._cache[key]


def default_scale(head_dim: int, sm_scale: float = 0.0) -> float:
    """Logit scale of Algorithm A (1/sqrt(d)); a non-zero float32 override is used as given."""
    if sm_scale and sm_scale > 0:
        return float(np.float32(sm_scale))
    return float(np.float32(1.0 / math.sqrt(head_dim)))


def tau_from_delta(delta: float, seq_len: int) -> float:
    """Skip threshold ln(Delta/N) of Eq. (skip), computed in float64 and rounded once to float32."""
    d32 = float(np.float32(delta))
    return float(np.float32(math.log(d32 / float(seq_len))))


def n_blocks(seq_len: int, block: int) -> int:
    return -(-seq_len // block)


# ----------------------------------------------------------------------------------------------
# Stage 1: Kernel-Aware Proxy (Sec. 4.2, Eq. (score), Algorithm A proxy stage)
# ----------------------------------------------------------------------------------------------
def _kap_unit(qw, kw, n, g, i, G, block, stride, scale, L):
    """Literal proxy steps for one (batch n, KV head g, query block i).

    Returns (s_i, hmax_i): the block scores s_ij = sum_r Pbar[r, j] over the sampled rows of all G
    query heads, and max_r Pbar[r, j] (the HRM flag is hmax == 1), for j = 0..nb-1.
    """
    spb = block // stride
    nb = n_blocks(L, block)
    n_samp = -(-L // stride)                     # sampled keys c with c*s < L
    ktil = kw(n, g)[0:n_samp * stride:stride]    # Stride(K): K~[c] = K[c s]
    r_idx = [i * spb + t for t in range(spb) if (i * spb + t) * stride < L]
    qtil = np.stack([qw(n, g * G + hh)[r * stride] for hh in range(G) for r in r_idx])
    r_of_row = np.array([r for hh in range(G) for r in r_idx])
    # approximate logits Q~ K~^T / sqrt(d) with the causal mask over sampled positions (c <= r)
    logits = scale * (qtil @ ktil.T)
    logits[np.arange(n_samp)[None, :] > r_of_row[:, None]] = -np.inf
    # row softmax
    e = np.exp(logits - logits.max(axis=1, keepdims=True))
    shat = e / e.sum(axis=1, keepdims=True)
    # MaxPool over the sampled keys K_j of every key block j (masked keys contribute 0)
    padded = np.zeros((shat.shape[0], nb * spb))
    padded[:, :n_samp] = shat
    pooled = padded.reshape(shat.shape[0], nb, spb).max(axis=2)
    # MaxNorm per sampled row
    pbar = pooled / pooled.max(axis=1, keepdims=True)
    # block score (sum over sampled rows of the G heads) and max for the HRM flag
    return pbar.sum(axis=0), pbar.max(axis=0)


def kap_score(q_bits, k_bits, *, n_kv_heads: int, block: int, stride: int, sm_scale: float = 0.0,
              units: Optional[Iterable[Tuple[int, int, int]]] = None):
    """KAP block score S^KAP and HRM flag H per (n, g, i, j) (Eq. (score)).

    q_bits [B,Hq,L,d], k_bits [B,Hkv,L,d] are bf16 bit patterns. Entries j > i (non-causal) are 0;
    units not requested are NaN (score) / 255 (hrm).
    """
    qw, kw = _Heads(q_bits), _Heads(k_bits)
    B, Hq, L, d = qw.shape
    G = Hq // n_kv_heads
    nb = n_blocks(L, block)
    scale = default_scale(d, sm_scale)
    score = np.full((B, n_kv_heads, nb, nb), np.nan)
    hrm = np.full((B, n_kv_heads, nb, nb), 255, dtype=np.uint8)
    if units is None:
        units = [(n, g, i) for n in range(B) for g in range(n_kv_heads) for i in range(nb)]
    for (n, g, i) in units:
        s_i, hmax_i = _kap_unit(qw, kw, n, g, i, G, block, stride, scale, L)
        s_i[i + 1:] = 0.0
        score[n, g, i] = s_i
        h = (hmax_i == 1.0).astype(np.uint8)
        h[i + 1:] = 0
        hrm[n, g, i] = h
    return score, hrm


def kap_block_max(q_bits, k_bits, *, n_kv_heads: int, block: int, stride: int, sm_scale: float,
                  n: int, g: int, i: int):
    """Block maxima beta[row, j] of the scaled sampled logits for one unit (rows = G*spb).

    Used by the parity rules to find rows whose arg-max block is within rounding of a runner-up.
    """
    qw, kw = _Heads(q_bits), _Heads(k_bits)
    _, Hq, L, d = qw.shape
    G = Hq // n_kv_heads
    spb = block // stride
    nb = n_blocks(L, block)
    scale = default_scale(d, sm_scale)
    n_samp = -(-L // stride)
    ktil = kw(n, g)[0:n_samp * stride:stride]
    rows = []
    for hh in range(G):
        for t in range(spb):
            r = i * spb + t
            if r * stride >= L:
                break
            logit = scale * (ktil[:r + 1] @ qw(n, g * G + hh)[r * stride])
            beta = np.full(nb, -np.inf)
            for j in range(i + 1):
                c0, c1 = j * spb, min((j + 1) * spb, r + 1)
                if c0 < c1:
                    beta[j] = logit[c0:c1].max()
            rows.append(beta)
    return np.array(rows)


# ----------------------------------------------------------------------------------------------
# Stage 1 (cont.): flag-grouped sort and the ordered mask (Eq. (mkap), Algorithm A proxy stage)
# ----------------------------------------------------------------------------------------------
def budget_micro(value: float) -> int:
    """A stage-1 budget or top-p mass as an integer number of millionths (round half up).

    The budget arrives as float32; 0.2f is 0.200000003, and ceil(0.2f * 5) would keep 2 blocks
    instead of 1. Taking the budget at 1e-6 resolution and counting in integers removes every such
    representation artefact.
    """
    return int(math.floor(float(np.float32(value)) * 1e6 + 0.5))


def stage1_count(mode: int, value: float, n_cand: int, scores_sorted: Sequence[float],
                 row_total: float) -> int:
    """Number K_i of retained blocks for one query block with n_cand causal candidates.

    Fraction: K_i = B1 * (candidates) (Eq. (mkap)), rounded up and clamped to [1, n_cand], over the
    causal candidates j <= i. Top-p: the shortest prefix of the HRM-first order whose score mass
    reaches p of the row total (Algorithm A, proxy stage). The running mass is a float64 sum taken
    in list order, one term after another, against p (at 1e-6 resolution) times the total.
    """
    if mode == SELECT_ALL:
        return n_cand
    if mode == SELECT_FRACTION:
        bm = budget_micro(value)
        return min(n_cand, max(1, (bm * n_cand + 999_999) // 1_000_000))
    if mode == SELECT_TOP_P:
        target = (budget_micro(value) / 1e6) * row_total
        cum = 0.0
        for kk, s in enumerate(scores_sorted):
            cum += s
            if cum >= target:
                return kk + 1
        return n_cand
    raise ValueError(f"unknown selection mode {mode}")


def kap_select(score, hrm, *, mode: int, value: float, order_mode: int = ORDER_KAP,
               units: Optional[Iterable[Tuple[int, int, int]]] = None):
    """Ordered block list M_KAP (int32, -1 padded) and K_i per (n, g, i).

    The order rho_i puts the HRM group first and each group by descending score
    (Sec. 4.2 "Flag-grouped sorting"); the leading K_i entries are kept (Eq. (mkap)). With
    ORDER_ASCENDING the same kept set is listed by ascending block index (the un-remapped visit
    order used for comparison).
    """
    B, Hkv, nb, _ = score.shape
    order = np.full((B, Hkv, nb, nb), -1, dtype=np.int32)
    count = np.zeros((B, Hkv, nb), dtype=np.int32)
    if units is None:
        units = [(n, g, i) for n in range(B) for g in range(Hkv) for i in range(nb)]
    for (n, g, i) in units:
        cands = list(range(i + 1))
        hrm_grp = [j for j in cands if hrm[n, g, i, j]]
        rest = [j for j in cands if not hrm[n, g, i, j]]
        by_score = lambda j: (-float(score[n, g, i, j]), j)
        rho = sorted(hrm_grp, key=by_score) + sorted(rest, key=by_score)
        # the row mass: a float64 sum taken in ascending block index, one term after another
        total = 0.0
        for j in cands:
            total += float(score[n, g, i, j])
        K = stage1_count(mode, value, i + 1, [float(score[n, g, i, j]) for j in rho], total)
        kept = rho[:K]
        if order_mode == ORDER_ASCENDING:
            kept = sorted(kept)
        order[n, g, i, :K] = kept
        count[n, g, i] = K
    return order, count


# ----------------------------------------------------------------------------------------------
# Stage 2: Ordered-Skipping Kernel (Sec. 4.3, Eq. (skip), Algorithm A attention loop)
# ----------------------------------------------------------------------------------------------
def _rows_of_block(i: int, block: int, L: int) -> Tuple[int, int]:
    return i * block, min((i + 1) * block, L)


def osk_unit(qw, kw, vw, n, h, g, i, blocks: Sequence[int], *, block, scale, skip_on, tau, L,
             force_skip: Optional[Sequence[bool]] = None):
    """Walk one query block's list in order (Algorithm A attention loop), step by step.

    qw/kw/vw map (n, head) to float64 [L, d] arrays. Returns (O_i [rows, d], visit codes, margins
    d_k in nats) for the listed blocks. force_skip (tests only) replaces the threshold rule by a
    given per-visit decision, to check the output against the restricted-softmax closed form for
    arbitrary skip sets.
    """
    t0, t1 = _rows_of_block(i, block, L)
    Qi = qw(n, h)[t0:t1]
    rows = np.arange(t0, t1)
    m = np.full(t1 - t0, -np.inf)
    l = np.zeros(t1 - t0)
    O = np.zeros((t1 - t0, qw.shape[-1]))
    visits, margins = [], []
    for j in blocks:
        c0, c1 = j * block, min((j + 1) * block, L)
        Kj, Vj = kw(n, g)[c0:c1], vw(n, g)[c0:c1]
        S = scale * (Qi @ Kj.T)
        S[np.arange(c0, c1)[None, :] > rows[:, None]] = -np.inf          # causal mask
        m_loc = S.max(axis=1)
        m_prev = m
        m = np.maximum(m, m_loc)
        d_k = float(np.max(m_loc - m))
        margins.append(d_k)
        skip = (d_k < tau and skip_on) if force_skip is None else bool(force_skip[len(margins) - 1])
        if skip:
            visits.append(VISIT_SKIPPED)
            continue
        P = np.exp(S - m[:, None])
        alpha = np.exp(m_prev - m)
        l = alpha * l + P.sum(axis=1)
        O = alpha[:, None] * O + P @ Vj
        visits.append(VISIT_COMPUTED)
    return O / l[:, None], visits, margins


def osk_attention(q_bits, k_bits, v_bits, order, count, *, block: int, sm_scale: float = 0.0,
                  skip_mode: int = SKIP_NONE, delta: float = 0.0,
                  units: Optional[Iterable[Tuple[int, int, int]]] = None):
    """OSK output and per-visit logs for query-head units (n, h, i).

    With units=None every unit is computed and the result holds full arrays: o [B,Hq,L,d] float64,
    visit uint8 [B,Hq,nb,nb] and margin float64 [B,Hq,nb,nb] indexed by list position (0 / NaN
    beyond count), n_computed int32 [B,Hq,nb]. With explicit units the same quantities are returned
    per unit in dicts keyed by (n, h, i) (o: [rows, d]; visit, margin: [count]; n_computed: int).
    """
    qw, kw, vw = _Heads(q_bits), _Heads(k_bits), _Heads(v_bits)
    B, Hq, L, d = qw.shape
    Hkv = kw.shape[1]
    G = Hq // Hkv
    nb = n_blocks(L, block)
    scale = default_scale(d, sm_scale)
    skip_on = skip_mode == SKIP_ROWMAX and delta > 0
    tau = tau_from_delta(delta, L) if skip_on else 0.0
    full = units is None
    if full:
        units = [(n, h, i) for n in range(B) for h in range(Hq) for i in range(nb)]
        o = np.full((B, Hq, L, d), np.nan)
        visit = np.zeros((B, Hq, nb, nb), dtype=np.uint8)
        margin = np.full((B, Hq, nb, nb), np.nan)
        ncomp = np.full((B, Hq, nb), -1, dtype=np.int32)
    else:
        o, visit, margin, ncomp = {}, {}, {}, {}
    for (n, h, i) in units:
        g = h // G
        blocks = [int(x) for x in order[n, g, i, :count[n, g, i]]]
        Oi, vis, mar = osk_unit(qw, kw, vw, n, h, g, i, blocks, block=block, scale=scale,
                                skip_on=skip_on, tau=tau, L=L)
        nc = sum(1 for x in vis if x == VISIT_COMPUTED)
        if full:
            t0, t1 = _rows_of_block(i, block, L)
            o[n, h, t0:t1] = Oi
            visit[n, h, i, :len(vis)] = vis
            margin[n, h, i, :len(mar)] = mar
            ncomp[n, h, i] = nc
        else:
            o[(n, h, i)] = Oi
            visit[(n, h, i)] = np.array(vis, dtype=np.uint8)
            margin[(n, h, i)] = np.array(mar)
            ncomp[(n, h, i)] = nc
    return {"o": o, "visit": visit, "margin": margin, "n_computed": ncomp, "tau": tau}


# ----------------------------------------------------------------------------------------------
# Dense causal attention (Sec. 3.1) and its restriction to a block set (closed forms)
# ----------------------------------------------------------------------------------------------
def restricted_attention_rows(qw, kw, vw, n, h, g, rows: np.ndarray, blocks: Iterable[int], *,
                              block: int, scale: float, L: int) -> np.ndarray:
    """softmax over the causal keys of the given key blocks, times V, for the given query rows."""
    keys = np.concatenate([np.arange(j * block, min((j + 1) * block, L)) for j in sorted(blocks)])
    S = scale * (qw(n, h)[rows] @ kw(n, g)[keys].T)
    S[keys[None, :] > rows[:, None]] = -np.inf
    S = S - S.max(axis=1, keepdims=True)
    P = np.exp(S)
    return (P @ vw(n, g)[keys]) / P.sum(axis=1, keepdims=True)


def dense_attention(q_bits, k_bits, v_bits, *, block: int, sm_scale: float = 0.0,
                    units: Optional[Iterable[Tuple[int, int, int]]] = None):
    """Causal softmax attention O = softmax(QK^T/sqrt(d) + causal mask) V.

    units=None: full array [B,Hq,L,d]; otherwise a dict (n, h, i) -> rows of query block i.
    """
    qw, kw, vw = _Heads(q_bits), _Heads(k_bits), _Heads(v_bits)
    B, Hq, L, d = qw.shape
    Hkv = kw.shape[1]
    G = Hq // Hkv
    nb = n_blocks(L, block)
    scale = default_scale(d, sm_scale)
    full = units is None
    if full:
        units = [(n, h, i) for n in range(B) for h in range(Hq) for i in range(nb)]
        o = np.full((B, Hq, L, d), np.nan)
    else:
        o = {}
    for (n, h, i) in units:
        t0, t1 = _rows_of_block(i, block, L)
        Oi = restricted_attention_rows(qw, kw, vw, n, h, h // G, np.arange(t0, t1), range(i + 1),
                                       block=block, scale=scale, L=L)
        if full:
            o[n, h, t0:t1] = Oi
        else:
            o[(n, h, i)] = Oi
    return o


def block_mass(q_bits, k_bits, *, n_kv_heads: int, block: int, sm_scale: float = 0.0,
               units: Optional[Iterable[Tuple[int, int, int]]] = None):
    """Exact attention mass that each query block puts on each key block, per KV group.

    The ground truth behind the proxy-fidelity comparison of Sec. 3.2 (Property 1): the "oracle
    mask" ranks the key blocks of a query block by the probability mass full attention assigns to
    them. For batch n, KV head g, query block i and key block j <= i:
        mass[n, g, i, j] = sum over the query heads h of group g and the rows r of block i of
                           sum over the keys c of block j with c <= r of P_h[r, c],
    with P_h[r, :] = softmax over the causal keys of sm_scale * Q_h[r] . K_g[c]. Each row's
    probabilities sum to one, so the masses of row block i sum to G times its row count.
    units=None: full array [B, Hkv, nb, nb] (entries j > i are 0); otherwise a dict
    (n, g, i) -> float64 [i + 1].
    """
    qw, kw = _Heads(q_bits), _Heads(k_bits)
    B, Hq, L, d = qw.shape
    G = Hq // n_kv_heads
    nb = n_blocks(L, block)
    scale = default_scale(d, sm_scale)
    full = units is None
    if full:
        units = [(n, g, i) for n in range(B) for g in range(n_kv_heads) for i in range(nb)]
        out = np.zeros((B, n_kv_heads, nb, nb))
    else:
        out = {}
    for (n, g, i) in units:
        t0, t1 = _rows_of_block(i, block, L)
        rows = np.arange(t0, t1)
        keys = np.arange(0, t1)
        acc = np.zeros(i + 1)
        for h in range(g * G, (g + 1) * G):
            S = scale * (qw(n, h)[rows] @ kw(n, g)[keys].T)
            S[keys[None, :] > rows[:, None]] = -np.inf
            P = np.exp(S - S.max(axis=1, keepdims=True))
            P /= P.sum(axis=1, keepdims=True)
            for j in range(i + 1):
                acc[j] += P[:, j * block:min((j + 1) * block, L)].sum()
        if full:
            out[n, g, i, :i + 1] = acc
        else:
            out[(n, g, i)] = acc
    return out


# ----------------------------------------------------------------------------------------------
# Budgets and the skip-scale calibration
# ----------------------------------------------------------------------------------------------
def causal_blocks(seq_len: int, block: int) -> int:
    nb = n_blocks(seq_len, block)
    return nb * (nb + 1) // 2


def realized_budgets(count, n_computed, *, seq_len: int, block: int, n_q_heads: int):
    """Realized stage-1 budget B1 = listed/causal and overall budget B = computed/causal.

    The overall budget is the stage-1 budget minus the in-kernel skip ratio (Sec. 5.3, footnote).
    Both are over query-head tiles: a KV head's list is walked once per query head of its group.
    """
    B, Hkv, nb = count.shape
    G = n_q_heads // Hkv
    total = B * n_q_heads * causal_blocks(seq_len, block)
    listed = int(count.sum()) * G
    computed = int(np.asarray(n_computed).sum())
    return listed / total, computed / total


def calibrate_delta(margins: np.ndarray, *, listed: int, total_causal: int, target_budget: float,
                    seq_len: int) -> Tuple[float, int]:
    """Choose Delta so that the kernel computes round(target * total_causal) of the listed visits.

    A visit's margin d_k does not depend on Delta (the running max is updated before the test and a
    skip never changes it while tau <= 0), so the computed set for threshold tau is exactly
    {d_k >= tau}. tau is put at the midpoint of the gap around the cut; margins of 0 can never be
    skipped, so the reachable budget is capped. Returns (Delta, expected number of skips).
    """
    m = np.sort(np.asarray(margins, dtype=np.float64).ravel())
    want_skip = listed - int(round(target_budget * total_causal))
    n_neg = int(np.searchsorted(m, 0.0, side="left"))
    n_skip = max(0, min(want_skip, n_neg))
    if n_skip == 0:
        tau = (m[0] - 1.0) if (len(m) and m[0] < 0) else -1.0   # below every margin: skip nothing
    else:
        hi = min(m[n_skip], 0.0) if n_skip < len(m) else 0.0
        tau = 0.5 * (m[n_skip - 1] + hi)
    delta = seq_len * math.exp(tau)
    return float(delta), n_skip


# ----------------------------------------------------------------------------------------------
# Packed variable-length batches: independent causal sequences along one token axis
# ----------------------------------------------------------------------------------------------
def packed_spans(cu_blocks: Sequence[int], block: int) -> List[Tuple[int, int, int, int]]:
    """(first block F, end block E, first token, end token) of every packed sequence; sequence q
    owns blocks [cu_blocks[q], cu_blocks[q + 1])."""
    cu = [int(x) for x in cu_blocks]
    return [(cu[q], cu[q + 1], cu[q] * block, cu[q + 1] * block) for q in range(len(cu) - 1)]


def prefill_varlen(q_bits, k_bits, v_bits, cu_blocks, *, n_kv_heads: int, block: int, stride: int,
                   sm_scale: float = 0.0, select_mode: int = SELECT_FRACTION,
                   select_value: float = 1.0, order_mode: int = ORDER_KAP,
                   skip_mode: int = SKIP_NONE, delta: float = 0.0):
    """Algorithm A on a pack of sequences, each one its own causal prefill problem.

    The proxy (Eq. (score)), the stage-1 cut (Eq. (mkap)) and the OSK walk (Eq. (skip), with N the
    sequence's own length in the threshold ln(Delta/N)) run on the tokens of one sequence alone;
    their block indices are then shifted by the sequence's first block into the packed arrays.
    Entries that pair blocks of different sequences stay at the unit-not-computed values (score
    NaN, hrm 255) and -1 in the order rows.
    """
    B, Hq, L, d = q_bits.shape
    nb = n_blocks(L, block)
    score = np.full((B, n_kv_heads, nb, nb), np.nan)
    hrm = np.full((B, n_kv_heads, nb, nb), 255, dtype=np.uint8)
    order = np.full((B, n_kv_heads, nb, nb), -1, dtype=np.int32)
    count = np.zeros((B, n_kv_heads, nb), dtype=np.int32)
    o = np.full((B, Hq, L, d), np.nan)
    visit = np.zeros((B, Hq, nb, nb), dtype=np.uint8)
    margin = np.full((B, Hq, nb, nb), np.nan)
    ncomp = np.full((B, Hq, nb), -1, dtype=np.int32)
    taus = []
    for (F, E, t0, t1) in packed_spans(cu_blocks, block):
        qs = np.ascontiguousarray(q_bits[:, :, t0:t1])
        ks = np.ascontiguousarray(k_bits[:, :, t0:t1])
        vs = np.ascontiguousarray(v_bits[:, :, t0:t1])
        sc, hr = kap_score(qs, ks, n_kv_heads=n_kv_heads, block=block, stride=stride,
                           sm_scale=sm_scale)
        od, ct = kap_select(sc, hr, mode=select_mode, value=select_value, order_mode=order_mode)
        res = osk_attention(qs, ks, vs, od, ct, block=block, sm_scale=sm_scale,
                            skip_mode=skip_mode, delta=delta)
        n_q = E - F
        for i in range(n_q):
            score[:, :, F + i, F:F + i + 1] = sc[:, :, i, :i + 1]
            hrm[:, :, F + i, F:F + i + 1] = hr[:, :, i, :i + 1]
        shifted = np.where(od >= 0, od + F, -1).astype(np.int32)
        order[:, :, F:E, :n_q] = shifted
        count[:, :, F:E] = ct
        o[:, :, t0:t1] = res["o"]
        visit[:, :, F:E, :n_q] = res["visit"]
        margin[:, :, F:E, :n_q] = res["margin"]
        ncomp[:, :, F:E] = res["n_computed"]
        taus.append(res["tau"])
    return {"score": score, "hrm": hrm, "order": order, "count": count, "o": o, "visit": visit,
            "margin": margin, "n_computed": ncomp, "tau": taus}


def dense_attention_varlen(q_bits, k_bits, v_bits, cu_blocks, *, block: int,
                           sm_scale: float = 0.0):
    """Causal softmax attention within each packed sequence (Sec. 3.1 per sequence)."""
    B, Hq, L, d = q_bits.shape
    o = np.full((B, Hq, L, d), np.nan)
    for (F, E, t0, t1) in packed_spans(cu_blocks, block):
        o[:, :, t0:t1] = dense_attention(np.ascontiguousarray(q_bits[:, :, t0:t1]),
                                         np.ascontiguousarray(k_bits[:, :, t0:t1]),
                                         np.ascontiguousarray(v_bits[:, :, t0:t1]), block=block,
                                         sm_scale=sm_scale)
    return o
