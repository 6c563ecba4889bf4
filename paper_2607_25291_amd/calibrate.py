"""Host-side choice of the skip scale Delta for a target overall budget (not part of the hot path).

The in-kernel skip (Eq. (skip)) skips a listed block when its margin d = max_r (m_loc - m) is below
tau = ln(Delta / N). The running max is updated before the test and a skip can only happen when the
block does not raise it, so the margins of a list walk are the same for every Delta: one walk with
the margin log enabled (cosa_osk_attention(..., margin_log=...), skipping off) gives all of them,
and the set computed at threshold tau is exactly {d >= tau}. Delta for a wanted number of skips is
therefore read off the sorted margins, with tau placed in the middle of the gap at the cut so that
float rounding of the logits cannot move a decision.
"""
from __future__ import annotations

import math

import numpy as np


def delta_for_budget(margins: np.ndarray, n_listed: int, n_causal: int, budget: float,
                     seq_len: int):
    """Return (delta, n_skipped, realized_budget) for an overall budget (computed / causal blocks).

    margins: every listed visit's margin (nats), n_listed of them; n_causal: number of causal
    (query-head tile, key block) pairs. Blocks with margin 0 (those that raise the running max, the
    first visit among them) can never be skipped, so the reachable budget is bounded below.
    """
    d = np.sort(np.asarray(margins, dtype=np.float64).reshape(-1))
    if d.size != n_listed:
        raise ValueError(f"{d.size} margins for {n_listed} listed visits")
    skippable = int(np.count_nonzero(d < 0.0))
    want = n_listed - int(round(budget * n_causal))
    k = min(max(want, 0), skippable)
    if k == 0:
        tau = float(d[0]) - 1.0 if d.size and d[0] < 0.0 else -1.0
    else:
        upper = float(d[k]) if k < d.size else 0.0
        tau = 0.5 * (float(d[k - 1]) + min(upper, 0.0))
    delta = seq_len * math.exp(tau)
    return delta, k, (n_listed - k) / n_causal


def delta_for_budget_packed(margins: np.ndarray, seq_lens: np.ndarray, n_causal: int,
                            budget: float):
    """delta_for_budget for packed sequences, where a visit of sequence q is skipped when its margin
    is below ln(delta / L_q) (Eq. (skip) with N = L_q). That is margin + ln L_q < ln delta, so one
    threshold on the shifted margins serves every sequence. delta is capped at the shortest
    length, which keeps every sequence's threshold <= 0.

    margins: every listed visit's margin (nats); seq_lens: the length of the sequence each visit
    belongs to (same shape). Returns (delta, n_skipped, realized_budget).
    """
    d = np.asarray(margins, dtype=np.float64).reshape(-1)
    lens = np.asarray(seq_lens, dtype=np.float64).reshape(-1)
    if d.shape != lens.shape:
        raise ValueError("one sequence length per margin")
    a = np.sort(d + np.log(lens))
    cap = math.log(float(lens.min())) if lens.size else 0.0
    skippable = int(np.count_nonzero(a < cap))
    want = a.size - int(round(budget * n_causal))
    k = min(max(want, 0), skippable)
    if k == 0:
        t = min(float(a[0]) - 1.0, cap) if a.size else cap
    else:
        upper = float(a[k]) if k < a.size else cap
        t = 0.5 * (float(a[k - 1]) + min(upper, cap))
    return math.exp(t), k, (a.size - k) / n_causal
