"""Pins of the oracle's flag-grouped sort, stage-1 cut and budget accounting (Sec. 4.2, Eq. (mkap)).

Checked by brute force and closed forms, not by re-running the oracle's own sort:
* every list is a set of distinct causal candidates, HRM group first, score non-increasing inside
  each group, ties by ascending index, and the kept set is the top-K_i under that key;
* K_i follows the fractional-budget formula; the tiny workload keeps 272 of 528 causal blocks;
* top-p keeps the shortest prefix of the HRM-first order reaching p of the row mass;
* ascending mode keeps the same set in index order.
"""
import itertools
import math

import numpy as np
import pytest

from oracle import cosa_oracle as O
from paper_2607_25291_amd.inputs import WORKLOADS, make_inputs


def _random_scores(nb, seed, ties=False):
    rng = np.random.default_rng(seed)
    s = rng.uniform(0.01, 8.0, (1, 1, nb, nb))
    if ties:
        s = np.round(s)            # many exact ties -> index tie-break matters
    h = (rng.uniform(size=(1, 1, nb, nb)) < 0.2).astype(np.uint8)
    for i in range(nb):
        s[0, 0, i, i + 1:] = 0
        h[0, 0, i, i + 1:] = 0
    return s, h


@pytest.mark.parametrize("ties", [False, True])
def test_order_properties_full_budget(ties):
    nb = 24
    s, h = _random_scores(nb, 3, ties)
    order, count = O.kap_select(s, h, mode=O.SELECT_ALL, value=1.0)
    for i in range(nb):
        lst = order[0, 0, i, :count[0, 0, i]].tolist()
        assert count[0, 0, i] == i + 1 and sorted(lst) == list(range(i + 1))
        assert (order[0, 0, i, i + 1:] == -1).all()
        keys = [(-int(h[0, 0, i, j]), -s[0, 0, i, j], j) for j in lst]
        assert all(a < b for a, b in zip(keys, keys[1:]))


def test_brute_force_top_k_tiny():
    """For i <= 5 enumerate every subset of size K_i: the kept set is the unique best one."""
    nb = 6
    s, h = _random_scores(nb, 5, ties=True)
    for frac in (0.2, 0.5, 0.75):
        order, count = O.kap_select(s, h, mode=O.SELECT_FRACTION, value=frac)
        for i in range(nb):
            K = count[0, 0, i]
            assert K == min(i + 1, max(1, math.ceil(round(frac * 1e6) * (i + 1) / 1e6 - 1e-12)))
            key = lambda j: (int(h[0, 0, i, j]), s[0, 0, i, j], -j)
            best = max(itertools.combinations(range(i + 1), K),
                       key=lambda c: sorted((key(j) for j in c), reverse=True))
            assert set(order[0, 0, i, :K].tolist()) == set(best)


def test_fraction_budget_closed_form():
    # tiny workload: nb = 32, B1 = 50% -> sum_i ceil((i+1)/2) = 272 of 528 causal blocks
    assert sum(min(i + 1, max(1, math.ceil(0.5 * (i + 1)))) for i in range(32)) == 272
    w = WORKLOADS["tiny_l2k"]
    q, k, _ = make_inputs(w)
    s, h = O.kap_score(q, k, n_kv_heads=1, block=w.block, stride=w.stride)
    order, count = O.kap_select(s, h, mode=O.SELECT_FRACTION, value=w.kap_budget)
    assert count.sum() == 272 and O.causal_blocks(w.seq_len, w.block) == 528
    b1, b = O.realized_budgets(count, count.repeat(1, axis=1), seq_len=w.seq_len, block=w.block,
                               n_q_heads=1)
    assert b1 == 272 / 528 and b == 272 / 528
    # float32 0.2 is 0.200000003: 5 candidates must keep 1 block, 15 keep 3, 16 keep 4
    assert O.stage1_count(O.SELECT_FRACTION, 0.2, 5, [], 0.0) == 1
    assert O.stage1_count(O.SELECT_FRACTION, 0.2, 15, [], 0.0) == 3
    assert O.stage1_count(O.SELECT_FRACTION, 0.2, 16, [], 0.0) == 4
    assert O.stage1_count(O.SELECT_FRACTION, 0.1, 1024, [], 0.0) == 103
    assert O.stage1_count(O.SELECT_FRACTION, 1e-7, 1024, [], 0.0) == 1


def test_top_p():
    s = np.zeros((1, 1, 3, 3))
    h = np.zeros((1, 1, 3, 3), np.uint8)
    s[0, 0, 2] = [0.5, 0.3, 0.2]
    for p, K, lst in [(0.8, 2, [0, 1]), (0.81, 3, [0, 1, 2]), (0.5, 1, [0]), (1.0, 3, [0, 1, 2])]:
        order, count = O.kap_select(s, h, mode=O.SELECT_TOP_P, value=np.float32(p))
        assert count[0, 0, 2] == K and order[0, 0, 2, :K].tolist() == lst, p
    # the HRM block comes first even with the lowest score; the mass is counted in that order
    h[0, 0, 2, 2] = 1
    order, count = O.kap_select(s, h, mode=O.SELECT_TOP_P, value=0.6)
    assert count[0, 0, 2] == 2 and order[0, 0, 2, :2].tolist() == [2, 0]   # 0.2 + 0.5 >= 0.6


def test_ascending_mode_same_set():
    nb = 20
    s, h = _random_scores(nb, 7)
    o1, c1 = O.kap_select(s, h, mode=O.SELECT_FRACTION, value=0.3)
    o2, c2 = O.kap_select(s, h, mode=O.SELECT_FRACTION, value=0.3, order_mode=O.ORDER_ASCENDING)
    assert np.array_equal(c1, c2)
    for i in range(nb):
        K = c1[0, 0, i]
        assert sorted(o1[0, 0, i, :K].tolist()) == o2[0, 0, i, :K].tolist()


@pytest.mark.parametrize("p", [0.3, 0.5, 0.9, 0.95, 0.999])
def test_top_p_exact_rational(p):
    """Top-p count against exact rational arithmetic: the smallest k whose prefix mass (in the
    HRM-first order) reaches p of the row mass. The oracle sums in float64, so the two may differ
    only where the exact prefix mass lies within float64 rounding of the target; such rows are
    counted and must be rare, every other row must agree exactly."""
    from fractions import Fraction
    nb = 64
    rng = np.random.default_rng(11)
    s = rng.gamma(0.7, 1.0, (1, 1, nb, nb)).astype(np.float32).astype(np.float64)
    h = (rng.uniform(size=(1, 1, nb, nb)) < 0.1).astype(np.uint8)
    for i in range(nb):
        s[0, 0, i, i + 1:] = 0
        h[0, 0, i, i + 1:] = 0
    order, count = O.kap_select(s, h, mode=O.SELECT_TOP_P, value=np.float32(p))
    pm = Fraction(O.budget_micro(np.float32(p)), 10 ** 6)
    near = 0
    for i in range(nb):
        row = [(-int(h[0, 0, i, j]), -s[0, 0, i, j], j) for j in range(i + 1)]
        rho = [j for (_, _, j) in sorted(row)]
        total = sum(Fraction(float(s[0, 0, i, j])) for j in range(i + 1))
        target = pm * total
        cum, k_exact, masses = Fraction(0), i + 1, []
        for k, j in enumerate(rho):
            cum += Fraction(float(s[0, 0, i, j]))
            masses.append(cum)
            if cum >= target:
                k_exact = k + 1
                break
        K = int(count[0, 0, i])
        assert order[0, 0, i, :K].tolist() == rho[:K]
        if K != k_exact:
            near += 1
            assert abs(float(masses[min(K, k_exact) - 1] - target)) <= 1e-12 * float(total), i
    assert near <= 1
