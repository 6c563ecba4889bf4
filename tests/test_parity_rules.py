"""The comparison rules of tests/parity.py reject planted mistakes and accept what they excuse.

Runs on the CPU: the "GPU" rows here are the oracle's own rows with a mistake planted in them.
"""
import numpy as np
import pytest

from oracle import cosa_oracle as O
from tests import parity as PR


def _row_case(nb=12, seed=3):
    rng = np.random.default_rng(seed)
    s = rng.uniform(0.5, 4.0, (1, 1, nb, nb))
    h = np.zeros((1, 1, nb, nb), np.uint8)
    for i in range(nb):
        s[0, 0, i, i + 1:] = 0
        h[0, 0, i, rng.integers(0, i + 1)] = 1
    return s, h


def test_identical_rows_pass():
    s, h = _row_case()
    o, c = O.kap_select(s, h, mode=O.SELECT_FRACTION, value=0.5)
    units = [(0, 0, i) for i in range(12)]
    same, exc = PR.check_orders(o.copy(), c.copy(), o, c, s, h, units)
    assert same == 12 and exc == 0


@pytest.mark.parametrize("plant", ["repeat", "out_of_range", "swap_far", "count", "hrm_group"])
def test_planted_list_mistakes_fail(plant):
    s, h = _row_case()
    o, c = O.kap_select(s, h, mode=O.SELECT_FRACTION, value=0.5)
    go, gc = o.copy(), c.copy()
    i = 11
    K = int(c[0, 0, i])
    if plant == "repeat":
        go[0, 0, i, 1] = go[0, 0, i, 0]
    elif plant == "out_of_range":
        go[0, 0, i, K - 1] = i + 1
    elif plant == "swap_far":           # replace a kept block by the worst dropped one
        dropped = [j for j in range(i + 1) if j not in go[0, 0, i, :K]]
        go[0, 0, i, K - 1] = min(dropped, key=lambda j: s[0, 0, i, j])
    elif plant == "count":
        gc[0, 0, i] = K - 1
        go[0, 0, i, K - 1] = -1
    else:                                # a non-HRM block moved ahead of the HRM one
        go[0, 0, i, [0, 1]] = go[0, 0, i, [1, 0]]
    with pytest.raises(AssertionError):
        PR.check_orders(go, gc, o, c, s, h, [(0, 0, i)])


def test_near_tie_swap_is_excused():
    s, h = _row_case()
    i = 9
    o, c = O.kap_select(s, h, mode=O.SELECT_ALL, value=1.0)
    a, b = int(o[0, 0, i, 3]), int(o[0, 0, i, 4])
    if h[0, 0, i, a] != h[0, 0, i, b]:
        pytest.skip("neighbours in different HRM groups")
    s[0, 0, i, b] = s[0, 0, i, a] * (1 - 1e-4)      # a near-tie, GPU lists them the other way
    o, c = O.kap_select(s, h, mode=O.SELECT_ALL, value=1.0)
    go = o.copy()
    go[0, 0, i, [3, 4]] = go[0, 0, i, [4, 3]]
    same, exc = PR.check_orders(go, c, o, c, s, h, [(0, 0, i)])
    assert exc == 1


def test_top_p_count_only_at_a_near_tie():
    """A count that differs from the oracle's passes only when the running mass sits at the cut."""
    s = np.zeros((1, 1, 4, 4))
    h = np.zeros((1, 1, 4, 4), np.uint8)
    s[0, 0, 3] = [0.4, 0.3, 0.2, 0.1]
    p = 0.7
    o, c = O.kap_select(s, h, mode=O.SELECT_TOP_P, value=np.float32(p))
    assert int(c[0, 0, 3]) == 2            # 0.4 + 0.3 reaches 0.7 of 1.0 (within float rounding)
    units = [(0, 0, 3)]
    # one more entry: the oracle's mass after 2 entries is 0.7, at the target: excused
    go, gc = o.copy(), c.copy()
    go[0, 0, 3, 2] = 2
    gc[0, 0, 3] = 3
    PR.check_orders(go, gc, o, c, s, h, units, top_p=p)
    # two more entries: the mass after 3 entries (0.9) is far from the target: rejected
    go2, gc2 = go.copy(), gc.copy()
    go2[0, 0, 3, 3] = 3
    gc2[0, 0, 3] = 4
    with pytest.raises(AssertionError):
        PR.check_orders(go2, gc2, o, c, s, h, units, top_p=p)
    # an extra entry that does not continue the oracle's order: rejected
    go3 = go.copy()
    go3[0, 0, 3, 2] = 3
    with pytest.raises(AssertionError):
        PR.check_orders(go3, gc, o, c, s, h, units, top_p=p)
    # without top_p every count difference fails
    with pytest.raises(AssertionError):
        PR.check_orders(go, gc, o, c, s, h, units)


def test_skip_decision_band():
    tau = -2.0
    ora_margin = np.array([0.0, -2.00001, -5.0])
    ora_visit = np.array([1, 2, 2], np.uint8)
    assert PR.check_visits(np.array([1, 1, 2], np.uint8), ora_visit, ora_margin, tau, 3) == 1
    with pytest.raises(AssertionError):
        PR.check_visits(np.array([1, 2, 1], np.uint8), ora_visit, ora_margin, tau, 3)


def test_output_bounds():
    ref = np.zeros((4, 8))
    PR.check_output(ref + 1e-3, ref)
    with pytest.raises(AssertionError):
        PR.check_output(ref + 3e-3, ref)                 # mean above 2e-3
    bad = ref.copy()
    bad[0, 0] = 3e-2
    with pytest.raises(AssertionError):
        PR.check_output(bad, ref)                        # max above 2e-2
