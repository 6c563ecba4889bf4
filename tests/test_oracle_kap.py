"""Pins of the oracle's Kernel-Aware Proxy (Sec. 4.2, Eq. (score), Algorithm A proxy stage).

The oracle follows the paper's literal steps (softmax -> MaxPool -> MaxNorm -> sum / HRM flag).
These tests fix it from outside:
* a hand-worked example with closed-form scores (stride sampling offset, causal mask, MaxNorm);
* the algebraic identity Pbar = exp(beta - mu) (the softmax normaliser cancels in the ratio);
* closed forms for Q = 0 (uniform softmax);
* invariances: tokens between stride samples do not matter, later keys do not matter (causality),
  permuting query heads inside a group does not matter, groups are independent.
"""
import math

import numpy as np
import pytest

from oracle import cosa_oracle as O
from paper_2607_25291_amd.inputs import WORKLOADS, f32_to_bf16_bits, make_inputs, random_inputs


def _bits(a):
    return f32_to_bf16_bits(np.asarray(a, np.float32))


def test_hand_example():
    """L=8, d=2, b=4 (2 blocks), s=2 (2 samples per block), scale 1.

    Sampled tokens 0,2,4,6. Sampled keys K~ = [(1,0), (0,1), (2,0), (0,0)], sampled queries
    Q~ = [(1,0), (0,1), (1,0), (0,2)]. Row r sees keys c <= r.
      r0: logits [1]            -> P = [1, 0]            Pbar = [1, 0]
      r1: logits [0, 1]         -> P = [e/(1+e), 0]      Pbar = [1, 0]
      r2: logits [1, 0, 2]      -> P = [e, e^2] / Z      Pbar = [1/e, 1]
      r3: logits [0, 2, 0, 0]   -> P = [e^2, 1] / Z      Pbar = [1, e^-2]
    Query block 0 (rows 0,1): s00 = 2, HRM on block 0.
    Query block 1 (rows 2,3): s10 = 1 + 1/e, s11 = 1 + e^-2, both blocks HRM.
    """
    rng = np.random.default_rng(1)
    q = rng.standard_normal((1, 1, 8, 2)).astype(np.float32) * 5   # odd tokens: noise
    k = rng.standard_normal((1, 1, 8, 2)).astype(np.float32) * 5
    q[0, 0, 0::2] = [(1, 0), (0, 1), (1, 0), (0, 2)]
    k[0, 0, 0::2] = [(1, 0), (0, 1), (2, 0), (0, 0)]
    score, hrm = O.kap_score(_bits(q), _bits(k), n_kv_heads=1, block=4, stride=2, sm_scale=1.0)
    assert abs(score[0, 0, 0, 0] - 2.0) < 1e-15
    assert abs(score[0, 0, 1, 0] - (1 + math.exp(-1))) < 1e-15
    assert abs(score[0, 0, 1, 1] - (1 + math.exp(-2))) < 1e-15
    assert score[0, 0, 0, 1] == 0.0
    assert hrm[0, 0].tolist() == [[1, 0], [1, 1]]
    order, count = O.kap_select(score, hrm, mode=O.SELECT_ALL, value=1.0)
    assert order[0, 0, 1].tolist() == [0, 1]
    order, count = O.kap_select(score, hrm, mode=O.SELECT_FRACTION, value=0.5)
    assert count[0, 0].tolist() == [1, 1] and order[0, 0, 1].tolist() == [0, -1]


def _exp_form(q_bits, k_bits, Hkv, block, stride):
    """Pbar = exp(beta - mu): beta = block max of scaled sampled logits, mu = its row max."""
    qf, kf = O.widen(q_bits), O.widen(k_bits)
    B, Hq, L, d = qf.shape
    G, spb, nb = Hq // Hkv, block // stride, O.n_blocks(L, block)
    scale = O.default_scale(d)
    score = np.zeros((B, Hkv, nb, nb))
    hrm = np.zeros((B, Hkv, nb, nb), np.uint8)
    for n in range(B):
        for g in range(Hkv):
            kt = kf[n, g, ::stride]
            for i in range(nb):
                for hh in range(G):
                    for t in range(spb):
                        r = i * spb + t
                        if r * stride >= L:
                            continue
                        x = scale * (kt[:r + 1] @ qf[n, g * G + hh, r * stride])
                        beta = np.array([x[j * spb:(j + 1) * spb].max() for j in range(i + 1)])
                        mu = beta.max()
                        score[n, g, i, :i + 1] += np.exp(beta - mu)
                        hrm[n, g, i, :i + 1] |= (beta == mu).astype(np.uint8)
    return score, hrm


@pytest.mark.parametrize("B,Hq,Hkv,L,d,block,stride", [
    (1, 1, 1, 256, 32, 32, 4),
    (2, 4, 2, 192, 16, 32, 8),
    (1, 2, 1, 200, 16, 32, 4),     # ragged
])
def test_literal_steps_equal_exp_form(B, Hq, Hkv, L, d, block, stride):
    q, k, _ = random_inputs(B, Hq, Hkv, L, d, seed=B * 100 + L, scale=2.0)
    s_lit, h_lit = O.kap_score(q, k, n_kv_heads=Hkv, block=block, stride=stride)
    s_exp, h_exp = _exp_form(q, k, Hkv, block, stride)
    nb = O.n_blocks(L, block)
    low = np.tril(np.ones((nb, nb), bool))
    assert np.allclose(s_lit[..., low], s_exp[..., low], rtol=1e-12, atol=0)
    assert np.array_equal(h_lit[..., low], h_exp[..., low])


def test_zero_queries_closed_form():
    """Q = 0: uniform softmax over the visible sampled keys, so every visible block has Pbar = 1.

    Every sampled row of block i sees the first sampled key of every block j <= i, hence
    s_ij = G * spb and H_ij = 1 for all j <= i.
    """
    B, Hq, Hkv, L, d, block, stride = 1, 4, 2, 256, 16, 32, 4
    _, k, _ = random_inputs(B, Hq, Hkv, L, d, seed=2)
    q = np.zeros((B, Hq, L, d), np.uint16)
    score, hrm = O.kap_score(q, k, n_kv_heads=Hkv, block=block, stride=stride)
    nb, G, spb = L // block, Hq // Hkv, block // stride
    low = np.tril(np.ones((nb, nb), bool))
    assert np.all(score[..., low] == G * spb)
    assert np.all(hrm[..., low] == 1)
    assert np.all(score[..., ~low] == 0)


def test_invariances():
    B, Hq, Hkv, L, d, block, stride = 1, 4, 2, 256, 16, 32, 4
    q, k, _ = random_inputs(B, Hq, Hkv, L, d, seed=9, scale=2.0)
    kw = dict(n_kv_heads=Hkv, block=block, stride=stride)
    s0, h0 = O.kap_score(q, k, **kw)
    # tokens between stride samples are never read
    q2, k2 = q.copy(), k.copy()
    rng = np.random.default_rng(0)
    mask = (np.arange(L) % stride) != 0
    q2[:, :, mask] = _bits(rng.standard_normal(q2[:, :, mask].shape) * 3)
    k2[:, :, mask] = _bits(rng.standard_normal(k2[:, :, mask].shape) * 3)
    s1, h1 = O.kap_score(q2, k2, **kw)
    assert np.array_equal(s0, s1) and np.array_equal(h0, h1)
    # ... but a sampled token is
    q3 = q.copy()
    q3[0, 0, 43 * stride] = _bits(rng.standard_normal(d) * 3)   # sampled row 43, query block 5
    s3, _ = O.kap_score(q3, k, **kw)
    assert not np.array_equal(s0, s3)
    # causality: changing keys of block 5 leaves query blocks 0..4 unchanged
    k4 = k.copy()
    k4[0, 0, 5 * block:6 * block] = _bits(rng.standard_normal((block, d)) * 3)
    s4, h4 = O.kap_score(q, k4, **kw)
    assert np.array_equal(s0[0, 0, :5], s4[0, 0, :5]) and np.array_equal(h0[0, 0, :5], h4[0, 0, :5])
    assert not np.array_equal(s0[0, 0, 5], s4[0, 0, 5])
    # group 1 does not depend on group 0's keys
    assert np.array_equal(s0[0, 1], s4[0, 1])
    # permuting the query heads inside a group leaves the group's scores unchanged
    q5 = q[:, [1, 0, 3, 2]]
    s5, h5 = O.kap_score(q5, k, **kw)
    assert np.allclose(s0, s5, rtol=1e-14, atol=0, equal_nan=True) and np.array_equal(h0, h5)


def test_bounds_on_structured_input():
    w = WORKLOADS["tiny_l2k"]
    q, k, _ = make_inputs(w)
    score, hrm = O.kap_score(q, k, n_kv_heads=1, block=w.block, stride=w.stride)
    nb = w.n_blocks
    spb = w.block // w.stride
    for i in range(nb):
        s = score[0, 0, i, :i + 1]
        assert np.all(s > 0) and np.all(s <= spb + 1e-12)
        assert 1 <= hrm[0, 0, i, :i + 1].sum() <= spb
        # a block that holds the maximum of every sampled row reaches the top score spb
        if hrm[0, 0, i, :i + 1].sum() == 1:
            assert abs(s[hrm[0, 0, i, :i + 1] == 1][0] - spb) < 1e-12


def test_units_subset_matches_full():
    w = WORKLOADS["tiny_l2k"]
    q, k, _ = make_inputs(w)
    full_s, full_h = O.kap_score(q, k, n_kv_heads=1, block=w.block, stride=w.stride)
    part_s, part_h = O.kap_score(q, k, n_kv_heads=1, block=w.block, stride=w.stride,
                                 units=[(0, 0, 7), (0, 0, 31)])
    for i in (7, 31):
        assert np.array_equal(full_s[0, 0, i], part_s[0, 0, i])
        assert np.array_equal(full_h[0, 0, i], part_h[0, 0, i])
    assert np.isnan(part_s[0, 0, 8]).all()


def test_block_max_helper_consistent():
    w = WORKLOADS["tiny_l2k"]
    q, k, _ = make_inputs(w)
    score, hrm = O.kap_score(q, k, n_kv_heads=1, block=w.block, stride=w.stride)
    i = 20
    beta = O.kap_block_max(q, k, n_kv_heads=1, block=w.block, stride=w.stride, sm_scale=0.0,
                           n=0, g=0, i=i)
    mu = beta.max(axis=1, keepdims=True)
    assert np.allclose(np.exp(beta[:, :i + 1] - mu).sum(axis=0), score[0, 0, i, :i + 1],
                       rtol=1e-12)
    assert np.array_equal((beta[:, :i + 1] == mu).any(axis=0).astype(np.uint8),
                          hrm[0, 0, i, :i + 1])
