"""Pins of the oracle's exact block attention mass (Sec. 3.2, Property 1 ground truth)."""
import math

import numpy as np
import pytest

from oracle import cosa_oracle as O
from paper_2607_25291_amd.inputs import random_inputs


def _bits(a):
    """float64 values exactly representable in bf16 -> bit patterns."""
    f = np.asarray(a, np.float32)
    return (f.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def test_rows_sum_to_one():
    q, k, v = random_inputs(2, 4, 2, 256, 128, 3, 1.0)
    m = O.block_mass(q, k, n_kv_heads=2, block=64)
    for i in range(4):
        np.testing.assert_allclose(m[:, :, i, :i + 1].sum(axis=-1), 2 * 64, rtol=1e-12)
        assert (m[:, :, i, i + 1:] == 0).all()


def test_zero_queries_closed_form():
    # Q = 0: every causal key of a row gets 1 / (r + 1); block j collects the keys of j up to r.
    q, k, v = random_inputs(1, 2, 1, 192, 128, 5, 1.0)
    q = np.zeros_like(q)
    m = O.block_mass(q, k, n_kv_heads=1, block=64)
    for i in range(3):
        for j in range(i + 1):
            want = 0.0
            for r in range(i * 64, (i + 1) * 64):
                n_keys = max(0, min(r, (j + 1) * 64 - 1) - j * 64 + 1)
                want += n_keys / (r + 1)
            assert m[0, 0, i, j] == pytest.approx(2 * want, rel=1e-12)


def test_equals_dense_attention_of_block_indicators():
    # Attention output with V[c] = one-hot(block of c) is, per row, the vector of block masses.
    Bt, Hq, Hkv, L, d, b = 1, 4, 2, 256, 128, 64
    q, k, _ = random_inputs(Bt, Hq, Hkv, L, d, 9, 1.0)
    nb = L // b
    v = np.zeros((Bt, Hkv, L, d), np.float32)
    for c in range(L):
        v[:, :, c, c // b] = 1.0
    o = O.dense_attention(q, k, _bits(v), block=b)
    m = O.block_mass(q, k, n_kv_heads=Hkv, block=b)
    G = Hq // Hkv
    for g in range(Hkv):
        for i in range(nb):
            rows = o[0, g * G:(g + 1) * G, i * b:(i + 1) * b, :nb].sum(axis=(0, 1))
            np.testing.assert_allclose(m[0, g, i], rows, rtol=1e-11, atol=1e-12)


def test_dominant_key_takes_the_mass():
    # One key with a huge logit for every row (a sink): its block receives almost all the mass.
    Bt, Hq, Hkv, L, d, b = 1, 2, 1, 192, 128, 64
    q = np.full((Bt, Hq, L, d), 0.25, np.float32)
    k = np.zeros((Bt, Hkv, L, d), np.float32)
    k[0, 0, 5] = 4.0            # logit 0.25 * 4 * 128 / sqrt(128) = 11.3 nats above the others
    m = O.block_mass(_bits(q), _bits(k), n_kv_heads=1, block=b)
    for i in range(1, 3):
        assert m[0, 0, i, 0] > 0.99 * 2 * b
    assert math.isclose(m[0, 0, 2].sum(), 2 * b, rel_tol=1e-12)


def test_units_match_full():
    q, k, v = random_inputs(1, 2, 1, 256, 128, 13, 1.0)
    full = O.block_mass(q, k, n_kv_heads=1, block=64)
    part = O.block_mass(q, k, n_kv_heads=1, block=64, units=[(0, 0, 3), (0, 0, 1)])
    np.testing.assert_array_equal(part[(0, 0, 3)], full[0, 0, 3, :4])
    np.testing.assert_array_equal(part[(0, 0, 1)], full[0, 0, 1, :2])
