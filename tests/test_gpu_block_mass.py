"""Exact block attention mass on the GPU (cosa_block_mass) against the oracle's definition."""
import sys

import numpy as np
import pytest

from oracle import cosa_oracle as O
from paper_2607_25291_amd import binding as B
from paper_2607_25291_amd.inputs import WORKLOADS, Workload, make_inputs
from tests.gpu_util import Run, torch

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


SMALL_GQA = Workload("small_gqa", 2, 8, 2, 2048, 128, 128, 16, 0.25, 0.125, 256, (0.005, 0.03))


def gpu_mass(w, q, k):
    p = B.Problem(w.batch, w.n_q_heads, w.n_kv_heads, w.seq_len, w.head_dim, w.block, w.stride)
    run = Run.upload(p, q, k, k)
    nb = w.n_blocks
    out = []
    for _ in range(2):
        m = run._zeros((w.batch, w.n_kv_heads, nb, nb), torch().float32)
        B.cosa_block_mass(p, run.q, run.k, m)
        torch().cuda.synchronize()
        out.append(m.cpu().numpy())
    assert np.array_equal(out[0], out[1]), "block mass is not deterministic"
    return out[0]


@pytest.mark.parametrize("name", ["tiny_l2k", "small_gqa"])
def test_block_mass_full(name):
    w = WORKLOADS["tiny_l2k"] if name == "tiny_l2k" else SMALL_GQA
    say(f"[block mass] {w.name}")
    q, k, v = make_inputs(w)
    G, b = w.n_q_heads // w.n_kv_heads, w.block
    got = gpu_mass(w, q, k)
    ref = O.block_mass(q, k, n_kv_heads=w.n_kv_heads, block=b)
    np.testing.assert_allclose(got, ref, rtol=2e-4, atol=1e-5 * G * b)
    nb = w.n_blocks
    tot = np.array([[[got[n, g, i, :i + 1].sum() for i in range(nb)] for g in range(w.n_kv_heads)]
                    for n in range(w.batch)])
    np.testing.assert_allclose(tot, G * b, rtol=1e-4)
    say(f"  max abs err {np.abs(got - ref).max():.2e} (row block total {G * b})")


def test_block_mass_sampled_32k():
    w = WORKLOADS["qwen3_8b_l32k"]
    say(f"[block mass] {w.name}, sampled units")
    q, k, v = make_inputs(w)
    G, b = w.n_q_heads // w.n_kv_heads, w.block
    got = gpu_mass(w, q, k)
    units = [(0, 0, 0), (0, 3, 130), (0, 7, w.n_blocks - 1)]
    ref = O.block_mass(q, k, n_kv_heads=w.n_kv_heads, block=b, units=units)
    for (n, g, i) in units:
        np.testing.assert_allclose(got[n, g, i, :i + 1], ref[(n, g, i)], rtol=2e-4,
                                   atol=1e-5 * G * b)
        assert abs(got[n, g, i, :i + 1].sum() - G * b) < 1e-4 * G * b
