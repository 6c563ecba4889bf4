"""Staged proxy scoring: cosa_kap_score_staged must equal cosa_kap_score bit for bit.

The staged path copies the sampled keys into a workspace in the order the matrix cores read them
and scores from that copy; with at most 32 proxy rows per query block it also scores two query
blocks per workgroup. The arithmetic and the summation order are the same, so score and HRM must
be identical. The cases cover every samples-per-block variant (4, 8, 16, 32) on both kernels, one
to four 32-row proxy tiles, a last chunk padded past the sampled keys, an odd number of query
blocks, batch > 1, and the 128K shape of the benchmark. The oracle
parity of the proxy itself is covered by the contiguous path's tests.
"""
import sys

import numpy as np
import pytest

from paper_2607_25291_amd import binding as B
from paper_2607_25291_amd.inputs import WORKLOADS, make_inputs, random_inputs
from tests.gpu_util import dev, torch

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


CASES = [
    # (B, Hq, Hkv, L, b, s)
    (1, 1, 1, 2048, 64, 8),      # 8 samples per block, one row tile
    (2, 8, 2, 2048, 128, 16),    # GQA 4:1, 32 proxy rows, batch 2
    (1, 4, 2, 1536, 64, 16),     # 4 samples per block
    (1, 4, 1, 1024, 128, 8),     # 16 samples per block, 64 rows (two tiles)
    (1, 4, 1, 1024, 128, 4),     # 32 samples per block, 128 rows (four tiles)
    (1, 2, 1, 320, 64, 16),      # 20 sampled keys: the only chunk is padded
    (1, 1, 1, 1024, 128, 8),     # 16 samples per block, 16 rows: paired query blocks
    (1, 2, 1, 2048, 128, 8),     # 16 samples per block, 32 rows: paired query blocks
    (1, 1, 1, 1024, 128, 4),     # 32 samples per block, 32 rows: paired query blocks
    (1, 4, 2, 1600, 64, 8),      # 25 query blocks: the last pair has one block
]


def scores(p, q, k, staged):
    t = torch()
    nb = p.n_blocks
    score = t.zeros((p.batch, p.n_kv_heads, nb, nb), dtype=t.float32, device="cuda")
    hrm = t.zeros((p.batch, p.n_kv_heads, nb, nb), dtype=t.uint8, device="cuda")
    if staged:
        nbytes = B.cosa_kap_score_workspace_bytes(p)
        ws = t.full((nbytes,), 0x7F, dtype=t.uint8, device="cuda")  # stale contents must not matter
        B.cosa_kap_score_staged(p, q, k, ws, nbytes, score, hrm)
    else:
        B.cosa_kap_score(p, q, k, score, hrm)
    t.cuda.synchronize()
    return score.cpu().numpy(), hrm.cpu().numpy()


@pytest.mark.parametrize("shape", CASES, ids=lambda c: "x".join(map(str, c)))
def test_staged_equals_in_place(shape):
    Bt, Hq, Hkv, L, b, s = shape
    say(f"[staged case] B={Bt} Hq={Hq} Hkv={Hkv} L={L} b={b} s={s}")
    q, k, _ = random_inputs(Bt, Hq, Hkv, L, 128, seed=L + s)
    p = B.Problem(Bt, Hq, Hkv, L, 128, b, s)
    qd, kd = dev(q), dev(k)
    s0, h0 = scores(p, qd, kd, staged=False)
    s1, h1 = scores(p, qd, kd, staged=True)
    assert np.array_equal(s0, s1)
    assert np.array_equal(h0, h1)
    assert h0.any()


def test_staged_equals_in_place_full_size():
    w = WORKLOADS["qwen3_8b_l128k"]
    say(f"[staged full size] {w.name}")
    q, k, _ = make_inputs(w)
    p = B.Problem(w.batch, w.n_q_heads, w.n_kv_heads, w.seq_len, w.head_dim, w.block, w.stride)
    qd, kd = dev(q), dev(k)
    del q, k
    s0, h0 = scores(p, qd, kd, staged=False)
    s1, h1 = scores(p, qd, kd, staged=True)
    assert np.array_equal(s0, s1)
    assert np.array_equal(h0, h1)
