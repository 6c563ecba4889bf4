"""The allocation-free prefill (cosa_prefill_noalloc, workspace in the library's static scratch
array) against cosa_prefill with a caller workspace, through the C ABI on the same inputs: two calls
in a row, the second on a smaller problem, each bit-identical to cosa_prefill's output (same
kernels, so nothing looser than bit equality is accepted). Also: a problem whose workspace exceeds
the scratch array is rejected before anything is enqueued, and the output buffer is left untouched.
"""
import math
import sys

import numpy as np
import pytest

from paper_2607_25291_amd import binding as B
from paper_2607_25291_amd.inputs import Workload, make_inputs, random_inputs
from tests.gpu_util import Run, host_bits, torch

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _pair(run, sel, sk):
    """(cosa_prefill output, cosa_prefill_noalloc output) on the same inputs."""
    t = torch()
    p = run.problem
    o_ref = run.prefill(sel, sk)[0]
    o = t.full((p.batch, p.n_q_heads, p.seq_len, p.head_dim), 0x7FC0, dtype=t.int16,
               device="cuda")
    B.cosa_prefill_noalloc(p, run.q, run.k, run.v, sel, sk, o)
    t.cuda.synchronize()
    return host_bits(o_ref), host_bits(o)


def test_noalloc_prefill_matches_prefill():
    # first call: GQA 8/2, batch 2, L = 4096, b = 128, structured inputs, fraction cut with skipping
    w = Workload("noalloc_gqa", 2, 8, 2, 4096, 128, 128, 16, 0.25, 0.125, 256, (0.005, 0.03))
    say(f"[noalloc] call 1: B={w.batch} Hq={w.n_q_heads} Hkv={w.n_kv_heads} L={w.seq_len}")
    q, k, v = make_inputs(w)
    p1 = B.Problem(w.batch, w.n_q_heads, w.n_kv_heads, w.seq_len, w.head_dim, w.block, w.stride)
    assert B.cosa_prefill_workspace_bytes(p1) <= B.NOALLOC_SCRATCH_BYTES
    run1 = Run.upload(p1, q, k, v)
    sel1 = B.select(B.SELECT_FRACTION, w.kap_budget)
    sk1 = B.skip(B.SKIP_ROWMAX, w.seq_len * math.exp(-1.0))
    ref, got = _pair(run1, sel1, sk1)
    assert np.array_equal(ref, got)
    say(f"  bit-identical ({ref.size} outputs)")

    # second call, smaller: 1/1 heads, L = 1024, b = 64, unstructured inputs, top-p cut
    say("[noalloc] call 2: B=1 Hq=1 Hkv=1 L=1024 b=64")
    q2, k2, v2 = random_inputs(1, 1, 1, 1024, 128, seed=7, scale=1.5)
    p2 = B.Problem(1, 1, 1, 1024, 128, 64, 8)
    run2 = Run.upload(p2, q2, k2, v2)
    sel2 = B.select(B.SELECT_TOP_P, 0.9)
    sk2 = B.skip(B.SKIP_ROWMAX, 1024 * math.exp(-2.0))
    ref2, got2 = _pair(run2, sel2, sk2)
    assert np.array_equal(ref2, got2)
    say(f"  bit-identical ({ref2.size} outputs)")

    # the first problem again: what the second call left in the scratch array does not matter
    ref3, got3 = _pair(run1, sel1, sk1)
    assert np.array_equal(ref3, got3) and np.array_equal(got3, got)
    say("  first problem again: bit-identical")


def test_noalloc_rejects_oversized_problem():
    t = torch()
    p = B.Problem(1, 32, 16, 131072, 128, 128, 16)       # 208 MiB of workspace
    assert B.cosa_prefill_workspace_bytes(p) > B.NOALLOC_SCRATCH_BYTES
    o = t.full((4,), 1234, dtype=t.int16, device="cuda")
    with pytest.raises(B.CosaError) as e:
        B.cosa_prefill_noalloc(p, o, o, o, B.select(B.SELECT_FRACTION, 0.1), None, o)
    assert e.value.status == B.COSA_ERR_WORKSPACE
    t.cuda.synchronize()
    assert (o.cpu().numpy() == 1234).all()
    say(f"  rejected: {e.value}")
