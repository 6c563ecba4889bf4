"""Persistent OSK with work queues: cosa_osk_attention_queued must equal cosa_osk_attention bit for bit.

The queued launch runs the same tile code on a grid of one workgroup per compute unit that takes
(query block, head pair) tiles from per-XCD queues, so every output, log entry and computed count is
the same as with one workgroup per tile. The cases cover two head slots per workgroup (b = 128 and
b = 64), one head slot (odd group size), batch > 1, a queue buffer holding stale values, repeated
calls on the same queue, and the 128K shape of the benchmark (skip threshold ln(Delta/L) = -3).
The oracle parity of the walk itself is covered by the hardware-dispatched path's tests, and
cosa_prefill, which runs the queued launch, is compared with the stage calls there.
"""
import math
import sys

import numpy as np
import pytest

from paper_2607_25291_amd import binding as B
from paper_2607_25291_amd.inputs import WORKLOADS, Workload, make_inputs
from tests.gpu_util import dev, torch

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


CASES = [
    # name, B, Hq, Hkv, L, d, b, s, stage-1 budget, (overall budget unused), window, salient keys
    Workload("pair_b128_batch2", 2, 8, 2, 2048, 128, 128, 16, 0.5, 0.25, 256, (0.005, 0.03)),
    Workload("pair_b64", 1, 4, 2, 1536, 128, 64, 8, 0.5, 0.25, 256, 0.02),
    Workload("single_slot_g3", 1, 6, 2, 2048, 128, 128, 16, 0.4, 0.2, 256, 0.02),
    Workload("one_head_full_budget", 1, 1, 1, 1024, 128, 64, 8, 1.0, 0.5, 128, 0.02),
]


def lists(p, q, k, budget):
    t = torch()
    nb = p.n_blocks
    shp = (p.batch, p.n_kv_heads, nb, nb)
    score = t.zeros(shp, dtype=t.float32, device="cuda")
    hrm = t.zeros(shp, dtype=t.uint8, device="cuda")
    order = t.zeros(shp, dtype=t.int32, device="cuda")
    count = t.zeros(shp[:3], dtype=t.int32, device="cuda")
    B.cosa_kap_score(p, q, k, score, hrm)
    B.cosa_kap_select_ordered(p, score, hrm, B.select(B.SELECT_FRACTION, budget), order, count)
    return order, count


def walk(p, q, k, v, order, count, sk, queue=None):
    t = torch()
    nb = p.n_blocks
    o = t.full_like(q, 0x7BCD)
    vis = t.zeros((p.batch, p.n_q_heads, nb, nb), dtype=t.uint8, device="cuda")
    mar = t.zeros((p.batch, p.n_q_heads, nb, nb), dtype=t.float32, device="cuda")
    nco = t.full((p.batch, p.n_q_heads, nb), -1, dtype=t.int32, device="cuda")
    if queue is None:
        B.cosa_osk_attention(p, q, k, v, order, count, sk, o, vis, mar, nco)
    else:
        B.cosa_osk_attention_queued(p, q, k, v, order, count, sk, o, queue, queue.numel(), vis, mar,
                                    nco)
    t.cuda.synchronize()
    return [x.cpu().numpy() for x in (o, vis, mar, nco)]


@pytest.mark.parametrize("w", CASES, ids=lambda w: w.name)
def test_queued_equals_one_workgroup_per_tile(w):
    say(f"[queued case] {w.name}: B={w.batch} Hq={w.n_q_heads} Hkv={w.n_kv_heads} L={w.seq_len} "
        f"b={w.block} s={w.stride} B1={w.kap_budget}")
    t = torch()
    q, k, v = make_inputs(w)
    p = B.Problem(w.batch, w.n_q_heads, w.n_kv_heads, w.seq_len, w.head_dim, w.block, w.stride)
    qd, kd, vd = dev(q), dev(k), dev(v)
    order, count = lists(p, qd, kd, w.kap_budget)
    # a threshold at the median margin of the listed visits, so that about half are skipped
    _, vis0, mar0, _ = walk(p, qd, kd, vd, order, count, None)
    margins = mar0[vis0 == B.VISIT_COMPUTED]
    tau = float(np.median(margins[margins < 0])) if (margins < 0).any() else -1.0
    sk = B.skip(B.SKIP_ROWMAX, min(w.seq_len * math.exp(tau), float(w.seq_len)))
    ref = walk(p, qd, kd, vd, order, count, sk)
    queue = t.full((B.cosa_osk_attention_queue_bytes(),), 0xFF, dtype=t.uint8, device="cuda")
    for rep in range(2):  # stale queue contents first, then the counters the first call left
        got = walk(p, qd, kd, vd, order, count, sk, queue)
        for a, g in zip(ref, got):
            assert np.array_equal(a, g), f"call {rep}"
    assert (ref[3] >= 1).all()  # every tile ran (the first listed block is always computed)
    assert (ref[1] == B.VISIT_SKIPPED).any() and (ref[1] == B.VISIT_COMPUTED).any()


def test_queued_equals_one_workgroup_per_tile_full_size():
    w = WORKLOADS["qwen3_8b_l128k"]
    say(f"[queued full size] {w.name}")
    t = torch()
    q, k, v = make_inputs(w)
    p = B.Problem(w.batch, w.n_q_heads, w.n_kv_heads, w.seq_len, w.head_dim, w.block, w.stride)
    qd, kd, vd = dev(q), dev(k), dev(v)
    del q, k, v
    order, count = lists(p, qd, kd, w.kap_budget)
    sk = B.skip(B.SKIP_ROWMAX, w.seq_len * math.exp(-3.0))
    nb = p.n_blocks
    outs = []
    for queued in (False, True):
        o = t.empty_like(qd)
        nco = t.full((p.batch, p.n_q_heads, nb), -1, dtype=t.int32, device="cuda")
        if queued:
            queue = t.zeros((B.cosa_osk_attention_queue_bytes(),), dtype=t.uint8, device="cuda")
            B.cosa_osk_attention_queued(p, qd, kd, vd, order, count, sk, o, queue, queue.numel(),
                                        None, None, nco)
        else:
            B.cosa_osk_attention(p, qd, kd, vd, order, count, sk, o, None, None, nco)
        t.cuda.synchronize()
        outs.append((o, nco.cpu().numpy()))
    assert t.equal(outs[0][0], outs[1][0])
    assert np.array_equal(outs[0][1], outs[1][1])
    assert (outs[0][1] >= 1).all()
