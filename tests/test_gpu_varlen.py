"""Packed variable-length batches on the GPU (several causal sequences along one token axis).

A pack must behave as its sequences run one at a time: the packed entry points are checked
* against the oracle's packed composition (scores, HRM flags, lists, skip decisions, outputs) with
  the comparison rules of tests/parity.py, on two small packs;
* bit for bit against separate GPU calls on each sequence alone (proxy tensors on each block's own
  candidates, lists shifted by the sequence's first block, logs and outputs), at small sizes and
  at the 128K-token shape of the benchmark split into four sequences;
* bit for bit between the paged and the contiguous packed prefill, and between the packed and the
  per-sequence dense kernel.
"""
import dataclasses
import sys

import numpy as np
import pytest

from oracle import cosa_oracle as O
from paper_2607_25291_amd import binding as B
from paper_2607_25291_amd.inputs import WORKLOADS, Workload, make_inputs
from tests import parity as PR
from tests.gpu_util import Run, bf16_to_f64, dev, host_bits, torch

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def packed_inputs(w: Workload, blocks, seed0=0):
    """Structured inputs of every sequence (own seed), concatenated along the token axis."""
    parts = [make_inputs(dataclasses.replace(w, seq_len=nb * w.block, seed=seed0 + s))
             for s, nb in enumerate(blocks)]
    cu = np.concatenate([[0], np.cumsum(blocks)]).astype(int).tolist()
    q, k, v = (np.ascontiguousarray(np.concatenate([p[x] for p in parts], axis=2)) for x in range(3))
    return q, k, v, cu


# (workload, blocks per packed sequence, Delta); Delta is at most the shortest sequence's length
# and large enough that the oracle skips some visits in every case.
SMALL = Workload("pack_small_gqa", 1, 8, 2, 0, 128, 128, 16, 0.75, 0.25, 256, (0.005, 0.03))
TINY = Workload("pack_tiny", 1, 1, 1, 0, 128, 64, 8, 0.5, 0.25, 256, 0.02)
CASES = {
    "small_gqa": (SMALL, [4, 2, 10, 6], 256.0),
    "tiny": (TINY, [5, 11, 16], 300.0),
}


def problem(w, L):
    return B.Problem(w.batch, w.n_q_heads, w.n_kv_heads, L, w.head_dim, w.block, w.stride)


def gpu_prefill_varlen(p, cu, run, sel, sk, paged=None):
    """Packed prefill with logs: proxy and list stages through the packed entry points, then the
    packed OSK with logs; returns host arrays."""
    t = torch()
    nb = p.n_blocks
    vl = B.varlen(cu)
    score = run._zeros((p.batch, p.n_kv_heads, nb, nb), t.float32)
    hrm = run._zeros((p.batch, p.n_kv_heads, nb, nb), t.uint8)
    order = run._zeros((p.batch, p.n_kv_heads, nb, nb), t.int32)
    count = run._zeros((p.batch, p.n_kv_heads, nb), t.int32)
    B.cosa_kap_score_varlen(p, vl, run.q, run.k, score, hrm)
    B.cosa_kap_select_ordered_varlen(p, vl, score, hrm, sel, order, count)
    o = run._zeros((p.batch, p.n_q_heads, p.seq_len, p.head_dim), t.int16)
    visit = run._zeros((p.batch, p.n_q_heads, nb, nb), t.uint8)
    margin = run._zeros((p.batch, p.n_q_heads, nb, nb), t.float32)
    ncomp = run._zeros((p.batch, p.n_q_heads, nb), t.int32)
    B.cosa_osk_attention_varlen(p, vl, run.q, run.k, run.v, order, count, sk, o, visit, margin,
                                ncomp)
    t.cuda.synchronize()
    return dict(score=score.cpu().numpy(), hrm=hrm.cpu().numpy(), order=order.cpu().numpy(),
                count=count.cpu().numpy(), o=host_bits(o), visit=visit.cpu().numpy(),
                margin=margin.cpu().numpy(), ncomp=ncomp.cpu().numpy())


def gpu_prefill_single(w, q, k, v, sel, sk):
    """Unpacked calls on one sequence; returns host arrays."""
    p = problem(w, q.shape[2])
    run = Run.upload(p, q, k, v)
    score, hrm = run.kap_score()
    order, count = run.kap_select(score, hrm, sel)
    o, visit, margin, ncomp = run.osk(order, count, sk)
    torch().cuda.synchronize()
    return dict(score=score.cpu().numpy(), hrm=hrm.cpu().numpy(), order=order.cpu().numpy(),
                count=count.cpu().numpy(), o=host_bits(o), visit=visit.cpu().numpy(),
                margin=margin.cpu().numpy(), ncomp=ncomp.cpu().numpy())


def assert_pack_equals_singles(w, q, k, v, cu, packed, sel, sk):
    for s in range(len(cu) - 1):
        F, E = cu[s], cu[s + 1]
        t0, t1 = F * w.block, E * w.block
        single = gpu_prefill_single(w, *(np.ascontiguousarray(x[:, :, t0:t1]) for x in (q, k, v)),
                                    sel, sk)
        n = E - F
        for i in range(n):
            assert np.array_equal(packed["score"][:, :, F + i, F:F + i + 1],
                                  single["score"][:, :, i, :i + 1]), (s, i)
            assert np.array_equal(packed["hrm"][:, :, F + i, F:F + i + 1],
                                  single["hrm"][:, :, i, :i + 1]), (s, i)
        shifted = np.where(single["order"] >= 0, single["order"] + F, -1)
        assert np.array_equal(packed["order"][:, :, F:E, :n], shifted), s
        assert (packed["order"][:, :, F:E, n:] == -1).all()
        assert np.array_equal(packed["count"][:, :, F:E], single["count"]), s
        assert np.array_equal(packed["o"][:, :, t0:t1], single["o"]), s
        assert np.array_equal(packed["visit"][:, :, F:E, :n], single["visit"]), s
        assert np.array_equal(packed["margin"][:, :, F:E, :n], single["margin"]), s
        assert np.array_equal(packed["ncomp"][:, :, F:E], single["ncomp"]), s


@pytest.fixture(scope="module", params=list(CASES))
def case(request):
    w, blocks, delta = CASES[request.param]
    q, k, v, cu = packed_inputs(w, blocks)
    L = cu[-1] * w.block
    say(f"[varlen case] {request.param}: Hq={w.n_q_heads} Hkv={w.n_kv_heads} b={w.block} "
        f"blocks {blocks} delta {delta}")
    p = problem(w, L)
    return dict(w=w, q=q, k=k, v=v, cu=cu, p=p, run=Run.upload(p, q, k, v), delta=delta)


def test_varlen_matches_oracle(case):
    w, p, cu = case["w"], case["p"], case["cu"]
    sel = B.select(B.SELECT_FRACTION, w.kap_budget)
    sk = B.skip(B.SKIP_ROWMAX, case["delta"])
    got = gpu_prefill_varlen(p, cu, case["run"], sel, sk)
    ora = O.prefill_varlen(case["q"], case["k"], case["v"], cu, n_kv_heads=w.n_kv_heads,
                           block=w.block, stride=w.stride, select_mode=O.SELECT_FRACTION,
                           select_value=w.kap_budget, skip_mode=O.SKIP_ROWMAX,
                           delta=case["delta"])
    spans = O.packed_spans(cu, w.block)
    # proxy and list, on each block's own candidates
    for (F, E, t0, t1) in spans:
        qs, ks = (np.ascontiguousarray(x[:, :, t0:t1]) for x in (case["q"], case["k"]))
        units = [(n, g, i) for n in range(w.batch) for g in range(w.n_kv_heads) for i in range(E - F)]
        frag = lambda n, g, i: PR.fragile_blocks(qs, ks, n_kv_heads=w.n_kv_heads, block=w.block,
                                                 stride=w.stride, sm_scale=0.0, n=n, g=g, i=i)
        sub = lambda a: a[:, :, F:E, F:E]
        PR.check_scores(sub(got["score"]), sub(got["hrm"]), sub(ora["score"]), sub(ora["hrm"]),
                        units, frag)
        shift = lambda a: np.where(a[:, :, F:E, :E - F] >= 0, a[:, :, F:E, :E - F] - F, -1)
        ora_sub_score = np.nan_to_num(sub(ora["score"]))
        PR.check_orders(shift(got["order"]), got["count"][:, :, F:E], shift(ora["order"]),
                        ora["count"][:, :, F:E], ora_sub_score, sub(ora["hrm"]), units, frag)
    # skip decisions and output, where the GPU walked the oracle's list (identical rows)
    G = w.n_q_heads // w.n_kv_heads
    excused = skipped = 0
    for (F, E, t0, t1) in spans:
        s = spans.index((F, E, t0, t1))
        for n in range(w.batch):
            for h in range(w.n_q_heads):
                for i in range(F, E):
                    c = int(ora["count"][n, h // G, i])
                    if not np.array_equal(got["order"][n, h // G, i, :c],
                                          ora["order"][n, h // G, i, :c]):
                        continue
                    excused += PR.check_visits(got["visit"][n, h, i], ora["visit"][n, h, i],
                                               ora["margin"][n, h, i], ora["tau"][s], c)
                    skipped += int((ora["visit"][n, h, i, :c] == O.VISIT_SKIPPED).sum())
    assert skipped > 0, "the case should exercise the skip rule"
    mx, mean = PR.check_output(bf16_to_f64(got["o"]), ora["o"])
    say(f"  oracle parity: {skipped} oracle skips, {excused} excused decisions, "
        f"max-abs {mx:.2e} mean-abs {mean:.2e}")


def test_varlen_equals_separate_calls(case):
    w = case["w"]
    sel = B.select(B.SELECT_FRACTION, w.kap_budget)
    sk = B.skip(B.SKIP_ROWMAX, case["delta"])
    got = gpu_prefill_varlen(case["p"], case["cu"], case["run"], sel, sk)
    assert_pack_equals_singles(w, case["q"], case["k"], case["v"], case["cu"], got, sel, sk)


def test_varlen_prefill_entry_points(case):
    """cosa_prefill_varlen and cosa_prefill_paged_varlen give the staged packed results."""
    w, p, cu, run = case["w"], case["p"], case["cu"], case["run"]
    t = torch()
    sel = B.select(B.SELECT_FRACTION, w.kap_budget)
    sk = B.skip(B.SKIP_ROWMAX, case["delta"])
    staged = gpu_prefill_varlen(p, cu, run, sel, sk)
    nbytes = B.cosa_prefill_workspace_bytes(p)
    ws = run._zeros((nbytes,), t.uint8)
    o = run._zeros((p.batch, p.n_q_heads, p.seq_len, p.head_dim), t.int16)
    vl = B.varlen(cu)
    B.cosa_prefill_varlen(p, vl, run.q, run.k, run.v, sel, sk, ws, nbytes, o)
    t.cuda.synchronize()
    assert np.array_equal(host_bits(o), staged["o"])
    # paged cache: a random page table over 32-token pages
    page = 32
    Bt, Hkv, L, d = case["k"].shape
    per_seq = L // page
    n_pages = Bt * per_seq + 5
    rng = np.random.default_rng(5)
    table = rng.permutation(n_pages).astype(np.int32)[:Bt * per_seq].reshape(Bt, per_seq)
    kc = rng.integers(0, 2 ** 16, size=(n_pages, Hkv, page, d), dtype=np.uint16) & np.uint16(0xBFFF)
    vc = rng.integers(0, 2 ** 16, size=(n_pages, Hkv, page, d), dtype=np.uint16) & np.uint16(0xBFFF)
    for n in range(Bt):
        for lp in range(per_seq):
            kc[table[n, lp]] = case["k"][n, :, lp * page:(lp + 1) * page, :]
            vc[table[n, lp]] = case["v"][n, :, lp * page:(lp + 1) * page, :]
    kcd, vcd, tbd = dev(kc), dev(vc), dev(table)
    kv = B.paged_kv(kcd, vcd, tbd, page, n_pages)
    o2 = run._zeros((p.batch, p.n_q_heads, p.seq_len, p.head_dim), t.int16)
    ws.zero_()
    B.cosa_prefill_paged_varlen(p, vl, run.q, kv, sel, sk, ws, nbytes, o2)
    t.cuda.synchronize()
    assert np.array_equal(host_bits(o2), staged["o"])


def test_dense_varlen_equals_separate_calls(case):
    w, p, cu, run = case["w"], case["p"], case["cu"], case["run"]
    t = torch()
    o = run._zeros((p.batch, p.n_q_heads, p.seq_len, p.head_dim), t.int16)
    B.cosa_dense_attention_varlen(p, B.varlen(cu), run.q, run.k, run.v, o)
    t.cuda.synchronize()
    packed = host_bits(o)
    for s in range(len(cu) - 1):
        t0, t1 = cu[s] * w.block, cu[s + 1] * w.block
        parts = [np.ascontiguousarray(x[:, :, t0:t1]) for x in (case["q"], case["k"], case["v"])]
        single = Run.upload(problem(w, t1 - t0), *parts).dense()
        t.cuda.synchronize()
        assert np.array_equal(packed[:, :, t0:t1], host_bits(single)), s
    ora = O.dense_attention_varlen(case["q"], case["k"], case["v"], cu, block=w.block)
    PR.check_output(bf16_to_f64(packed), ora)


def test_varlen_full_size_equals_separate_calls():
    """The 128K-token benchmark shape (32 query / 8 KV heads) packed as 64K + 32K + 16K + 16K."""
    w = WORKLOADS["qwen3_8b_l128k"]
    blocks = [512, 256, 128, 128]
    say(f"[varlen full size] {w.name} split into blocks {blocks}")
    q, k, v, cu = packed_inputs(w, blocks, seed0=100)
    p = problem(w, cu[-1] * w.block)
    run = Run.upload(p, q, k, v)
    sel = B.select(B.SELECT_FRACTION, w.kap_budget)
    sk = B.skip(B.SKIP_ROWMAX, 4096.0)
    got = gpu_prefill_varlen(p, cu, run, sel, sk)
    del run
    assert_pack_equals_singles(w, q, k, v, cu, got, sel, sk)
    skipped = int((got["visit"] == B.VISIT_SKIPPED).sum())
    say(f"  {int(got['count'].sum())} listed entries, {skipped} skipped visits")
    assert skipped > 0
