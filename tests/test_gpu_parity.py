"""Parity of the HIP path (through the C ABI) with the float64 oracle on the same seeded inputs.

Small problems are compared in full; the Qwen3-8B-shaped problems at 32K, 64K (8:1 GQA) and 128K run
the full GPU path in the benchmark's launch configuration and are compared on sampled
(head, query block) units that the oracle computes one by one. The comparison rules are in
tests/parity.py.
"""
import dataclasses
import math
import sys

import numpy as np
import pytest

from oracle import cosa_oracle as O
from paper_2607_25291_amd import binding as B
from paper_2607_25291_amd.calibrate import delta_for_budget
from paper_2607_25291_amd.inputs import WORKLOADS, Workload, make_inputs, random_inputs
from tests import parity as PR
from tests.gpu_util import Run, bf16_to_f64, dev, host_bits, tau_of, torch

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def problem_of(w: Workload) -> B.Problem:
    return B.Problem(w.batch, w.n_q_heads, w.n_kv_heads, w.seq_len, w.head_dim, w.block, w.stride)


SMALL_GQA = Workload("small_gqa", 2, 8, 2, 2048, 128, 128, 16, 0.25, 0.125, 256, (0.005, 0.03))
TINY = WORKLOADS["tiny_l2k"]


@pytest.fixture(scope="module", params=["tiny_l2k", "small_gqa"])
def case(request):
    w = TINY if request.param == "tiny_l2k" else SMALL_GQA
    say(f"[case] {w.name}: B={w.batch} Hq={w.n_q_heads} Hkv={w.n_kv_heads} L={w.seq_len} b={w.block}")
    q, k, v = make_inputs(w)
    run = Run.upload(problem_of(w), q, k, v)
    ora_s, ora_h = O.kap_score(q, k, n_kv_heads=w.n_kv_heads, block=w.block, stride=w.stride)
    return dict(w=w, q=q, k=k, v=v, run=run, ora_s=ora_s, ora_h=ora_h)


def all_units(w, per_q=False):
    H = w.n_q_heads if per_q else w.n_kv_heads
    return [(n, h, i) for n in range(w.batch) for h in range(H) for i in range(w.n_blocks)]


def fragile_fn(c):
    w = c["w"]
    return lambda n, g, i: PR.fragile_blocks(c["q"], c["k"], n_kv_heads=w.n_kv_heads,
                                             block=w.block, stride=w.stride, sm_scale=0.0,
                                             n=n, g=g, i=i)


def test_kap_score_full(case):
    w, run = case["w"], case["run"]
    say("[kap_score]", w.name)
    s, h = run.kap_score()
    gs, gh = s.cpu().numpy(), h.cpu().numpy()
    worst, excused = PR.check_scores(gs, gh, case["ora_s"], case["ora_h"], all_units(w),
                                     fragile_fn(case))
    say(f"  max rel score err {worst:.2e}, excused hrm flags {excused}")


@pytest.mark.parametrize("mode,value,order_mode", [
    (B.SELECT_FRACTION, None, B.ORDER_KAP), (B.SELECT_FRACTION, None, B.ORDER_ASCENDING),
    (B.SELECT_TOP_P, 0.95, B.ORDER_KAP), (B.SELECT_ALL, 1.0, B.ORDER_KAP)])
def test_kap_select(case, mode, value, order_mode):
    w, run = case["w"], case["run"]
    value = w.kap_budget if value is None else value
    say(f"[kap_select] {w.name} mode={mode} value={value} order={order_mode}")
    s, h = run.kap_score()
    order, count = run.kap_select(s, h, B.select(mode, value, order_mode))
    go, gc = order.cpu().numpy(), count.cpu().numpy()
    # (a) same scores in, the selection must be bit-exact with the oracle's rule
    gs64 = s.cpu().numpy().astype(np.float64)
    oo, oc = O.kap_select(gs64, h.cpu().numpy(), mode=mode, value=value, order_mode=order_mode)
    if mode == B.SELECT_TOP_P:
        same, exc = PR.check_orders(go, gc, oo, oc, gs64, h.cpu().numpy(), all_units(w),
                                    count_exact=False)
        assert exc <= max(1, len(all_units(w)) // 100)
    else:
        assert np.array_equal(gc, oc) and np.array_equal(go, oo)
    # (b) end to end against the oracle's own scores (near-ties excused)
    oo2, oc2 = O.kap_select(case["ora_s"], case["ora_h"], mode=mode, value=value,
                            order_mode=order_mode)
    same, exc = PR.check_orders(go, gc, oo2, oc2, case["ora_s"], case["ora_h"], all_units(w),
                                fragile_fn(case), count_exact=(mode != B.SELECT_TOP_P))
    say(f"  rows identical {same}, excused {exc}")
    assert exc <= max(2, len(all_units(w)) // 50)


def _oracle_lists(case, budget=None):
    w = case["w"]
    return O.kap_select(case["ora_s"], case["ora_h"], mode=O.SELECT_FRACTION,
                        value=w.kap_budget if budget is None else budget)


def test_osk_full_budget_is_dense(case):
    w, run, q, k, v = case["w"], case["run"], case["q"], case["k"], case["v"]
    say("[osk full budget]", w.name)
    ref = O.dense_attention(q, k, v, block=w.block)
    dense = bf16_to_f64(host_bits(run.dense()))
    mx, mean = PR.check_output(dense, ref)
    say(f"  dense max-abs {mx:.2e} mean-abs {mean:.2e}")
    nb = w.n_blocks
    for variant in ("ascending", "reversed", "kap"):
        if variant == "kap":
            order, count = O.kap_select(case["ora_s"], case["ora_h"], mode=O.SELECT_ALL, value=1.0)
        else:
            order = np.full((w.batch, w.n_kv_heads, nb, nb), -1, np.int32)
            count = np.zeros((w.batch, w.n_kv_heads, nb), np.int32)
            for i in range(nb):
                lst = np.arange(i + 1) if variant == "ascending" else np.arange(i, -1, -1)
                order[:, :, i, :i + 1] = lst
                count[:, :, i] = i + 1

        o, visit, margin, ncomp = run.osk(dev(order), dev(count))
        got = bf16_to_f64(host_bits(o))
        mx, mean = PR.check_output(got, ref)
        say(f"  {variant}: max-abs {mx:.2e} mean-abs {mean:.2e}")
        assert (ncomp.cpu().numpy() == np.repeat(count, w.n_q_heads // w.n_kv_heads, axis=1)).all()
        if variant == "ascending":
            assert np.array_equal(host_bits(o), host_bits(run.dense()))   # same tile code


def test_osk_skip_parity(case):
    w, run, q, k, v = case["w"], case["run"], case["q"], case["k"], case["v"]
    say("[osk skip]", w.name)

    order, count = _oracle_lists(case)
    base = O.osk_attention(q, k, v, order, count, block=w.block)
    total = w.batch * w.n_q_heads * O.causal_blocks(w.seq_len, w.block)
    mask = ~np.isnan(base["margin"])
    G = w.n_q_heads // w.n_kv_heads
    delta, n_skip = O.calibrate_delta(base["margin"][mask], listed=int(count.sum()) * G,
                                      total_causal=total, target_budget=w.osk_budget,
                                      seq_len=w.seq_len)
    ora = O.osk_attention(q, k, v, order, count, block=w.block, skip_mode=O.SKIP_ROWMAX,
                          delta=delta)
    o, visit, margin, ncomp = run.osk(dev(order), dev(count), B.skip(B.SKIP_ROWMAX, delta))
    gv, gm, gn = visit.cpu().numpy(), margin.cpu().numpy(), ncomp.cpu().numpy()
    # margins (nats) agree to fp32 accuracy; decisions bit-exact (band-excused)
    assert np.abs(gm[mask] - base["margin"][mask]).max() < 1e-4
    tau = ora["tau"]
    assert tau == tau_of(delta, w.seq_len)
    excused = 0
    for n in range(w.batch):
        for h in range(w.n_q_heads):
            for i in range(w.n_blocks):
                c = int(count[n, h // G, i])
                excused += PR.check_visits(gv[n, h, i], ora["visit"][n, h, i],
                                           ora["margin"][n, h, i], tau, c)
    say(f"  delta {delta:.4g} (tau {tau:.4f}), skips {n_skip}, excused decisions {excused}")
    assert excused == 0
    assert np.array_equal(gn, ora["n_computed"])
    mx, mean = PR.check_output(bf16_to_f64(host_bits(o)), ora["o"])
    say(f"  O max-abs {mx:.2e} mean-abs {mean:.2e}")


def test_osk_decisions_without_margin_log(case):
    """Without a margin log the kernel takes each skip decision from whether some row's margin
    reaches tau, instead of from the tile's maximum margin; decisions, counts and O must be the
    same bit for bit. Thresholds: the calibrated one, tau = 0 (Delta = L: only blocks where some
    row's maximum does not fall are computed) and a small Delta (almost nothing is skipped)."""
    w, run = case["w"], case["run"]
    say("[osk decisions without margin log]", w.name)
    order, count = _oracle_lists(case)
    od, cd = dev(order), dev(count)
    _, _, margin, _ = run.osk(od, cd, None)
    gm = margin.cpu().numpy()
    total = w.batch * w.n_q_heads * O.causal_blocks(w.seq_len, w.block)
    G = w.n_q_heads // w.n_kv_heads
    mask = np.arange(w.n_blocks)[None, None, None, :] < np.repeat(count, G, axis=1)[..., None]
    delta_cal, _, _ = delta_for_budget(gm[mask], int(count.sum()) * G, total, w.osk_budget,
                                       w.seq_len)
    t = torch()
    for delta in (delta_cal, float(w.seq_len), w.seq_len * math.exp(-8.0)):
        sk = B.skip(B.SKIP_ROWMAX, delta)
        o_ref, vis_ref, _, nco_ref = run.osk(od, cd, sk)
        o = t.zeros_like(o_ref)
        vis = t.zeros_like(vis_ref)
        nco = t.full_like(nco_ref, -1)
        B.cosa_osk_attention(run.problem, run.q, run.k, run.v, od, cd, sk, o, vis, None, nco)
        t.cuda.synchronize()
        assert np.array_equal(vis.cpu().numpy(), vis_ref.cpu().numpy()), delta
        assert np.array_equal(nco.cpu().numpy(), nco_ref.cpu().numpy()), delta
        assert np.array_equal(host_bits(o), host_bits(o_ref)), delta
        skipped = int((vis.cpu().numpy() == B.VISIT_SKIPPED).sum())
        say(f"  delta {delta:.4g}: {skipped} skipped of {int(count.sum()) * G} listed")


def test_prefill_matches_stages(case):
    w, run = case["w"], case["run"]
    say("[prefill]", w.name)
    sel = B.select(B.SELECT_FRACTION, w.kap_budget)
    sk = B.skip(B.SKIP_ROWMAX, w.seq_len * math.exp(-2.0))
    o, s, h, order, count = run.prefill(sel, sk)
    s2, h2 = run.kap_score()
    order2, count2 = run.kap_select(s2, h2, sel)
    o2, _, _, _ = run.osk(order2, count2, sk, logs=False)
    nb = w.n_blocks
    low = np.tril(np.ones((nb, nb), bool))
    assert np.array_equal(s.cpu().numpy()[..., low], s2.cpu().numpy()[..., low])
    assert np.array_equal(h.cpu().numpy()[..., low], h2.cpu().numpy()[..., low])
    assert np.array_equal(order.cpu().numpy(), order2.cpu().numpy())
    assert np.array_equal(count.cpu().numpy(), count2.cpu().numpy())
    assert np.array_equal(host_bits(o), host_bits(o2))
    # end-to-end against the oracle replaying the GPU's list
    ora = O.osk_attention(case["q"], case["k"], case["v"], order.cpu().numpy(),
                          count.cpu().numpy(), block=w.block, skip_mode=O.SKIP_ROWMAX,
                          delta=w.seq_len * math.exp(-2.0))
    PR.check_output(bf16_to_f64(host_bits(o)), ora["o"])


def test_repeatable(case):
    """Bit-identical results across repeated runs (no races in LDS or the vote)."""
    w, run = case["w"], case["run"]
    sel = B.select(B.SELECT_FRACTION, w.kap_budget)
    sk = B.skip(B.SKIP_ROWMAX, w.seq_len * math.exp(-2.0))
    outs = [run.prefill(sel, sk) for _ in range(3)]
    for o, s, h, order, count in outs[1:]:
        assert np.array_equal(host_bits(o), host_bits(outs[0][0]))
        assert np.array_equal(order.cpu().numpy(), outs[0][3].cpu().numpy())


def test_edge_single_block_and_batch():
    """L == b (one block, diagonal only), batch 3, unstructured inputs."""
    for (Bt, Hq, Hkv, L, b, s) in [(3, 4, 2, 128, 128, 16), (1, 2, 2, 64, 64, 8),
                                   (2, 2, 1, 384, 128, 32), (1, 1, 1, 256, 64, 16)]:
        say(f"[edge] B={Bt} Hq={Hq} Hkv={Hkv} L={L} b={b} s={s}")
        q, k, v = random_inputs(Bt, Hq, Hkv, L, 128, seed=L + Bt, scale=1.5)
        p = B.Problem(Bt, Hq, Hkv, L, 128, b, s)
        run = Run.upload(p, q, k, v)
        ref = O.dense_attention(q, k, v, block=b)
        PR.check_output(bf16_to_f64(host_bits(run.dense())), ref)
        o, sc, hr, order, count = run.prefill(B.select(B.SELECT_ALL), None)
        PR.check_output(bf16_to_f64(host_bits(o)), ref)
        os_, oh = O.kap_score(q, k, n_kv_heads=Hkv, block=b, stride=s)
        nb = L // b
        units = [(n, g, i) for n in range(Bt) for g in range(Hkv) for i in range(nb)]
        PR.check_scores(sc.cpu().numpy(), hr.cpu().numpy(), os_, oh, units,
                        lambda n, g, i: PR.fragile_blocks(q, k, n_kv_heads=Hkv, block=b, stride=s,
                                                          sm_scale=0.0, n=n, g=g, i=i))


def test_empty_problem_on_gpu():
    import torch
    p = B.Problem(0, 4, 2, 1024)
    B.cosa_prefill(p, None, None, None, B.select(B.SELECT_ALL), None, None, 0, None)
    torch.cuda.synchronize()


# --------------------------------------------------------------------------------------------
# Full-size workloads: whole GPU path, sampled oracle units
# --------------------------------------------------------------------------------------------
def _sample_units(w, n_heads, n_blocks_sample, per_q):
    nb = w.n_blocks
    G = w.n_q_heads // w.n_kv_heads
    blocks = sorted(set(np.linspace(0, nb - 1, n_blocks_sample).round().astype(int).tolist()))
    if per_q:
        heads = [0, w.n_q_heads - 1] if n_heads >= 2 else [0]
        heads = heads + [G * (w.n_kv_heads // 2) + 1][:max(0, n_heads - 2)]
    else:
        heads = [0, w.n_kv_heads - 1][:n_heads]
    return [(0, h, i) for h in heads for i in blocks]


@pytest.mark.parametrize("name,n_blocks_sample", [("qwen3_8b_l32k", 12), ("wide_gqa_l64k", 8),
                                                  ("qwen3_8b_l128k", 8)])
def test_full_size_sampled(name, n_blocks_sample):
    w = WORKLOADS[name]
    say(f"[full-size] {name}: generating inputs")
    q, k, v = make_inputs(w)
    p = problem_of(w)
    run = Run.upload(p, q, k, v)
    G = w.n_q_heads // w.n_kv_heads
    sel = B.select(B.SELECT_FRACTION, w.kap_budget)
    say("  GPU proxy")
    s, h = run.kap_score()
    order, count = run.kap_select(s, h, sel)
    gs, gh = s.cpu().numpy(), h.cpu().numpy()
    go, gc = order.cpu().numpy(), count.cpu().numpy()
    # calibrate Delta on the GPU's own margins (skip off) for the OSK budget
    say("  GPU margins + calibration")
    _, visit0, margin0, _ = run.osk(order, count, None)
    total = w.batch * w.n_q_heads * O.causal_blocks(w.seq_len, w.block)
    listed = int(gc.sum()) * G
    cnt_q = np.repeat(gc, G, axis=1)
    pos = np.arange(w.n_blocks)[None, None, None, :] < cnt_q[..., None]
    delta, n_skip, b_real = delta_for_budget(margin0.cpu().numpy()[pos], listed, total,
                                             w.osk_budget, w.seq_len)
    sk = B.skip(B.SKIP_ROWMAX, delta)
    o, visit, margin, ncomp = run.osk(order, count, sk)
    gv, gm, gn = visit.cpu().numpy(), margin.cpu().numpy(), ncomp.cpu().numpy()
    assert int(gn.sum()) == listed - n_skip
    o_pf = run.prefill(sel, sk)[0]
    assert np.array_equal(host_bits(o_pf), host_bits(o))       # prefill == its three stages
    say(f"  B1 {listed / total:.4f}  B {b_real:.4f}  delta {delta:.2f}")
    # proxy on sampled KV-head units
    kv_units = _sample_units(w, 2, n_blocks_sample, per_q=False)
    say(f"  oracle KAP on {len(kv_units)} units")
    os_, oh = O.kap_score(q, k, n_kv_heads=w.n_kv_heads, block=w.block, stride=w.stride,
                          units=kv_units)
    ffn = lambda n, g, i: PR.fragile_blocks(q, k, n_kv_heads=w.n_kv_heads, block=w.block,
                                            stride=w.stride, sm_scale=0.0, n=n, g=g, i=i)
    PR.check_scores(gs, gh, os_, oh, kv_units, ffn)
    oo, oc = O.kap_select(os_, oh, mode=O.SELECT_FRACTION, value=w.kap_budget, units=kv_units)
    PR.check_orders(go, gc, oo, oc, os_, oh, kv_units, ffn)
    # OSK on sampled query-head units, oracle replaying the GPU's list
    q_units = _sample_units(w, 3, n_blocks_sample, per_q=True)
    say(f"  oracle OSK on {len(q_units)} units")
    ora = O.osk_attention(q, k, v, go, gc, block=w.block, skip_mode=O.SKIP_ROWMAX, delta=delta,
                          units=q_units)
    tau = ora["tau"]
    gout = host_bits(o)
    excused = 0
    for (n, hq, i) in q_units:
        c = int(gc[n, hq // G, i])
        assert np.abs(gm[n, hq, i, :c] - ora["margin"][(n, hq, i)]).max() < 1e-4
        excused += PR.check_visits(gv[n, hq, i], ora["visit"][(n, hq, i)],
                                   ora["margin"][(n, hq, i)], tau, c)
        assert gn[n, hq, i] == ora["n_computed"][(n, hq, i)] or excused
        rows = slice(i * w.block, (i + 1) * w.block)
        PR.check_output(bf16_to_f64(gout[n, hq, rows]), ora["o"][(n, hq, i)])
    say(f"  excused skip decisions {excused}")
    assert excused <= 1
