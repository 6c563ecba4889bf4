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
    (B.SELECT_TOP_P, 0.95, B.ORDER_KAP), (B.SELECT_TOP_P, 0.5, B.ORDER_KAP),
    (B.SELECT_TOP_P, 0.95, B.ORDER_ASCENDING), (B.SELECT_ALL, 1.0, B.ORDER_KAP)])
def test_kap_select(case, mode, value, order_mode):
    w, run = case["w"], case["run"]
    value = w.kap_budget if value is None else value
    say(f"[kap_select] {w.name} mode={mode} value={value} order={order_mode}")
    s, h = run.kap_score()
    order, count = run.kap_select(s, h, B.select(mode, value, order_mode))
    go, gc = order.cpu().numpy(), count.cpu().numpy()
    # (a) same scores in, the selection must be bit-exact with the oracle's rule (top-p included:
    # both sides sum in float64 in the same order)
    gs64 = s.cpu().numpy().astype(np.float64)
    oo, oc = O.kap_select(gs64, h.cpu().numpy(), mode=mode, value=value, order_mode=order_mode)
    assert np.array_equal(gc, oc) and np.array_equal(go, oo)
    # (b) end to end against the oracle's own scores (near-ties excused)
    oo2, oc2 = O.kap_select(case["ora_s"], case["ora_h"], mode=mode, value=value,
                            order_mode=order_mode)
    top_p = value if mode == B.SELECT_TOP_P else None
    same, exc = PR.check_orders(go, gc, oo2, oc2, case["ora_s"], case["ora_h"], all_units(w),
                                fragile_fn(case), top_p=top_p)
    say(f"  rows identical {same}, excused {exc}, kept {int(gc.sum())} of "
        f"{w.batch * w.n_kv_heads * O.causal_blocks(w.seq_len, w.block)}")
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
def _sample_units(w, n_blocks_sample):
    """Query-head units (first head, last head, a second-group head of the middle KV group) on
    query blocks spread over [0, nb), and the KV-head units of every group those heads walk."""
    nb = w.n_blocks
    G = w.n_q_heads // w.n_kv_heads
    blocks = sorted(set(np.linspace(0, nb - 1, n_blocks_sample).round().astype(int).tolist()))
    q_heads = sorted({0, w.n_q_heads - 1, G * (w.n_kv_heads // 2) + 1})
    kv_heads = sorted({h // G for h in q_heads})
    return ([(0, g, i) for g in kv_heads for i in blocks],
            [(0, h, i) for h in q_heads for i in blocks])


def _check_sampled_osk(w, q, k, v, go, gc, gv, gm, gn, gout, delta, q_units):
    """OSK margins, skip decisions, computed counts and output on sampled query-head units, the
    oracle replaying the GPU's list. Returns the number of excused decisions."""
    G = w.n_q_heads // w.n_kv_heads
    ora = O.osk_attention(q, k, v, go, gc, block=w.block, skip_mode=O.SKIP_ROWMAX, delta=delta,
                          units=q_units)
    tau = ora["tau"]
    excused = 0
    for (n, hq, i) in q_units:
        c = int(gc[n, hq // G, i])
        assert np.abs(gm[n, hq, i, :c] - ora["margin"][(n, hq, i)]).max() < 1e-4
        exc_u = PR.check_visits(gv[n, hq, i], ora["visit"][(n, hq, i)],
                                ora["margin"][(n, hq, i)], tau, c)
        assert abs(int(gn[n, hq, i]) - int(ora["n_computed"][(n, hq, i)])) <= exc_u, (n, hq, i)
        excused += exc_u
        rows = slice(i * w.block, (i + 1) * w.block)
        PR.check_output(bf16_to_f64(gout[n, hq, rows]), ora["o"][(n, hq, i)])
    return excused


# The largest sequence the proxy supports at 32 proxy rows per query block: nb = 1239 blocks of 128,
# whose block maxima (32 x 1240 floats) and the kernel's static LDS fill the 160 KiB exactly (the
# paired kernel does not fit there; the one-query-block proxy kernel runs). One KV group of the
# Qwen3-8B shape keeps it quick.
MAX_L = Workload("max_l158k", 1, 4, 1, 1239 * 128, 128, 128, 16, 0.10, 0.05, 1024, (0.005, 0.03))
FULL_SIZE = dict(WORKLOADS, max_l158k=MAX_L)


@pytest.mark.parametrize("name,n_blocks_sample", [("qwen3_8b_l32k", 12), ("wide_gqa_l64k", 8),
                                                  ("qwen3_8b_l128k", 8), ("max_l158k", 6)])
def test_full_size_sampled(name, n_blocks_sample):
    w = FULL_SIZE[name]
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
    # the kernel computes exactly the visits whose fp32 margin reaches the fp32 threshold
    tau32 = np.float32(tau_of(delta, w.seq_len))
    assert int(gn.sum()) == int(np.count_nonzero(margin0.cpu().numpy()[pos] >= tau32))
    assert abs(int(gn.sum()) - (listed - n_skip)) <= 2   # calibration lands on the target
    o_pf = run.prefill(sel, sk)[0]
    assert np.array_equal(host_bits(o_pf), host_bits(o))       # prefill == its three stages
    say(f"  B1 {listed / total:.4f}  B {b_real:.4f}  delta {delta:.2f}")
    # the selection, fed the GPU's own scores: every row bit-exact with the oracle's rule
    oo_g, oc_g = O.kap_select(gs.astype(np.float64), gh, mode=O.SELECT_FRACTION,
                              value=w.kap_budget)
    assert np.array_equal(gc, oc_g) and np.array_equal(go, oo_g)
    say(f"  selection on the GPU's scores: all {gc.size} rows bit-exact")
    kv_units, q_units = _sample_units(w, n_blocks_sample)
    # proxy on sampled KV-head units (every group the sampled query heads walk)
    say(f"  oracle KAP on {len(kv_units)} units")
    os_, oh = O.kap_score(q, k, n_kv_heads=w.n_kv_heads, block=w.block, stride=w.stride,
                          units=kv_units)
    ffn = lambda n, g, i: PR.fragile_blocks(q, k, n_kv_heads=w.n_kv_heads, block=w.block,
                                            stride=w.stride, sm_scale=0.0, n=n, g=g, i=i)
    worst, exc_h = PR.check_scores(gs, gh, os_, oh, kv_units, ffn)
    oo, oc = O.kap_select(os_, oh, mode=O.SELECT_FRACTION, value=w.kap_budget, units=kv_units)
    same, exc_o = PR.check_orders(go, gc, oo, oc, os_, oh, kv_units, ffn)
    say(f"  max rel score err {worst:.2e}, excused hrm flags {exc_h}; rows identical {same}, "
        f"excused {exc_o}")
    # OSK on sampled query-head units, oracle replaying the GPU's list
    say(f"  oracle OSK on {len(q_units)} units")
    excused = _check_sampled_osk(w, q, k, v, go, gc, gv, gm, gn, host_bits(o), delta, q_units)
    say(f"  excused skip decisions {excused}")
    assert excused <= 1
    # the dense kernel (the speedup's denominator) on the same units
    say("  GPU dense + oracle dense")
    dense = host_bits(run.dense())
    ora_d = O.dense_attention(q, k, v, block=w.block, units=q_units)
    worst_d = 0.0
    for (n, hq, i) in q_units:
        rows = slice(i * w.block, (i + 1) * w.block)
        mx, _ = PR.check_output(bf16_to_f64(dense[n, hq, rows]), ora_d[(n, hq, i)])
        worst_d = max(worst_d, mx)
    say(f"  dense max-abs {worst_d:.2e} on {len(q_units)} units")


@pytest.mark.parametrize("name,n_blocks_sample", [("qwen3_8b_l32k", 8), ("qwen3_8b_l128k", 6)])
def test_full_size_top_p(name, n_blocks_sample):
    """The paper's own stage-1 mode (top-p, p = 0.95) through cosa_prefill at full size: sampled
    scores, lists (counts within the near-tie band of the cut) and OSK output, with Delta
    calibrated to half the realized stage-1 budget."""
    w = WORKLOADS[name]
    say(f"[full-size top-p] {name}: generating inputs")
    q, k, v = make_inputs(w)
    p = problem_of(w)
    run = Run.upload(p, q, k, v)
    G = w.n_q_heads // w.n_kv_heads
    P_MASS = 0.95
    sel = B.select(B.SELECT_TOP_P, P_MASS)
    say("  GPU prefill (skip off) and margins")
    _, s, h, order, count = run.prefill(sel, None)
    gs, gh = s.cpu().numpy(), h.cpu().numpy()
    go, gc = order.cpu().numpy(), count.cpu().numpy()
    total = w.batch * w.n_q_heads * O.causal_blocks(w.seq_len, w.block)
    listed = int(gc.sum()) * G
    b1 = listed / total
    _, _, margin0, _ = run.osk(order, count, None)
    cnt_q = np.repeat(gc, G, axis=1)
    pos = np.arange(w.n_blocks)[None, None, None, :] < cnt_q[..., None]
    delta, n_skip, b_real = delta_for_budget(margin0.cpu().numpy()[pos], listed, total, b1 / 2,
                                             w.seq_len)
    sk = B.skip(B.SKIP_ROWMAX, delta)
    o_pf, _, _, order2, count2 = run.prefill(sel, sk)
    assert np.array_equal(order2.cpu().numpy(), go) and np.array_equal(count2.cpu().numpy(), gc)
    o, visit, margin, ncomp = run.osk(order, count, sk)
    assert np.array_equal(host_bits(o_pf), host_bits(o))
    gv, gm, gn = visit.cpu().numpy(), margin.cpu().numpy(), ncomp.cpu().numpy()
    tau32 = np.float32(tau_of(delta, w.seq_len))
    assert int(gn.sum()) == int(np.count_nonzero(margin0.cpu().numpy()[pos] >= tau32))
    assert abs(int(gn.sum()) - (listed - n_skip)) <= 2
    say(f"  realized B1 {b1:.4f}  B {b_real:.4f}  delta {delta:.2f}")
    kv_units, q_units = _sample_units(w, n_blocks_sample)
    say(f"  oracle KAP on {len(kv_units)} units")
    os_, oh = O.kap_score(q, k, n_kv_heads=w.n_kv_heads, block=w.block, stride=w.stride,
                          units=kv_units)
    ffn = lambda n, g, i: PR.fragile_blocks(q, k, n_kv_heads=w.n_kv_heads, block=w.block,
                                            stride=w.stride, sm_scale=0.0, n=n, g=g, i=i)
    worst, exc_h = PR.check_scores(gs, gh, os_, oh, kv_units, ffn)
    # same scores in: bit-exact with the oracle's rule
    oo_g, oc_g = O.kap_select(gs.astype(np.float64), gh, mode=O.SELECT_TOP_P, value=P_MASS,
                              units=kv_units)
    for (n, g, i) in kv_units:
        assert gc[n, g, i] == oc_g[n, g, i] and np.array_equal(go[n, g, i], oo_g[n, g, i]), i
    # end to end against the oracle's own scores
    oo, oc = O.kap_select(os_, oh, mode=O.SELECT_TOP_P, value=P_MASS, units=kv_units)
    same, exc_o = PR.check_orders(go, gc, oo, oc, os_, oh, kv_units, ffn, top_p=P_MASS)
    say(f"  max rel score err {worst:.2e}, excused hrm flags {exc_h}; rows identical {same}, "
        f"excused {exc_o}; sampled kept {[int(gc[n, g, i]) for (n, g, i) in kv_units]}")
    say(f"  oracle OSK on {len(q_units)} units")
    excused = _check_sampled_osk(w, q, k, v, go, gc, gv, gm, gn, host_bits(o), delta, q_units)
    say(f"  excused skip decisions {excused}")
    assert excused <= 1
