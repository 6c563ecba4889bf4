"""Paged KV cache (Sec. 4.3 "Physical jumping over pages"; appendix D.1: a logical block resolves
through one or more physical pages when the page size differs from the block size).

The paged entry points read K and V through a page table from a [n_pages, Hkv, page, d] cache. On
the same data they must give results bit-identical to the contiguous entry points, which the
oracle parity tests cover; the tiny case is also checked against the oracle directly. Unused pages
hold random values, so a wrong page lookup cannot go unnoticed.
"""
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


SMALL_GQA = Workload("small_gqa", 2, 8, 2, 2048, 128, 128, 16, 0.25, 0.125, 256, (0.005, 0.03))
# Page sizes below, at and above the block size, and one page holding a whole sequence (the block's
# rows then sit deep inside their page).
CASES = {"tiny_l2k": (WORKLOADS["tiny_l2k"], [16, 64, 256, 2048]),
         "small_gqa": (SMALL_GQA, [16, 128, 512, 2048])}


def make_paged(k, v, page, extra, seed):
    """Scatter contiguous K/V [B, Hkv, L, d] into a paged cache through a random page table."""
    Bt, Hkv, L, d = k.shape
    per_seq = L // page
    n_pages = Bt * per_seq + extra
    rng = np.random.default_rng(seed)
    perm = rng.permutation(n_pages).astype(np.int32)
    table = perm[:Bt * per_seq].reshape(Bt, per_seq)
    kc = rng.integers(0, 2 ** 16, size=(n_pages, Hkv, page, d), dtype=np.uint16) & np.uint16(0xBFFF)
    vc = rng.integers(0, 2 ** 16, size=(n_pages, Hkv, page, d), dtype=np.uint16) & np.uint16(0xBFFF)
    for n in range(Bt):
        for lp in range(per_seq):
            kc[table[n, lp]] = k[n, :, lp * page:(lp + 1) * page, :]
            vc[table[n, lp]] = v[n, :, lp * page:(lp + 1) * page, :]
    return kc, vc, table, n_pages


@pytest.fixture(scope="module", params=list(CASES))
def case(request):
    w, pages = CASES[request.param]
    say(f"[paged case] {w.name}: B={w.batch} Hq={w.n_q_heads} Hkv={w.n_kv_heads} L={w.seq_len} "
        f"b={w.block}, pages {pages}")
    q, k, v = make_inputs(w)
    p = B.Problem(w.batch, w.n_q_heads, w.n_kv_heads, w.seq_len, w.head_dim, w.block, w.stride)
    return dict(w=w, p=p, q=q, k=k, v=v, run=Run.upload(p, q, k, v), pages=pages)


def paged_run(c, page, extra=3, seed=1):
    kc, vc, table, n_pages = make_paged(c["k"], c["v"], page, extra, seed)
    kc_d, vc_d, t_d = dev(kc), dev(vc), dev(table)
    kv = B.paged_kv(kc_d, vc_d, t_d, page, n_pages)
    return kv, (kc_d, vc_d, t_d), table, n_pages


def test_paged_kap_score_bit_exact(case):
    w, p, run = case["w"], case["p"], case["run"]
    s_ref, h_ref = run.kap_score()
    for page in case["pages"]:
        say(f"[paged kap_score] {w.name} page {page}")
        kv, keep, _, _ = paged_run(case, page)
        s, h = run._zeros(s_ref.shape, torch().float32), run._zeros(h_ref.shape, torch().uint8)
        B.cosa_kap_score_paged(p, run.q, kv, s, h)
        torch().cuda.synchronize()
        assert torch().equal(s, s_ref) and torch().equal(h, h_ref)


def test_paged_osk_bit_exact(case):
    w, p, run = case["w"], case["p"], case["run"]
    s, h = run.kap_score()
    order, count = run.kap_select(s, h, B.select(B.SELECT_FRACTION, w.kap_budget))
    sk = B.skip(B.SKIP_ROWMAX, w.seq_len * float(np.exp(-2.0)))
    o_ref, vis_ref, mar_ref, nc_ref = run.osk(order, count, sk)
    for page in case["pages"]:
        say(f"[paged osk] {w.name} page {page}")
        kv, keep, _, _ = paged_run(case, page)
        o = run._zeros(o_ref.shape, torch().int16)
        vis, mar, nc = (run._zeros(x.shape, x.dtype) for x in (vis_ref, mar_ref, nc_ref))
        B.cosa_osk_attention_paged(p, run.q, kv, order, count, sk, o, vis, mar, nc)
        torch().cuda.synchronize()
        assert torch().equal(o, o_ref)
        assert torch().equal(vis, vis_ref) and torch().equal(mar, mar_ref)
        assert torch().equal(nc, nc_ref)


def test_paged_prefill_bit_exact_and_oracle(case):
    w, p, run = case["w"], case["p"], case["run"]
    sel = B.select(B.SELECT_FRACTION, w.kap_budget)
    sk = B.skip(B.SKIP_ROWMAX, w.seq_len * float(np.exp(-2.0)))
    o_ref, _, _, order_ref, count_ref = run.prefill(sel, sk)
    nbytes = B.cosa_prefill_workspace_bytes(p)
    for page in case["pages"]:
        say(f"[paged prefill] {w.name} page {page}")
        kv, keep, _, _ = paged_run(case, page, seed=page)
        ws = run._zeros((nbytes,), torch().uint8)
        o = run._zeros(o_ref.shape, torch().int16)
        B.cosa_prefill_paged(p, run.q, kv, sel, sk, ws, nbytes, o)
        torch().cuda.synchronize()
        assert torch().equal(o, o_ref)
    if w.name == "tiny_l2k":
        # the paged output against the oracle walking the same lists
        ref = O.osk_attention(case["q"], case["k"], case["v"], order_ref.cpu().numpy(),
                              count_ref.cpu().numpy(), block=w.block, skip_mode=O.SKIP_ROWMAX,
                              delta=w.seq_len * float(np.exp(-2.0)))["o"]
        mx, mean = PR.check_output(bf16_to_f64(host_bits(o)), ref)
        say(f"  paged O vs oracle: max-abs {mx:.2e} mean-abs {mean:.2e}")


def test_paged_out_of_range_entries_read_page_zero(case):
    """Table entries outside [0, n_pages) are read as physical page 0 (never outside the cache)."""
    w, p, run = case["w"], case["p"], case["run"]
    page = case["pages"][0]
    kc, vc, table, n_pages = make_paged(case["k"], case["v"], page, 3, 7)
    bad = table.copy()
    bad[0, 1] = n_pages + 5
    bad[-1, -1] = -3
    as_zero = bad.copy()
    as_zero[0, 1] = 0
    as_zero[-1, -1] = 0
    sel = B.select(B.SELECT_FRACTION, w.kap_budget)
    nbytes = B.cosa_prefill_workspace_bytes(p)
    outs = []
    for t in (bad, as_zero):
        say(f"[paged out of range] {w.name} page {page}")
        kc_d, vc_d, t_d = dev(kc), dev(vc), dev(t)
        kv = B.paged_kv(kc_d, vc_d, t_d, page, n_pages)
        ws = run._zeros((nbytes,), torch().uint8)
        o = run._zeros((w.batch, w.n_q_heads, w.seq_len, w.head_dim), torch().int16)
        B.cosa_prefill_paged(p, run.q, kv, sel, None, ws, nbytes, o)
        torch().cuda.synchronize()
        outs.append((o.cpu(), ws.cpu()))
    assert torch().equal(outs[0][0], outs[1][0]) and torch().equal(outs[0][1], outs[1][1])
