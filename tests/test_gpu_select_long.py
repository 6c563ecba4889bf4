"""Stage-1 selection on long rows: nb = 1024 candidate blocks per row (the 128K benchmark at
b = 128) and nb = 4096 (a 512K-token sequence), the row lengths where the kernel's LDS exceeds the
default dynamic limit, the kept set outgrows one wavefront's sort and the top-p running mass covers
hundreds of entries. The fraction cut runs on one wavefront per row up to 2048 candidates and on a
workgroup per row beyond, so both kernels are covered; a second test puts the cut inside runs of
tied scores on rows of 1 to 2048 candidates.

The scores and flags are seeded random inputs fed to both sides: the HIP selection must match the
oracle's rule (Sec. 4.2 "Flag-grouped sorting", Eq. (mkap); Algorithm A, proxy stage, top-p) bit for
bit on sampled rows, for the fraction cut at two budgets (kept sets of up to 82 and up to 410
blocks), top-p at p = 0.5 and 0.95 (the paper's operating point) in both visit orders, the
ascending visit order, and keep-all.
"""
import sys

import numpy as np
import pytest

from oracle import cosa_oracle as O
from paper_2607_25291_amd import binding as B
from tests.gpu_util import torch

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", params=[1024, 4096])
def rows(request):
    nb = request.param
    rng = np.random.default_rng(20261202 + nb)
    score = rng.gamma(2.0, 1.0, size=(1, 1, nb, nb)).astype(np.float32)
    hrm = (rng.random((1, 1, nb, nb)) < 0.002).astype(np.uint8)
    fixed = [0, 1, 2, 127, 128, 129, 255, 256, 257, 511, 512, nb // 2 - 1, nb // 2, nb - 2, nb - 1]
    if nb > 1024:
        fixed += [1023, 1024, 2047, 2048, 3071]
    sample = sorted(set(fixed + [int(x) for x in rng.integers(0, nb, 16)]))
    return nb, score, hrm, sample


@pytest.mark.parametrize("mode,value,order_mode", [
    (B.SELECT_FRACTION, 0.02, B.ORDER_KAP), (B.SELECT_FRACTION, 0.10, B.ORDER_KAP),
    (B.SELECT_FRACTION, 0.10, B.ORDER_ASCENDING), (B.SELECT_ALL, 1.0, B.ORDER_KAP),
    (B.SELECT_TOP_P, 0.5, B.ORDER_KAP), (B.SELECT_TOP_P, 0.95, B.ORDER_KAP),
    (B.SELECT_TOP_P, 0.95, B.ORDER_ASCENDING)])
def test_select_long_rows(rows, mode, value, order_mode):
    NB, score, hrm, sample = rows
    say(f"[select long rows] nb={NB} mode={mode} value={value} order={order_mode}")
    t = torch()
    p = B.Problem(1, 1, 1, NB * 128, 128, 128, 16)
    sd = t.from_numpy(score).cuda()
    hd = t.from_numpy(hrm).cuda()
    order = t.full((1, 1, NB, NB), -7, dtype=t.int32, device="cuda")
    count = t.full((1, 1, NB), -7, dtype=t.int32, device="cuda")
    B.cosa_kap_select_ordered(p, sd, hd, B.select(mode, value, order_mode), order, count)
    t.cuda.synchronize()
    units = [(0, 0, i) for i in sample]
    oo, oc = O.kap_select(score.astype(np.float64), hrm, mode=mode, value=value,
                          order_mode=order_mode, units=units)
    go, gc = order.cpu().numpy(), count.cpu().numpy()
    for (n, g, i) in units:
        assert gc[n, g, i] == oc[n, g, i], i
        assert np.array_equal(go[n, g, i], oo[n, g, i]), i
    kept = [int(gc[0, 0, i]) for i in sample]
    say(f"  {len(units)} rows identical; largest kept set {max(kept)}, "
        f"kept {sum(kept)} of {sum(i + 1 for i in sample)} candidates on the sampled rows")


@pytest.mark.parametrize("nb", [1, 40, 64, 65, 300, 2048])
@pytest.mark.parametrize("value", [0.02, 0.10, 0.50, 1.0])
@pytest.mark.parametrize("order_mode", [B.ORDER_KAP, B.ORDER_ASCENDING])
def test_fraction_cut_ties_and_row_lengths(nb, value, order_mode):
    """The fraction cut on rows whose length straddles whole wavefronts (1, 40, 64, 65, 300 and
    2048 candidates) with heavy score ties: scores drawn from {0, a denormal, 0.5, 1, 2} plus a
    continuous share, so the cut falls inside runs of equal scores and the block-index tie-break
    decides. Every row (sampled rows at nb = 2048) must equal the oracle's ordering."""
    say(f"[fraction cut ties] nb={nb} value={value} order={order_mode}")
    rng = np.random.default_rng(7 * nb + int(value * 100) + 1000 * order_mode)
    levels = np.array([0.0, 1e-40, 0.5, 1.0, 2.0], np.float32)
    score = levels[rng.integers(0, len(levels), size=(1, 1, nb, nb))]
    cont = rng.random((1, 1, nb, nb)) < 0.3
    score = np.where(cont, rng.gamma(2.0, 1.0, size=score.shape).astype(np.float32), score)
    hrm = (rng.random((1, 1, nb, nb)) < 0.01).astype(np.uint8)
    t = torch()
    p = B.Problem(1, 1, 1, nb * 128, 128, 128, 16)
    sd = t.from_numpy(score).cuda()
    hd = t.from_numpy(hrm).cuda()
    order = t.full((1, 1, nb, nb), -7, dtype=t.int32, device="cuda")
    count = t.full((1, 1, nb), -7, dtype=t.int32, device="cuda")
    B.cosa_kap_select_ordered(p, sd, hd, B.select(B.SELECT_FRACTION, value, order_mode), order,
                              count)
    t.cuda.synchronize()
    if nb <= 300:
        sample = list(range(nb))
    else:
        sample = sorted(set([0, 1, 63, 64, 65, 1023, 1024, nb - 2, nb - 1] +
                            [int(x) for x in rng.integers(0, nb, 24)]))
    units = [(0, 0, i) for i in sample]
    oo, oc = O.kap_select(score.astype(np.float64), hrm, mode=B.SELECT_FRACTION, value=value,
                          order_mode=order_mode, units=units)
    go, gc = order.cpu().numpy(), count.cpu().numpy()
    for (n, g, i) in units:
        assert gc[n, g, i] == oc[n, g, i], i
        assert np.array_equal(go[n, g, i], oo[n, g, i]), i
    say(f"  {len(units)} rows identical")
