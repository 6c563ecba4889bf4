"""Host-side checks of the C ABI that need no GPU: the library loads, exports every function the
header declares, and rejects invalid arguments before touching the device."""
import ctypes
import math
import os
import subprocess

import numpy as np
import pytest

from paper_2607_25291_amd import binding as B
from paper_2607_25291_amd.calibrate import delta_for_budget, delta_for_budget_packed

EXPECTED = {"cosa_status_string", "cosa_last_error", "cosa_kap_score", "cosa_kap_select_ordered",
            "cosa_osk_attention", "cosa_dense_attention", "cosa_prefill_workspace_bytes",
            "cosa_prefill_workspace_layout", "cosa_prefill", "cosa_kap_score_paged",
            "cosa_osk_attention_paged", "cosa_prefill_paged", "cosa_masked_attention",
            "cosa_block_mass", "cosa_kap_score_varlen", "cosa_kap_select_ordered_varlen",
            "cosa_osk_attention_varlen", "cosa_dense_attention_varlen", "cosa_prefill_varlen",
            "cosa_prefill_paged_varlen", "cosa_kap_score_workspace_bytes",
            "cosa_kap_score_staged", "cosa_osk_attention_queue_bytes", "cosa_osk_attention_queued",
            "cosa_prefill_noalloc"}


def test_header_declares_the_abi():
    assert set(B.declared_symbols()) == EXPECTED


def test_library_exports_every_declared_symbol():
    L = B.lib()
    for name in B.declared_symbols():
        assert hasattr(L, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    assert EXPECTED <= exported


def test_status_strings():
    names = ["COSA_OK", "COSA_ERR_INVALID_ARG", "COSA_ERR_UNSUPPORTED", "COSA_ERR_WORKSPACE",
             "COSA_ERR_HIP"]
    for i, n in enumerate(names):
        assert B.cosa_status_string(i) == n
    assert B.cosa_status_string(99) == "COSA_ERR_UNKNOWN"


GOOD = B.Problem(1, 8, 2, 1024, 128, 128, 16)


@pytest.mark.parametrize("change,status", [
    (dict(n_q_heads=6, n_kv_heads=4), B.COSA_ERR_INVALID_ARG),
    (dict(n_kv_heads=0), B.COSA_ERR_INVALID_ARG),
    (dict(batch=-1), B.COSA_ERR_INVALID_ARG),
    (dict(stride=24), B.COSA_ERR_INVALID_ARG),
    (dict(sm_scale=-1.0), B.COSA_ERR_INVALID_ARG),
    (dict(sm_scale=float("nan")), B.COSA_ERR_INVALID_ARG),
    (dict(causal=2), B.COSA_ERR_INVALID_ARG),
    (dict(causal=0), B.COSA_ERR_UNSUPPORTED),
    (dict(head_dim=64), B.COSA_ERR_UNSUPPORTED),
    (dict(block=32, stride=4), B.COSA_ERR_UNSUPPORTED),
    (dict(seq_len=1000), B.COSA_ERR_UNSUPPORTED),
    (dict(seq_len=128 * 8193), B.COSA_ERR_UNSUPPORTED),
])
def test_problem_validation(change, status):
    p = B.Problem(**{**GOOD.__dict__, **change})
    with pytest.raises(B.CosaError) as e:
        B.cosa_dense_attention(p, 16, 16, 16, 16, stream=0)
    assert e.value.status == status
    assert B.cosa_status_string(status) in str(e.value)


def test_proxy_limits():
    # 2 samples per block, too many proxy rows per unit (G * spb > 128), and block maxima that do
    # not fit the LDS: 32 proxy rows x (nb + 1) floats plus 5 KiB of static LDS fit 160 KiB up to
    # nb = 1239 (the largest size, run on the GPU), not at nb = 1240
    for p in [B.Problem(1, 8, 2, 1024, 128, 128, 64), B.Problem(1, 64, 2, 1024, 128, 128, 16),
              B.Problem(1, 4, 1, 1240 * 128, 128, 128, 16)]:
        with pytest.raises(B.CosaError) as e:
            B.cosa_kap_score(p, 16, 16, 16, 16, stream=0)
        assert e.value.status == B.COSA_ERR_UNSUPPORTED
        # attention alone does not depend on the proxy limits: it fails only on the NULL pointers
        with pytest.raises(B.CosaError) as e:
            B.cosa_dense_attention(p, 16, 16, None, 16, stream=0)
        assert e.value.status == B.COSA_ERR_INVALID_ARG


def test_argument_validation():
    with pytest.raises(B.CosaError) as e:
        B.cosa_kap_score(GOOD, 16, None, 16, 16, stream=0)
    assert e.value.status == B.COSA_ERR_INVALID_ARG
    for sel in [B.select(B.SELECT_FRACTION, 0.0), B.select(B.SELECT_TOP_P, 1.5),
                B.select(7, 0.5), B.select(B.SELECT_FRACTION, 0.5, order=5)]:
        with pytest.raises(B.CosaError) as e:
            B.cosa_kap_select_ordered(GOOD, 16, 16, sel, 16, 16, stream=0)
        assert e.value.status == B.COSA_ERR_INVALID_ARG
    for sk in [B.skip(B.SKIP_ROWMAX, 0.0), B.skip(B.SKIP_ROWMAX, 2000.0),
               B.skip(B.SKIP_ROWMAX, float("inf")), B.skip(3, 1.0)]:
        with pytest.raises(B.CosaError) as e:
            B.cosa_osk_attention(GOOD, 16, 16, 16, 16, 16, sk, 16, stream=0)
        assert e.value.status == B.COSA_ERR_INVALID_ARG
    ws = B.cosa_prefill_workspace_bytes(GOOD)
    with pytest.raises(B.CosaError) as e:
        B.cosa_prefill(GOOD, 16, 16, 16, B.select(B.SELECT_FRACTION, 0.5), None, 16, ws - 1, 16,
                       stream=0)
    assert e.value.status == B.COSA_ERR_WORKSPACE
    with pytest.raises(B.CosaError) as e:
        B.cosa_prefill(GOOD, 16, 16, 16, B.select(B.SELECT_FRACTION, 0.5), None, None, ws, 16,
                       stream=0)
    assert e.value.status == B.COSA_ERR_WORKSPACE


def test_queued_osk_validation():
    """The queued OSK checks what cosa_osk_attention checks, plus its queue buffer."""
    qb = B.cosa_osk_attention_queue_bytes()
    for queue, nbytes, status in [(None, qb, B.COSA_ERR_WORKSPACE), (256, qb - 1, B.COSA_ERR_WORKSPACE),
                                  (258, qb, B.COSA_ERR_INVALID_ARG)]:
        with pytest.raises(B.CosaError) as e:
            B.cosa_osk_attention_queued(GOOD, 16, 16, 16, 16, 16, None, 16, queue, nbytes, stream=0)
        assert e.value.status == status
    with pytest.raises(B.CosaError) as e:
        B.cosa_osk_attention_queued(GOOD, 16, 16, 16, 16, 16, B.skip(B.SKIP_ROWMAX, 0.0), 16, 256,
                                    qb, stream=0)
    assert e.value.status == B.COSA_ERR_INVALID_ARG
    with pytest.raises(B.CosaError) as e:
        B.cosa_osk_attention_queued(GOOD, 16, 16, 16, None, 16, None, 16, 256, qb, stream=0)
    assert e.value.status == B.COSA_ERR_INVALID_ARG
    # an empty problem launches nothing, whatever the pointers
    B.cosa_osk_attention_queued(B.Problem(0, 8, 2, 1024), None, None, None, None, None, None, None,
                                None, 0, stream=0)
    assert B.cosa_last_error() == ""


def test_paged_validation():
    def kv(page=64, n_pages=16, k=16, v=16, table=16):
        return B.CosaPagedKv(k, v, table, page, n_pages)
    sel = B.select(B.SELECT_FRACTION, 0.5)
    ws = B.cosa_prefill_workspace_bytes(GOOD)
    for bad in [kv(page=48), kv(page=8), kv(page=1 << 21), kv(page=2048), kv(n_pages=0),
                kv(n_pages=2 ** 40), kv(table=None), kv(k=None), kv(v=None)]:
        with pytest.raises(B.CosaError) as e:
            B.cosa_osk_attention_paged(GOOD, 16, bad, 16, 16, None, 16, stream=0)
        assert e.value.status == B.COSA_ERR_INVALID_ARG
        with pytest.raises(B.CosaError) as e:
            B.cosa_prefill_paged(GOOD, 16, bad, sel, None, 16, ws, 16, stream=0)
        assert e.value.status == B.COSA_ERR_INVALID_ARG
    for bad in [kv(page=48), kv(table=None), kv(k=None)]:
        with pytest.raises(B.CosaError) as e:
            B.cosa_kap_score_paged(GOOD, 16, bad, 16, 16, stream=0)
        assert e.value.status == B.COSA_ERR_INVALID_ARG
    with pytest.raises(B.CosaError) as e:
        B.cosa_prefill_paged(GOOD, 16, None, sel, None, 16, ws, 16, stream=0)
    assert e.value.status == B.COSA_ERR_INVALID_ARG
    # the proxy alone does not need the V cache (an empty problem validates and launches nothing)
    B.cosa_kap_score_paged(B.Problem(0, 8, 2, 1024), None, kv(v=None), None, None, stream=0)
    B.cosa_prefill_paged(B.Problem(0, 8, 2, 1024), None, kv(), sel, None, None, 0, None, stream=0)
    assert B.cosa_last_error() == ""


def test_staged_score_validation():
    ws = B.cosa_kap_score_workspace_bytes(GOOD)
    assert ws > 0
    with pytest.raises(B.CosaError) as e:
        B.cosa_kap_score_staged(GOOD, 16, 16, 256, ws - 1, 16, 16, stream=0)
    assert e.value.status == B.COSA_ERR_WORKSPACE
    with pytest.raises(B.CosaError) as e:
        B.cosa_kap_score_staged(GOOD, 16, 16, None, ws, 16, 16, stream=0)
    assert e.value.status == B.COSA_ERR_WORKSPACE
    with pytest.raises(B.CosaError) as e:
        B.cosa_kap_score_staged(GOOD, 16, 16, 8, ws, 16, 16, stream=0)
    assert e.value.status == B.COSA_ERR_INVALID_ARG
    sel = B.select(B.SELECT_ALL)
    nbytes = B.cosa_prefill_workspace_bytes(GOOD)
    with pytest.raises(B.CosaError) as e:
        B.cosa_prefill(GOOD, 16, 16, 16, sel, None, 8, nbytes, 16, stream=0)
    assert e.value.status == B.COSA_ERR_INVALID_ARG
    B.cosa_kap_score_staged(B.Problem(0, 8, 2, 1024), None, None, None, 0, None, None, stream=0)
    assert B.cosa_last_error() == ""


def test_varlen_validation():
    """Packing offsets must start at 0, increase strictly and end at nb (= 8 here); at most 128
    sequences; skipping needs delta <= the shortest sequence."""
    sel = B.select(B.SELECT_FRACTION, 0.5)
    ws = B.cosa_prefill_workspace_bytes(GOOD)
    bad_offsets = [[0], [1, 8], [0, 3, 3, 8], [0, 5, 2, 8], [0, 7], [0, 9], list(range(0, 130))]
    for cu in bad_offsets:
        vl = B.varlen(cu)
        calls = [
            lambda: B.cosa_kap_score_varlen(GOOD, vl, 16, 16, 16, 16, stream=0),
            lambda: B.cosa_kap_select_ordered_varlen(GOOD, vl, 16, 16, sel, 16, 16, stream=0),
            lambda: B.cosa_osk_attention_varlen(GOOD, vl, 16, 16, 16, 16, 16, None, 16, stream=0),
            lambda: B.cosa_dense_attention_varlen(GOOD, vl, 16, 16, 16, 16, stream=0),
            lambda: B.cosa_prefill_varlen(GOOD, vl, 16, 16, 16, sel, None, 16, ws, 16, stream=0),
        ]
        for call in calls:
            with pytest.raises(B.CosaError) as e:
                call()
            assert e.value.status == B.COSA_ERR_INVALID_ARG, cu
    for call in [lambda: B.cosa_dense_attention_varlen(GOOD, None, 16, 16, 16, 16, stream=0),
                 lambda: B.cosa_prefill_varlen(GOOD, None, 16, 16, 16, sel, None, 16, ws, 16,
                                               stream=0)]:
        with pytest.raises(B.CosaError) as e:
            call()
        assert e.value.status == B.COSA_ERR_INVALID_ARG
    # Delta is checked against each sequence: blocks of 128 tokens, sequences of 256 and 768 tokens
    vl = B.varlen([0, 2, 8])
    for delta in (257.0, 700.0):
        with pytest.raises(B.CosaError) as e:
            B.cosa_osk_attention_varlen(GOOD, vl, 16, 16, 16, 16, 16,
                                        B.skip(B.SKIP_ROWMAX, delta), 16, stream=0)
        assert e.value.status == B.COSA_ERR_INVALID_ARG
        assert "sequence 0" in B.cosa_last_error()
    # the same delta is accepted without packing (seq_len 1024)
    assert B.MAX_PACKED_SEQS == 128


def test_masked_attention_validation():
    with pytest.raises(B.CosaError) as e:
        B.cosa_masked_attention(GOOD, 16, 16, 16, None, 16, stream=0)
    assert e.value.status == B.COSA_ERR_INVALID_ARG
    B.cosa_masked_attention(B.Problem(0, 8, 2, 1024), None, None, None, None, None, stream=0)
    assert B.cosa_last_error() == ""


def test_empty_problems_launch_nothing():
    for p in [B.Problem(0, 8, 2, 1024), B.Problem(1, 8, 2, 0)]:
        # NULL pointers are fine: nothing is launched
        B.cosa_dense_attention(p, None, None, None, None, stream=0)
        B.cosa_kap_score(p, None, None, None, None, stream=0)
        B.cosa_prefill(p, None, None, None, B.select(B.SELECT_ALL), None, None, 0, None, stream=0)
        assert B.cosa_last_error() == ""


def test_workspace_layout():
    for (Bt, Hkv, L, b) in [(1, 8, 131072, 128), (2, 2, 2048, 64), (1, 1, 128, 128)]:
        p = B.Problem(Bt, Hkv * 4, Hkv, L, 128, b, b // 8)
        lay = B.cosa_prefill_workspace_layout(p)
        nb = L // b
        cells = Bt * Hkv * nb * nb
        al = lambda x: (x + 255) // 256 * 256
        assert lay.score == 0
        assert lay.hrm == al(4 * cells)
        assert lay.order == al(lay.hrm + cells)
        assert lay.count == al(lay.order + 4 * cells)
        assert lay.keys == al(lay.count + 4 * Bt * Hkv * nb)
        # staged sampled keys: every KV head's L / s keys in 32-key chunks of 32 x 128 bf16, then
        # (G * spb = 32 rows per query block) the block maxima of the paired proxy kernel's second
        # query block: [nb][32] floats for each workgroup of its persistent grid (a multiple of 8,
        # at most 256, one item per KV head and pair of query blocks)
        keys = Bt * Hkv * -(-(L // (b // 8)) // 32) * 32 * 128 * 2
        grid = min(256, -(-(Bt * Hkv * -(-nb // 2)) // 8) * 8)
        staged = al(keys) + grid * nb * 32 * 4
        assert B.cosa_kap_score_workspace_bytes(p) == staged
        # the OSK work-queue counters (one per XCD, 128 bytes apart) close the workspace
        assert lay.queue == al(lay.keys + staged)
        assert B.cosa_osk_attention_queue_bytes() == 8 * 128
        assert lay.total == al(lay.queue + 8 * 128)
        assert B.cosa_prefill_workspace_bytes(p) == lay.total
    # 128K, 8 KV heads: 72 MiB of proxy tensors + 16 MiB of staged keys + 32 MiB of paired-proxy
    # block maxima + 1 KiB of queue counters
    assert (B.cosa_prefill_workspace_bytes(B.Problem(1, 32, 8, 131072))
            == 120 * 2 ** 20 + 32 * 2 ** 10 + 1024)


def test_delta_for_budget_host_helper():
    rng = np.random.default_rng(0)
    m = np.concatenate([np.zeros(100), -rng.exponential(2.0, 900)])
    n_causal = 2000
    delta, k, b = delta_for_budget(m, 1000, n_causal, 0.3, 4096)
    tau = math.log(delta / 4096)
    assert k == 400 and (m < tau).sum() == 400 and b == 0.3
    assert np.min(np.abs(m - tau)) > 0
    # unreachable: only the 900 negative margins can be skipped
    delta, k, b = delta_for_budget(m, 1000, n_causal, 0.01, 4096)
    assert k == 900 and (m < math.log(delta / 4096)).sum() == 900
    # nothing to skip
    delta, k, b = delta_for_budget(m, 1000, n_causal, 0.9, 4096)
    assert k == 0 and (m < math.log(delta / 4096)).sum() == 0


def test_delta_for_budget_packed_host_helper():
    """Packed sequences: visit v of sequence q is skipped iff m_v < ln(delta / L_q), evaluated as the
    kernel does (float32 delta and threshold)."""
    rng = np.random.default_rng(1)
    lens = np.array([4096, 1024, 16384])
    per = [600, 200, 1200]
    m = np.concatenate([np.concatenate([np.zeros(n // 10), -rng.exponential(2.0, n - n // 10)])
                        for n in per])
    seq = np.repeat(lens, per)
    n_causal = 6000

    def skipped(delta):
        tau = np.array([np.float32(math.log(float(np.float32(delta)) / L)) for L in seq])
        return int((m.astype(np.float32) < tau).sum())

    for budget in (0.3, 0.25):  # 200 and 500 skips; at most 718 fit under delta <= 1024
        delta, k, b = delta_for_budget_packed(m, seq, n_causal, budget)
        assert delta <= lens.min()
        assert skipped(delta) == k == len(m) - round(budget * n_causal)
        assert b == (len(m) - k) / n_causal
    # a budget below what delta <= min(L_q) allows is capped there
    delta, k, b = delta_for_budget_packed(m, seq, n_causal, 0.01)
    assert abs(delta - lens.min()) < 1e-6 * lens.min() or delta < lens.min()
    assert skipped(delta) == k
    assert k == int(((m + np.log(seq)) < math.log(lens.min())).sum())
    # nothing to skip
    delta, k, b = delta_for_budget_packed(m, seq, n_causal, 0.9)
    assert k == 0 and skipped(delta) == 0
    # one sequence reduces to the unpacked helper
    one = m[:600]
    d1, k1, _ = delta_for_budget_packed(one, np.full(600, 4096), 2000, 0.2)
    d0, k0, _ = delta_for_budget(one, 600, 2000, 0.2, 4096)
    assert k1 == k0 and abs(d1 - d0) < 1e-9 * d0


def test_noalloc_prefill_rejects_before_the_device():
    """cosa_prefill_noalloc validates like cosa_prefill and refuses a problem whose workspace
    exceeds its static scratch array, before any HIP call (so this runs without a GPU)."""
    big = B.Problem(1, 32, 16, 131072, 128, 128, 16)
    assert B.cosa_prefill_workspace_bytes(big) > B.NOALLOC_SCRATCH_BYTES
    with pytest.raises(B.CosaError) as e:
        B.cosa_prefill_noalloc(big, 16, 16, 16, B.select(B.SELECT_FRACTION, 0.1), None, 16,
                               stream=0)
    assert e.value.status == B.COSA_ERR_WORKSPACE and "static scratch" in str(e.value)
    # the 128K benchmark layer (32 / 8 heads) fits
    assert B.cosa_prefill_workspace_bytes(B.Problem(1, 32, 8, 131072)) <= B.NOALLOC_SCRATCH_BYTES
    for sel, sk, status in [(B.select(B.SELECT_FRACTION, 0.0), None, B.COSA_ERR_INVALID_ARG),
                            (B.select(B.SELECT_TOP_P, 1.5), None, B.COSA_ERR_INVALID_ARG),
                            (B.select(), B.skip(B.SKIP_ROWMAX, 1e9), B.COSA_ERR_INVALID_ARG)]:
        with pytest.raises(B.CosaError) as e:
            B.cosa_prefill_noalloc(GOOD, 16, 16, 16, sel, sk, 16, stream=0)
        assert e.value.status == status
    # an empty problem is a no-op
    B.cosa_prefill_noalloc(B.Problem(0, 8, 2, 1024), None, None, None, B.select(), None, None,
                           stream=0)
    with pytest.raises(B.CosaError) as e:
        B.cosa_prefill_noalloc(B.Problem(1, 8, 2, 1024, head_dim=64), 16, 16, 16, B.select(),
                               None, 16, stream=0)
    assert e.value.status == B.COSA_ERR_UNSUPPORTED
