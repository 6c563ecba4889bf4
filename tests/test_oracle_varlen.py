"""Pins of the oracle's packed variable-length composition on the CPU.

A pack is several independent causal sequences laid end to end along the token axis, each on whole
blocks. What fixes the values here is not the composition code itself:
* dense attention over a pack must equal one masked softmax over the whole packed axis with a
  block-diagonal causal mask (key c visible to row t iff both lie in the same sequence and c <= t),
  computed by PyTorch's scaled_dot_product_attention in float64;
* at full budget with skipping off, the packed OSK output must equal that same masked softmax
  (Algorithm A reduces to exact attention, Sec. 3.1);
* a sequence gives the same proxy scores, lists (shifted by its first block), skip decisions and
  outputs whether it is alone or packed behind another sequence (translation), and changing one
  sequence's inputs leaves every other sequence's results unchanged (independence);
* the skip threshold of each sequence uses its own length N = L_q in ln(Delta / N) (Eq. (skip)),
  so a long and a short sequence with the same Delta have different thresholds.
"""
import numpy as np
import pytest
import torch

from oracle import cosa_oracle as O
from paper_2607_25291_amd.inputs import random_inputs

BLOCK, STRIDE, D = 16, 4, 32


def masked_softmax_f64(q_bits, k_bits, v_bits, cu_blocks, scale):
    """Block-diagonal causal attention over the whole packed axis (independent formulation)."""
    q = torch.from_numpy(O.widen(q_bits))
    k = torch.from_numpy(O.widen(k_bits))
    v = torch.from_numpy(O.widen(v_bits))
    G = q.shape[1] // k.shape[1]
    k = k.repeat_interleave(G, dim=1)
    v = v.repeat_interleave(G, dim=1)
    L = q.shape[2]
    seq = np.zeros(L, dtype=np.int64)
    for s in range(len(cu_blocks) - 1):
        seq[cu_blocks[s] * BLOCK:cu_blocks[s + 1] * BLOCK] = s
    t = np.arange(L)
    allowed = (seq[:, None] == seq[None, :]) & (t[None, :] <= t[:, None])
    mask = torch.from_numpy(allowed)
    return torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=mask,
                                                            scale=scale).numpy()


def pack(parts):
    """Concatenate per-sequence (q, k, v) bit arrays along the token axis."""
    return tuple(np.ascontiguousarray(np.concatenate([p[x] for p in parts], axis=2))
                 for x in range(3))


def run(q, k, v, cu, **kw):
    args = dict(n_kv_heads=k.shape[1], block=BLOCK, stride=STRIDE)
    args.update(kw)
    return O.prefill_varlen(q, k, v, cu, **args)


@pytest.mark.parametrize("cu", [[0, 6], [0, 2, 3, 6], [0, 1, 2, 3, 4, 5, 6]])
def test_dense_varlen_is_block_diagonal_causal_softmax(cu):
    q, k, v = random_inputs(2, 4, 2, cu[-1] * BLOCK, D, seed=len(cu))
    scale = O.default_scale(D)
    got = O.dense_attention_varlen(q, k, v, cu, block=BLOCK)
    want = masked_softmax_f64(q, k, v, cu, scale)
    assert np.abs(got - want).max() < 1e-12


def test_full_budget_without_skip_is_exact_packed_attention():
    cu = [0, 3, 4, 8]
    q, k, v = random_inputs(1, 4, 2, cu[-1] * BLOCK, D, seed=11)
    res = run(q, k, v, cu, select_mode=O.SELECT_ALL)
    want = masked_softmax_f64(q, k, v, cu, O.default_scale(D))
    assert np.abs(res["o"] - want).max() < 1e-12
    # every listed block belongs to the query block's own sequence and is causal
    for (F, E, _, _) in O.packed_spans(cu, BLOCK):
        for i in range(F, E):
            lst = res["order"][0, :, i, :res["count"][0, 0, i]]
            assert ((lst >= F) & (lst <= i)).all()
            assert (res["count"][0, :, i] == i - F + 1).all()


def test_single_sequence_pack_is_the_unpacked_problem():
    q, k, v = random_inputs(1, 2, 1, 5 * BLOCK, D, seed=3)
    res = run(q, k, v, [0, 5], select_mode=O.SELECT_FRACTION, select_value=0.5,
              skip_mode=O.SKIP_ROWMAX, delta=20.0)
    sc, hr = O.kap_score(q, k, n_kv_heads=1, block=BLOCK, stride=STRIDE)
    od, ct = O.kap_select(sc, hr, mode=O.SELECT_FRACTION, value=0.5)
    osk = O.osk_attention(q, k, v, od, ct, block=BLOCK, skip_mode=O.SKIP_ROWMAX, delta=20.0)
    tri = np.tril(np.ones((5, 5), bool))
    assert np.array_equal(res["score"][0, 0][tri], sc[0, 0][tri])
    assert np.array_equal(res["order"], od) and np.array_equal(res["count"], ct)
    assert np.array_equal(res["o"], osk["o"])
    assert np.array_equal(res["visit"], osk["visit"])
    assert res["tau"] == [osk["tau"]]


def test_translation_and_independence():
    """Sequence A (7 blocks) alone, behind a 3-block sequence X, and behind a different X'."""
    a = random_inputs(1, 4, 2, 7 * BLOCK, D, seed=21)
    x = random_inputs(1, 4, 2, 3 * BLOCK, D, seed=22)
    x2 = random_inputs(1, 4, 2, 3 * BLOCK, D, seed=23)
    kw = dict(select_mode=O.SELECT_FRACTION, select_value=0.6, skip_mode=O.SKIP_ROWMAX, delta=40.0)
    alone = run(*a, [0, 7], **kw)
    packed = run(*pack([x, a]), [0, 3, 10], **kw)
    packed2 = run(*pack([x2, a]), [0, 3, 10], **kw)
    F = 3
    for res in (packed, packed2):
        assert np.array_equal(res["o"][:, :, F * BLOCK:], alone["o"])
        assert np.array_equal(res["count"][:, :, F:], alone["count"])
        shifted = np.where(alone["order"] >= 0, alone["order"] + F, -1)
        assert np.array_equal(res["order"][:, :, F:, :7], shifted)
        assert (res["order"][:, :, F:, 7:] == -1).all()
        assert np.array_equal(res["visit"][:, :, F:, :7], alone["visit"])
        for i in range(7):
            assert np.array_equal(res["score"][:, :, F + i, F:F + i + 1],
                                  alone["score"][:, :, i, :i + 1])
    # the first sequence's results do depend on its own inputs
    assert not np.array_equal(packed["o"][:, :, :F * BLOCK], packed2["o"][:, :, :F * BLOCK])


def test_threshold_uses_each_sequence_length():
    cu = [0, 2, 10]
    q, k, v = random_inputs(1, 2, 1, cu[-1] * BLOCK, D, seed=31)
    delta = 24.0
    res = run(q, k, v, cu, select_mode=O.SELECT_ALL, skip_mode=O.SKIP_ROWMAX, delta=delta)
    lens = [2 * BLOCK, 8 * BLOCK]
    assert res["tau"] == [O.tau_from_delta(delta, n) for n in lens]
    assert res["tau"][0] > res["tau"][1]
    # every skip decision follows its own sequence's threshold
    for s, (F, E, _, _) in enumerate(O.packed_spans(cu, BLOCK)):
        for i in range(F, E):
            c = int(res["count"][0, 0, i])
            m = res["margin"][0, :, i, :c]
            want = np.where(m < res["tau"][s], O.VISIT_SKIPPED, O.VISIT_COMPUTED)
            assert np.array_equal(res["visit"][0, :, i, :c], want)
