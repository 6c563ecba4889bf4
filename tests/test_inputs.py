"""The seeded input generator: determinism, bf16 rounding, and the injected structure."""
import numpy as np
import torch

from paper_2607_25291_amd.inputs import (WORKLOADS, bf16_bits_to_f32, f32_to_bf16_bits, make_group,
                                         make_inputs, random_inputs, sweep_workloads)


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))).astype(np.float32)
    x[:4] = [0.0, -0.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8]        # ties to even both ways
    ours = f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    assert np.array_equal(bf16_bits_to_f32(ours), torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_determinism_and_shapes():
    w = WORKLOADS["tiny_l2k"]
    a = make_inputs(w)
    b = make_inputs(w)
    for x, y in zip(a, b):
        assert x.dtype == np.uint16 and np.array_equal(x, y)
    assert a[0].shape == (1, 1, 2048, 128) and a[1].shape == (1, 1, 2048, 128)
    c = make_inputs(w, seed=1)
    assert not np.array_equal(a[1], c[1])
    q, k, v = random_inputs(2, 4, 2, 64, 16, seed=3)
    assert q.shape == (2, 4, 64, 16) and k.shape == (2, 2, 64, 16) and v.shape == k.shape


def test_structure():
    w = WORKLOADS["tiny_l2k"]
    q, k, v = make_group(w, 0, 0)
    kn = np.linalg.norm(k, axis=1)
    assert kn[:4].mean() > 5 * np.median(kn[4:])                   # sinks
    # local window: neighbouring queries are correlated, distant ones are not
    qh = q[0]
    near = np.mean(np.sum(qh[1:] * qh[:-1], axis=1)) / 128
    far = np.mean(np.sum(qh[1000:] * qh[:-1000], axis=1)) / 128
    assert near > 0.4 and abs(far) < 0.1
    gq = make_group(WORKLOADS["qwen3_8b_l32k"], 0, 3)[0]
    assert gq.shape == (4, 32768, 128)
    assert len(sweep_workloads()) == 12
