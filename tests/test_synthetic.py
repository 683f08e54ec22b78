"""Checks of the seeded input generators (no GPU)."""
import numpy as np
import torch

import synthetic as sy


def test_bf16_cast_is_round_to_nearest_even():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 30,
                        np.array([1.00390625, 1.01171875, -2.5e-39, 0.0, -0.0], np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(sy.to_bf16_bits(x), ref)


def test_generators_are_deterministic_and_shaped():
    w = sy.workload(1)
    a, b = sy.round_inputs(w), sy.round_inputs(w)
    for key in a:
        np.testing.assert_array_equal(a[key], b[key])
    assert a["drafter_logits"].shape == (w.batch * w.depth, w.vocab)
    assert a["rho"].shape == (w.batch, w.depth, w.k, w.k, w.k)
    assert (a["rho"] <= 0).all() and np.isfinite(a["rho"]).all()
    att = sy.attention_inputs(w)
    assert att["q"].shape == (w.batch, w.n_max, w.hq, w.head_dim)
    assert att["k_cache"].shape == (int(att["ctx_offsets"][-1]), w.hkv, w.head_dim)


def test_planted_peaks_top_each_row():
    w = sy.workload(4, batch=1, vocab=4096)
    F = sy.field(w)
    for r in range(w.depth + 1):
        v = np.sort(F[0, r])[::-1]
        # 1..3 planted tokens stand 4..10 above the Gaussian maximum v[m]
        assert any(v[m - 1] - v[m] >= 4 - 1e-4 and v[0] - v[m] <= 10 + 1e-4 for m in (1, 2, 3))
    w2 = sy.workload(2, vocab=4096)
    F2 = sy.field(w2)
    for r in range(w2.depth + 1):
        v = np.sort(F2[0, r])[::-1]
        assert abs((v[0] - v[1]) - 8) < 1e-4


def test_ragged_context_lengths():
    w = sy.workload(3)
    ctx = sy.ctx_lengths(w)
    assert ctx.shape == (16,) and ctx.min() >= 1024 and ctx.max() <= 8192
    assert len(set(ctx.tolist())) > 1
