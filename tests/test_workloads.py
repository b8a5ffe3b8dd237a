"""The seeded input generator: determinism, bf16 rounding, distributions."""

import numpy as np
import torch

import workloads as W


def test_same_seed_same_bits_and_different_seed_differs():
    w = W.custom(W.EXIT_MLP, 33, 64, 100, 128, name="t")
    a, b, c = W.make_batch(w, 3), W.make_batch(w, 3), W.make_batch(w, 4)
    np.testing.assert_array_equal(a.hidden[0], b.hidden[0])
    np.testing.assert_array_equal(a.exits[0].w_down, b.exits[0].w_down)
    np.testing.assert_array_equal(a.targets, b.targets)
    assert not np.array_equal(a.hidden[0], c.hidden[0])


def test_bf16_rounding_matches_torch_cast():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10,
                        np.array([0.0, -0.0, 1e-40, 3.0e38, -1.5, np.inf, -np.inf], np.float32)])
    ours = W.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    back = W.bf16_bits_to_f32(ours)
    np.testing.assert_array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_zipf_targets_shape_and_skew():
    rng = np.random.default_rng(1)
    y = W.zipf_targets(rng, 200000, 32000)
    assert y.min() >= 0 and y.max() < 32000
    counts = np.bincount(y, minlength=32000)
    top = counts.max() / len(y)
    assert 0.12 < top < 0.16            # P(rank 1) = 1 / H_{32000,1.1} ~ 0.14
    # frequent ids are spread across the vocabulary, not packed in one tile
    top_ids = np.argsort(counts)[-64:]
    assert np.ptp(top_ids) > 16000


def test_workload_recipes():
    b = W.make_batch(W.WORKLOADS["tiny_norm_f32"], 0)
    assert b.hidden[0].dtype == np.float32 and b.hidden[0].shape == (512, 256)
    assert np.all(b.exits[0].gamma == 1.0)
    assert abs(np.std(b.exits[0].w_out) - 0.02) < 0.001
    w = W.custom(W.EXIT_NORM, 2048, 64, 50, row_scale=True, name="rs")
    x = W.decode(W.make_batch(w, 0).hidden[0])
    rms = np.sqrt(np.mean(x * x, axis=1))
    assert abs(np.std(np.log(rms)) - 0.5) < 0.05       # lognormal(0, 0.5) rows
