"""The seeded generators: reproducible bits, the documented recipes and sizes."""
import numpy as np
import torch

import workloads as W


def test_bf16_bits_match_torch():
    x = np.random.default_rng(3).standard_normal(10000).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(W.f32_to_bf16_bits(x), ref)


def test_same_seed_same_bits():
    w = W.workload("tiny_mha8_d64_p512_s128_f32")
    a, b = W.single_episode(w), W.single_episode(w)
    for name in ("q", "k", "v", "cq", "ck", "cv"):
        np.testing.assert_array_equal(getattr(a, name), getattr(b, name))


def test_episode_shapes_and_shared_prefix():
    w = W.workload("tiny_mha8_d64_p512_s128_f32")
    ep = W.single_episode(w)
    assert ep.q.shape == (640, 8, 64) and ep.k.shape == (640, 8, 64)
    assert ep.ck.shape == (128, 8, 64)
    ck = ep.contaminated("k")
    np.testing.assert_array_equal(ck[:512], ep.k[:512])
    assert not np.array_equal(ck[512:], ep.k[512:])


def test_llama8b_reading_of_the_crop():
    w = W.workload("llama8b_p8189_s2048_bf16")
    assert w.prefix == 8189 and w.suffix == 2048 and w.t_contaminated == 10240
    assert w.t_sanitized == 10237 and w.prefix % w.block_size == 13


def test_ragged_lengths_recipe():
    _, lens = W.draw_ragged_lengths(2, 16)
    assert len(lens) == 16
    for t, p, s in lens:
        assert 4096 <= t <= 16384 and p + s == t
        assert int(0.10 * t) <= p <= int(0.90 * t) + 1
    _, again = W.draw_ragged_lengths(2, 16)
    assert again == lens
