"""Pins of the oracle's bfloat16 rounding (8 significant bits, ties to even,
fp32's exponent range), used at the storage points of the stacked layers."""
import numpy as np
import torch

import oracle
from workloads import f32_to_bf16_bits, bf16_bits_to_f32


def test_matches_torch_on_fp32_inputs():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(200000) * np.exp(rng.uniform(-30, 30, 200000))).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(oracle.bf16_round(x.astype(np.float64)), ref)


def test_matches_integer_rounding_of_the_generator():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(100000).astype(np.float32)
    np.testing.assert_array_equal(oracle.bf16_round(x.astype(np.float64)),
                                  bf16_bits_to_f32(f32_to_bf16_bits(x)).astype(np.float64))


def test_hand_values():
    cases = [
        (1.0 + 2.0 ** -8, 1.0),                       # tie -> even mantissa 0
        (1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -6),       # tie -> even (mantissa 2)
        (1.0 + 2.0 ** -8 + 2.0 ** -40, 1.0 + 2.0 ** -7),  # just above the tie: up
        (-(1.0 + 2.0 ** -8 + 2.0 ** -40), -(1.0 + 2.0 ** -7)),
        (3.4e38, float("inf")),                       # past the midpoint to 2**128
        ((2.0 - 2.0 ** -8 - 2.0 ** -20) * 2.0 ** 127, (2.0 - 2.0 ** -7) * 2.0 ** 127),  # below it
        ((2.0 - 2.0 ** -7) * 2.0 ** 127, (2.0 - 2.0 ** -7) * 2.0 ** 127),
        (2.0 ** -133, 2.0 ** -133),                   # smallest subnormal
        (2.0 ** -134, 0.0),                           # tie between 0 and 2**-133 -> 0
        (3 * 2.0 ** -134, 2.0 ** -132),               # tie -> even
        (0.0, 0.0),
    ]
    x = np.array([c[0] for c in cases])
    want = np.array([c[1] for c in cases])
    np.testing.assert_array_equal(oracle.bf16_round(x), want)


def test_one_rounding_not_two():
    # Rounding through fp32 first would land on the tie and go down.
    x = np.array([1.0 + 2.0 ** -8 + 2.0 ** -40])
    assert np.float64(np.float32(x[0])) == 1.0 + 2.0 ** -8
    assert oracle.bf16_round(x)[0] == 1.0 + 2.0 ** -7
